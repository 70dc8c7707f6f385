// Block scoring (Sec. 3.1) and the global linear term o_bar = phi(q) S_bar
// (Sec. 3.2, Eq. 15).
//
// score: every (sequence, KV head) streams all of its block statistics once.
// One wavefront handles one tile of 64 blocks, lane = block, so each
// 16-byte load of the tile-interleaved statistics is a contiguous 1 KiB per
// wavefront. For head m of the group the log block mass is
//   ell_m(i) = s q_m.mu_i + ln n_i + ln(1 + 1/2 s^2 sum_j q_mj^2 M2_ij / n_i)
// (Eqs. 8 and 10 with the diagonal covariance M2/n), accumulated in fp64.
// The tile then writes exp(ell - tile max) per head and block, and the
// tile's (max, sum) per head, from which the selection forms each head's
// normaliser Z (Eq. 9) without another pass over the statistics.
#include "spla_device.h"
#include "spla_kernels.h"

namespace spla {

constexpr int kScoreWaves = 4;

template <int G, typename T>
__global__ __launch_bounds__(256) void score_kernel(
    Dims m, const float* __restrict__ stats, const int32_t* __restrict__ seq_lens,
    const T* __restrict__ q, double s, int first_order, float* __restrict__ e_vals,
    double* __restrict__ tile_part) {
  __shared__ double sq[G][128];
  __shared__ double sq2[G][128];
  const int bh = blockIdx.y;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int D = m.d;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int e = tid; e < G * D; e += 256) {
    const int mm = e / D, j = e % D;
    const double x = (double)Elem<T>::load(q, ((int64_t)b * m.hq + h * G + mm) * D + j);
    sq[mm][j] = s * x;
    sq2[mm][j] = 0.5 * s * s * x * x;
  }
  __syncthreads();
  const int L = seq_lens[b];
  const int nb = (L + m.B - 1) / m.B;
  const int tile = blockIdx.x * kScoreWaves + w;
  if (tile >= m.n_tiles || tile * kTileBlocks >= nb) return;
  const int i = tile * kTileBlocks + lane;
  const bool valid = i < nb;

  double am[G], av[G];
#pragma unroll
  for (int mm = 0; mm < G; ++mm) am[mm] = av[mm] = 0.0;
  const float4* pm = reinterpret_cast<const float4*>(stats + stats_off4(m, bh, i, 0, 0));
  const float4* pv = reinterpret_cast<const float4*>(stats + stats_off4(m, bh, i, 1, 0));
  for (int j4 = 0; j4 < D / 4; ++j4) {
    const float4 mu = pm[j4 * kTileBlocks];
    const float4 m2 = pv[j4 * kTileBlocks];
    const double mv[4] = {mu.x, mu.y, mu.z, mu.w};
    const double vv[4] = {m2.x, m2.y, m2.z, m2.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
#pragma unroll
      for (int mm = 0; mm < G; ++mm) {
        am[mm] = fma(sq[mm][4 * j4 + e], mv[e], am[mm]);
        av[mm] = fma(sq2[mm][4 * j4 + e], vv[e], av[mm]);
      }
    }
  }
  const int n_i = valid ? block_count(L, m.B, i) : 1;
  const double ln_n = log((double)n_i);
  float* ev = e_vals + (int64_t)bh * G * m.n_tiles * kTileBlocks;
  double* tp = tile_part + ((int64_t)bh * m.n_tiles + tile) * G * 2;
#pragma unroll
  for (int mm = 0; mm < G; ++mm) {
    double ell = am[mm] + ln_n;
    if (!first_order) ell += log1p(av[mm] / n_i);
    if (!valid) ell = -INFINITY;
    const double mx = wave_max(ell);
    const double e = valid ? exp(ell - mx) : 0.0;
    const double sum = wave_sum(e);
    ev[(int64_t)mm * m.n_tiles * kTileBlocks + i] = (float)e;
    if (lane == 0) {
      tp[mm * 2 + 0] = mx;
      tp[mm * 2 + 1] = sum;
    }
  }
}

// o_bar[m][c] = sum_j phi(q_m)_j S_bar[j][c]  and  zq[m] = <phi(q_m), z_bar>.
template <typename T, int D>
__global__ __launch_bounds__(256) void linear_kernel(Dims m, const float* __restrict__ S,
                                                     const float* __restrict__ zbar,
                                                     const int32_t* __restrict__ seq_lens,
                                                     const T* __restrict__ q,
                                                     float* __restrict__ obar,
                                                     float* __restrict__ zq) {
  constexpr int NRG = 256 / D;
  __shared__ float sphi[SPLA_MAX_GROUP][D];
  __shared__ float sred[NRG][SPLA_MAX_GROUP][D];
  const int bh = blockIdx.x;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int mm = w; mm < G; mm += 4) {
    float x[D / 64];
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      x[e] = Elem<T>::load(q, ((int64_t)b * m.hq + h * G + mm) * D + lane + 64 * e);
      mx = fmaxf(mx, x[e]);
    }
    mx = wave_max(mx);
    float sum = 0.f;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      x[e] = expf(x[e] - mx);
      sum += x[e];
    }
    sum = wave_sum(sum);
#pragma unroll
    for (int e = 0; e < D / 64; ++e) sphi[mm][lane + 64 * e] = x[e] / sum;
  }
  __syncthreads();
  const int col = tid % D, rg = tid / D;
  float acc[SPLA_MAX_GROUP];
#pragma unroll
  for (int mm = 0; mm < SPLA_MAX_GROUP; ++mm) acc[mm] = 0.f;
  const float* Sb = S + (int64_t)bh * D * D;
  for (int j = rg; j < D; j += NRG) {
    const float sv = Sb[j * D + col];
#pragma unroll
    for (int mm = 0; mm < SPLA_MAX_GROUP; ++mm)
      if (mm < G) acc[mm] = fmaf(sphi[mm][j], sv, acc[mm]);
  }
#pragma unroll
  for (int mm = 0; mm < SPLA_MAX_GROUP; ++mm)
    if (mm < G) sred[rg][mm][col] = acc[mm];
  __syncthreads();
  for (int e = tid; e < G * D; e += 256) {
    const int mm = e / D, c = e % D;
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < NRG; ++r) s += sred[r][mm][c];
    obar[((int64_t)bh * G + mm) * D + c] = s;
  }
  for (int mm = w; mm < G; mm += 4) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) s += sphi[mm][lane + 64 * e] * zbar[(int64_t)bh * D + lane + 64 * e];
    s = wave_sum(s);
    if (lane == 0) zq[(int64_t)bh * G + mm] = s;
  }
  (void)seq_lens;
}

template <int G, typename T>
static void score_g(const Dims& m, const spla_config& cfg, const spla_cache& c, const void* q,
                    const DecodeWs& ws, char* base, hipStream_t st) {
  const double s = cfg.softmax_scale > 0.f ? (double)cfg.softmax_scale : 1.0 / sqrt((double)m.d);
  dim3 grid((unsigned)ceil_div(m.n_tiles, kScoreWaves), (unsigned)m.bh);
  hipLaunchKernelGGL((score_kernel<G, T>), grid, dim3(256), 0, st, m, (const float*)c.blk_stats,
                     (const int32_t*)c.seq_lens, (const T*)q, s,
                     (int)((cfg.flags & SPLA_FLAG_FIRST_ORDER) != 0), (float*)(base + ws.e_vals),
                     (double*)(base + ws.tile_part));
}

template <typename T>
static void score_t(const Dims& m, const spla_config& cfg, const spla_cache& c, const void* q,
                    const DecodeWs& ws, char* base, hipStream_t st) {
  switch (m.group) {
#define SPLA_G(g) case g: score_g<g, T>(m, cfg, c, q, ws, base, st); break;
    SPLA_G(1) SPLA_G(2) SPLA_G(3) SPLA_G(4) SPLA_G(5) SPLA_G(6) SPLA_G(7) SPLA_G(8)
    SPLA_G(9) SPLA_G(10) SPLA_G(11) SPLA_G(12) SPLA_G(13) SPLA_G(14) SPLA_G(15) SPLA_G(16)
#undef SPLA_G
    default: break;
  }
}

hipError_t launch_score(const Dims& m, const spla_config& cfg, const spla_cache& c,
                        const void* q, const DecodeWs& ws, char* base, hipStream_t st) {
  if (m.elem == 4) score_t<float>(m, cfg, c, q, ws, base, st);
  else score_t<bf16_t>(m, cfg, c, q, ws, base, st);
  return hipGetLastError();
}

hipError_t launch_linear(const Dims& m, const spla_config& cfg, const spla_cache& c,
                         const void* q, const DecodeWs& ws, char* base, hipStream_t st) {
  (void)cfg;
  float* obar = (float*)(base + ws.obar);
  float* zq = (float*)(base + ws.zq);
  if (m.elem == 4) {
    if (m.d == 64)
      hipLaunchKernelGGL((linear_kernel<float, 64>), dim3(m.bh), dim3(256), 0, st, m,
                         c.lin_state, c.lin_norm, c.seq_lens, (const float*)q, obar, zq);
    else
      hipLaunchKernelGGL((linear_kernel<float, 128>), dim3(m.bh), dim3(256), 0, st, m,
                         c.lin_state, c.lin_norm, c.seq_lens, (const float*)q, obar, zq);
  } else {
    if (m.d == 64)
      hipLaunchKernelGGL((linear_kernel<bf16_t, 64>), dim3(m.bh), dim3(256), 0, st, m,
                         c.lin_state, c.lin_norm, c.seq_lens, (const bf16_t*)q, obar, zq);
    else
      hipLaunchKernelGGL((linear_kernel<bf16_t, 128>), dim3(m.bh), dim3(256), 0, st, m,
                         c.lin_state, c.lin_norm, c.seq_lens, (const bf16_t*)q, obar, zq);
  }
  return hipGetLastError();
}

}  // namespace spla
