// Block scoring (Sec. 3.1) and the global linear term o_bar = phi(q) S_bar
// (Sec. 3.2, Eq. 15), one kernel.
//
// Scoring workgroups: one per tile of 64 blocks of a (sequence, KV head);
// each wavefront takes 16 blocks, lane = (block, quarter of the head
// dimension). All of the lane's statistics loads are issued before any
// arithmetic and before the query coefficients are read (16 x 16 B in
// flight per lane), and every 16-byte load of the
// tile-interleaved statistics is a contiguous 256 B run per 16 lanes. For
// head m of the group the log block mass is
//   ell_m(i) = s q_m.mu_i + ln n_i + ln(1 + 1/2 s^2 sum_j q_mj^2 M2_ij / n_i)
// (Eqs. 8 and 10, diagonal covariance M2/n): four coordinates at a time in
// fp32, those partial sums accumulated in fp64 and summed over the four
// quarters with cross-lane shuffles; lane (block, quarter) then finishes
// heads quarter, quarter+4, ... The workgroup writes exp(ell - tile max) per
// head and block and the (max, sum) of its 64 blocks per head, from which
// the selection forms each head's normaliser Z (Eq. 9) without another pass
// over the statistics.
//
// Linear workgroups (blockIdx.x >= n_tiles): 16 rows of S_bar each,
// o_bar partial[m][c] = sum_{j in rows} phi(q_m)_j S_bar[j][c] and
// zq partial[m] = sum_{j in rows} phi(q_m)_j z_bar[j]; the merge adds the
// partials.
#include "spla_device.h"
#include "spla_kernels.h"

namespace spla {

constexpr int kScoreGroup = 16;  // blocks per wavefront

template <int G, typename T, int D>
__device__ __forceinline__ void linear_part(const Dims& m, const float* __restrict__ S,
                                            const float* __restrict__ zbar, const T* __restrict__ q,
                                            float* __restrict__ obar_part,
                                            float* __restrict__ zq_part, float (*sphi)[D],
                                            float (*sred)[G][D]) {
  constexpr int NRG = 256 / D;
  const int bh = blockIdx.y;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int chunk = blockIdx.x - m.n_tiles;
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
  const int col = tid % D, sub = tid / D;
  const int row0 = chunk * kLinRows;
  float acc[G];
#pragma unroll
  for (int mm = 0; mm < G; ++mm) acc[mm] = 0.f;
  const float* Sb = S + (int64_t)bh * D * D;
#pragma unroll
  for (int r = sub; r < kLinRows; r += NRG) {
    const float sv = Sb[(row0 + r) * D + col];
#pragma unroll
    for (int mm = 0; mm < G; ++mm) acc[mm] = fmaf(sphi[mm][row0 + r], sv, acc[mm]);
  }
#pragma unroll
  for (int mm = 0; mm < G; ++mm) sred[sub][mm][col] = acc[mm];
  __syncthreads();
  float* op = obar_part + ((int64_t)bh * (D / kLinRows) + chunk) * G * D;
  for (int e = tid; e < G * D; e += 256) {
    const int mm = e / D, c = e % D;
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < NRG; ++r) s += sred[r][mm][c];
    op[mm * D + c] = s;
  }
  if (tid < G) {
    float s = 0.f;
    for (int r = 0; r < kLinRows; ++r) s += sphi[tid][row0 + r] * zbar[(int64_t)bh * D + row0 + r];
    zq_part[((int64_t)bh * (D / kLinRows) + chunk) * G + tid] = s;
  }
}

template <int G, typename T, int D>
__global__ __launch_bounds__(256) void score_linear_kernel(
    Dims m, const float* __restrict__ stats, const float* __restrict__ S,
    const float* __restrict__ zbar, const int32_t* __restrict__ seq_lens, const T* __restrict__ q,
    double s, int first_order, float* __restrict__ e_vals, double* __restrict__ tile_part,
    float* __restrict__ obar_part, float* __restrict__ zq_part) {
  constexpr int Q = D / 4;         // coordinates per lane (one quarter of d)
  constexpr int NJ = Q / 4;        // float4 loads per lane and statistics part
  // coefficient tables, [head][group of 4 coordinates][quarter][4]: the four
  // quarters read adjacent 16-byte words (distinct banks)
  __shared__ float4 sq[G][NJ][4];
  __shared__ float4 sq2[G][NJ][4];
  __shared__ float sphi[G][D];
  __shared__ float sred[256 / D][G][D];
  __shared__ double s_part[4][G][2];
  const int bh = blockIdx.y;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if ((int)blockIdx.x >= m.n_tiles) {
    linear_part<G, T, D>(m, S, zbar, q, obar_part, zq_part, sphi, sred);
    return;
  }
  const int L = seq_lens[b];
  const int nb = (L + m.B - 1) / m.B;
  const int tile = blockIdx.x;
  if (tile * kTileBlocks >= nb) return;
  const int grp = tile * (kTileBlocks / kScoreGroup) + w;
  const bool grp_live = grp * kScoreGroup < nb;
  const int blk = grp * kScoreGroup + (lane & 15);
  const int qt = lane >> 4;  // quarter of the head dimension
  // statistics loads first; the coefficient table is built while they fly
  float4 mu[NJ], m2[NJ];
  if (grp_live) {
    const float4* pm = reinterpret_cast<const float4*>(stats + stats_off4(m, bh, blk, 0, qt * NJ));
    const float4* pv = reinterpret_cast<const float4*>(stats + stats_off4(m, bh, blk, 1, qt * NJ));
#pragma unroll
    for (int t = 0; t < NJ; ++t) mu[t] = pm[t * kTileBlocks];
    if (!first_order) {
#pragma unroll
      for (int t = 0; t < NJ; ++t) m2[t] = pv[t * kTileBlocks];
    }
  }
  for (int e = tid; e < G * D; e += 256) {
    const int mm = e / D, j = e % D;
    const float x = Elem<T>::load(q, ((int64_t)b * m.hq + h * G + mm) * D + j);
    const int qq = j / Q, jj = j % Q;
    reinterpret_cast<float*>(&sq[mm][jj / 4][qq])[jj % 4] = (float)(s * x);
    reinterpret_cast<float*>(&sq2[mm][jj / 4][qq])[jj % 4] = (float)(0.5 * s * s * x * x);
  }
  __syncthreads();
  double am[G], av[G];
#pragma unroll
  for (int mm = 0; mm < G; ++mm) am[mm] = av[mm] = 0.0;
  if (grp_live) {
    // four coordinates at a time in fp32, accumulated across groups in fp64
#pragma unroll
    for (int t = 0; t < NJ; ++t) {
#pragma unroll
      for (int mm = 0; mm < G; ++mm) {
        const float4 c = sq[mm][t][qt];
        float pa = c.x * mu[t].x;
        pa = fmaf(c.y, mu[t].y, pa);
        pa = fmaf(c.z, mu[t].z, pa);
        pa = fmaf(c.w, mu[t].w, pa);
        am[mm] += (double)pa;
        asm volatile("" : "+v"(am[mm]));  // add in coordinate order; keeps few partials live
      }
      if (!first_order) {
#pragma unroll
        for (int mm = 0; mm < G; ++mm) {
          const float4 c = sq2[mm][t][qt];
          float pb = c.x * m2[t].x;
          pb = fmaf(c.y, m2[t].y, pb);
          pb = fmaf(c.z, m2[t].z, pb);
          pb = fmaf(c.w, m2[t].w, pb);
          av[mm] += (double)pb;
          asm volatile("" : "+v"(av[mm]));
        }
      }
    }
#pragma unroll
    for (int mm = 0; mm < G; ++mm) {
      am[mm] += __shfl_xor(am[mm], 16, kWave);
      am[mm] += __shfl_xor(am[mm], 32, kWave);
      av[mm] += __shfl_xor(av[mm], 16, kWave);
      av[mm] += __shfl_xor(av[mm], 32, kWave);
    }
  }
  // every lane now holds all G sums of its block; lane (block, qt) finishes
  // heads qt, qt+4, ...: one fp64 log1p / exp per head and lane
  const bool valid = grp_live && blk < nb;
  const int n_i = valid ? block_count(L, m.B, blk) : 1;
  const double ln_n = log((double)n_i);
  const int nbp = m.n_tiles * kTileBlocks;
  float* ev = e_vals + (int64_t)bh * G * nbp;
  constexpr int U = (G + 3) / 4;
  double ell[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int mm = qt + 4 * u;
    double a = 0.0, v = 0.0;
#pragma unroll
    for (int c = 0; c < G; ++c)
      if (c == mm) {
        a = am[c];
        v = av[c];
      }
    double x = a + ln_n;
    if (!first_order) x += log1p(v / n_i);
    ell[u] = valid ? x : -INFINITY;
    double mx = ell[u];
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) mx = fmax(mx, __shfl_xor(mx, o, kWave));
    if ((lane & 15) == 0 && mm < G) s_part[w][mm][0] = mx;
  }
  __syncthreads();
  // exp(ell - tile max): the tile's 64 blocks share one offset per head
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int mm = qt + 4 * u;
    if (mm < G) {
      double tmx = -INFINITY;
#pragma unroll
      for (int x = 0; x < 4; ++x) tmx = fmax(tmx, s_part[x][mm][0]);
      const double e = valid ? exp(ell[u] - tmx) : 0.0;
      double sum = e;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) sum += __shfl_xor(sum, o, kWave);
      if (grp_live) ev[(int64_t)mm * nbp + blk] = (float)e;
      if ((lane & 15) == 0) s_part[w][mm][1] = sum;
    }
  }
  __syncthreads();
  if (tid < G) {
    double mx = -INFINITY, sum = 0.0;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      mx = fmax(mx, s_part[x][tid][0]);
      sum += s_part[x][tid][1];
    }
    double* tp = tile_part + (((int64_t)bh * m.n_tiles + tile) * G + tid) * 2;
    tp[0] = mx;
    tp[1] = sum;
  }
}

template <int G, typename T, int D>
static void score_gtd(const Dims& m, const spla_config& cfg, const spla_cache& c, const void* q,
                      const DecodeWs& ws, char* base, hipStream_t st) {
  const double s = cfg.softmax_scale > 0.f ? (double)cfg.softmax_scale : 1.0 / sqrt((double)m.d);
  dim3 grid((unsigned)(m.n_tiles + ws.n_lin), (unsigned)m.bh);
  hipLaunchKernelGGL((score_linear_kernel<G, T, D>), grid, dim3(256), 0, st, m,
                     (const float*)c.blk_stats, (const float*)c.lin_state,
                     (const float*)c.lin_norm, (const int32_t*)c.seq_lens, (const T*)q, s,
                     (int)((cfg.flags & SPLA_FLAG_FIRST_ORDER) != 0), (float*)(base + ws.e_vals),
                     (double*)(base + ws.tile_part), (float*)(base + ws.obar_part),
                     (float*)(base + ws.zq_part));
}

template <typename T, int D>
static void score_td(const Dims& m, const spla_config& cfg, const spla_cache& c, const void* q,
                     const DecodeWs& ws, char* base, hipStream_t st) {
  switch (m.group) {
#define SPLA_G(g) case g: score_gtd<g, T, D>(m, cfg, c, q, ws, base, st); break;
    SPLA_G(1) SPLA_G(2) SPLA_G(3) SPLA_G(4) SPLA_G(5) SPLA_G(6) SPLA_G(7) SPLA_G(8)
    SPLA_G(9) SPLA_G(10) SPLA_G(11) SPLA_G(12) SPLA_G(13) SPLA_G(14) SPLA_G(15) SPLA_G(16)
#undef SPLA_G
    default: break;
  }
}

hipError_t launch_score(const Dims& m, const spla_config& cfg, const spla_cache& c,
                        const void* q, const DecodeWs& ws, char* base, hipStream_t st) {
  if (m.elem == 4) {
    if (m.d == 64) score_td<float, 64>(m, cfg, c, q, ws, base, st);
    else score_td<float, 128>(m, cfg, c, q, ws, base, st);
  } else {
    if (m.d == 64) score_td<bf16_t, 64>(m, cfg, c, q, ws, base, st);
    else score_td<bf16_t, 128>(m, cfg, c, q, ws, base, st);
  }
  return hipGetLastError();
}

}  // namespace spla
