// Fused pass over the selected blocks and the merge (Secs. 2.2, 3.2, 3.3).
//
// sparse: workgroup (split, sequence x KV head) reads its selected blocks
// once, 32 tokens at a time, and from that single read accumulates
//   - the exact softmax branch of Eq. (5): online max m, normaliser l and
//     acc = sum_t exp(s q.k_t - m) v_t for each of the G heads, and
//   - the selected-token linear term of Eq. (16):
//     accw = sum_t <phi(q), phi(k_t)> v_t, zw = sum_t <phi(q), phi(k_t)>.
// merge: combines the splits, forms r = o_bar - o_tilde (Eq. 14; exactly 0
// when every token is selected), and writes
//   out = o_sparse + gamma * r / sqrt(mean(r^2) + eps)   (Sec. 3.3).
#include "spla_device.h"
#include "spla_kernels.h"

namespace spla {

template <typename T, int D>
__global__ __launch_bounds__(256) void sparse_valu_kernel(
    Dims m, float s, const T* __restrict__ kc, const T* __restrict__ vc,
    const T* __restrict__ q, const int32_t* __restrict__ sel, const int32_t* __restrict__ meta,
    int n_splits, int bps, int stride, float* __restrict__ part) {
  constexpr int MG = SPLA_MAX_GROUP;
  constexpr int PER = (MG * D + 255) / 256;  // (head, coord) pairs per thread
  __shared__ float sq[MG][D];
  __shared__ float sphq[MG][D];
  __shared__ float sK[kSubTokens][D + 1];
  __shared__ float sE[kSubTokens][D + 1];
  __shared__ float sV[D][kSubTokens + 1];
  __shared__ float sP[MG][kSubTokens];
  __shared__ float sW[MG][kSubTokens];
  __shared__ float s_m[MG], s_l[MG], s_alpha[MG], s_zw[MG];
  const int bh = blockIdx.y, split = blockIdx.x;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nsel = meta[bh * 4 + 0];
  const int L = meta[bh * 4 + 2];
  const int p0 = split * bps, p1 = min(p0 + bps, nsel);

  for (int mm = w; mm < G; mm += 4) {
    float x[D / 64];
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      x[e] = Elem<T>::load(q, ((int64_t)b * m.hq + h * G + mm) * D + lane + 64 * e);
      sq[mm][lane + 64 * e] = s * x[e];
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
    for (int e = 0; e < D / 64; ++e) sphq[mm][lane + 64 * e] = x[e] / sum;
  }
  if (tid < MG) {
    s_m[tid] = -INFINITY;
    s_l[tid] = 0.f;
    s_zw[tid] = 0.f;
  }
  float acc[PER], accw[PER];
#pragma unroll
  for (int r = 0; r < PER; ++r) acc[r] = accw[r] = 0.f;
  __syncthreads();

  for (int p = p0; p < p1; ++p) {
    const int blk = sel[(int64_t)bh * m.k + p];
    const int n_i = block_count(L, m.B, blk);
    for (int sub = 0; sub * kSubTokens < n_i; ++sub) {
      const int t0 = blk * m.B + sub * kSubTokens;
      const int nt = min(kSubTokens, n_i - sub * kSubTokens);
      for (int e = tid; e < kSubTokens * D; e += 256) {
        const int row = e / D, col = e % D;
        sK[row][col] = row < nt ? Elem<T>::load(kc, k_off(m, bh, t0 + row, col)) : 0.f;
        const int c2 = e / kSubTokens, r2 = e % kSubTokens;
        sV[c2][r2] = r2 < nt ? Elem<T>::load(vc, v_off(m, bh, t0 + r2, c2)) : 0.f;
      }
      __syncthreads();
      for (int r = 0; r < kSubTokens / 4; ++r) {  // phi(k) rows
        const int row = w * (kSubTokens / 4) + r;
        float x[D / 64];
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < D / 64; ++e) {
          x[e] = sK[row][lane + 64 * e];
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
        const float inv = row < nt ? 1.0f / sum : 0.f;
#pragma unroll
        for (int e = 0; e < D / 64; ++e) sE[row][lane + 64 * e] = x[e] * inv;
      }
      __syncthreads();
      for (int e = tid; e < G * kSubTokens; e += 256) {  // logits and linear weights
        const int mm = e / kSubTokens, t = e % kSubTokens;
        float a = 0.f, wl = 0.f;
        for (int j = 0; j < D; ++j) {
          a = fmaf(sq[mm][j], sK[t][j], a);
          wl = fmaf(sphq[mm][j], sE[t][j], wl);
        }
        sP[mm][t] = t < nt ? a : -INFINITY;
        sW[mm][t] = t < nt ? wl : 0.f;
      }
      __syncthreads();
      if (tid < G) {  // online softmax bookkeeping, one head per thread
        const int mm = tid;
        float mx = s_m[mm];
        for (int t = 0; t < nt; ++t) mx = fmaxf(mx, sP[mm][t]);
        const float alpha = expf(s_m[mm] - mx);
        float l = s_l[mm] * alpha, zw = s_zw[mm];
        for (int t = 0; t < kSubTokens; ++t) {
          const float pv = t < nt ? expf(sP[mm][t] - mx) : 0.f;
          sP[mm][t] = pv;
          l += pv;
          zw += sW[mm][t];
        }
        s_m[mm] = mx;
        s_l[mm] = l;
        s_alpha[mm] = alpha;
        s_zw[mm] = zw;
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < PER; ++r) {
        const int idx = tid + 256 * r;
        if (idx < G * D) {
          const int mm = idx / D, c = idx % D;
          float a = acc[r] * s_alpha[mm], aw = accw[r];
          for (int t = 0; t < nt; ++t) {
            a = fmaf(sP[mm][t], sV[c][t], a);
            aw = fmaf(sW[mm][t], sV[c][t], aw);
          }
          acc[r] = a;
          accw[r] = aw;
        }
      }
      __syncthreads();
    }
  }
  float* out = part + ((int64_t)bh * n_splits + split) * G * stride;
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int idx = tid + 256 * r;
    if (idx < G * D) {
      const int mm = idx / D, c = idx % D;
      out[mm * stride + 4 + c] = acc[r];
      out[mm * stride + 4 + D + c] = accw[r];
    }
  }
  if (tid < G) {
    out[tid * stride + 0] = s_m[tid];
    out[tid * stride + 1] = s_l[tid];
    out[tid * stride + 2] = s_zw[tid];
    out[tid * stride + 3] = 0.f;
  }
}

template <typename T, int D>
__global__ __launch_bounds__(256) void merge_kernel(
    Dims m, float eps, uint32_t flags, const float* __restrict__ gamma,
    const int32_t* __restrict__ meta, const float* __restrict__ part, int n_splits, int bps,
    int stride, const float* __restrict__ obar, const float* __restrict__ zq, T* __restrict__ out) {
  const int bh = blockIdx.x;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nsel = meta[bh * 4 + 0];
  const int all_sel = meta[bh * 4 + 1];
  const int L = meta[bh * 4 + 2];
  const int n_used = (nsel + bps - 1) / bps;
  const float* pb = part + (int64_t)bh * n_splits * G * stride;
  for (int mm = w; mm < G; mm += 4) {
    const int64_t orow = ((int64_t)b * m.hq + h * G + mm) * D;
    if (L == 0) {
#pragma unroll
      for (int e = 0; e < D / 64; ++e) Elem<T>::store(out, orow + lane + 64 * e, 0.f);
      continue;
    }
    float M = -INFINITY;
    for (int x = 0; x < n_used; ++x) M = fmaxf(M, pb[((int64_t)x * G + mm) * stride]);
    float l = 0.f, zt = 0.f;
    float osp[D / 64], ot[D / 64];
#pragma unroll
    for (int e = 0; e < D / 64; ++e) osp[e] = ot[e] = 0.f;
    for (int x = 0; x < n_used; ++x) {
      const float* px = pb + ((int64_t)x * G + mm) * stride;
      const float sc = expf(px[0] - M);
      l = fmaf(px[1], sc, l);
      zt += px[2];
#pragma unroll
      for (int e = 0; e < D / 64; ++e) {
        osp[e] = fmaf(px[4 + lane + 64 * e], sc, osp[e]);
        ot[e] += px[4 + D + lane + 64 * e];
      }
    }
    float r[D / 64];
    float ss = 0.f;
    const bool rla = !(flags & SPLA_FLAG_NO_RLA);
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      osp[e] /= l;
      r[e] = 0.f;
      if (rla && !all_sel) r[e] = obar[((int64_t)bh * G + mm) * D + lane + 64 * e] - ot[e];
    }
    if (rla && !all_sel && (flags & SPLA_FLAG_RLA_NORMALIZE)) {
      const float den = zq[(int64_t)bh * G + mm] - zt;
#pragma unroll
      for (int e = 0; e < D / 64; ++e) r[e] /= den;
    }
#pragma unroll
    for (int e = 0; e < D / 64; ++e) ss += r[e] * r[e];
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / D + eps);
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      const int c = lane + 64 * e;
      float o = osp[e];
      if (rla) o = fmaf(gamma[(int64_t)(h * G + mm) * D + c] * r[e], inv, o);
      Elem<T>::store(out, orow + c, o);
    }
  }
}

template <typename T, int D>
static void sparse_td(const Dims& m, float s, const spla_cache& c, const void* q,
                      const DecodeWs& ws, char* base, hipStream_t st) {
  hipLaunchKernelGGL((sparse_valu_kernel<T, D>), dim3(ws.n_splits, m.bh), dim3(256), 0, st, m, s,
                     (const T*)c.k_cache, (const T*)c.v_cache, (const T*)q,
                     (const int32_t*)(base + ws.sel), (const int32_t*)(base + ws.meta),
                     ws.n_splits, ws.blocks_per_split, ws.split_stride,
                     (float*)(base + ws.split));
}

hipError_t launch_sparse(const Dims& m, const spla_config& cfg, const spla_cache& c,
                         const void* q, const DecodeWs& ws, char* base, hipStream_t st) {
  const float s = cfg.softmax_scale > 0.f ? cfg.softmax_scale : (float)(1.0 / sqrt((double)m.d));
  if (m.elem == 4) {
    if (m.d == 64) sparse_td<float, 64>(m, s, c, q, ws, base, st);
    else sparse_td<float, 128>(m, s, c, q, ws, base, st);
  } else {
    if (m.d == 64) sparse_td<bf16_t, 64>(m, s, c, q, ws, base, st);
    else sparse_td<bf16_t, 128>(m, s, c, q, ws, base, st);
  }
  return hipGetLastError();
}

template <typename T, int D>
static void merge_td(const Dims& m, const spla_config& cfg, const float* gamma, void* out,
                     const DecodeWs& ws, char* base, hipStream_t st) {
  hipLaunchKernelGGL((merge_kernel<T, D>), dim3(m.bh), dim3(256), 0, st, m, cfg.rms_eps,
                     cfg.flags, gamma, (const int32_t*)(base + ws.meta),
                     (const float*)(base + ws.split), ws.n_splits, ws.blocks_per_split,
                     ws.split_stride, (const float*)(base + ws.obar),
                     (const float*)(base + ws.zq), (T*)out);
}

hipError_t launch_merge(const Dims& m, const spla_config& cfg, const float* gamma, void* out,
                        const DecodeWs& ws, char* base, hipStream_t st) {
  if (m.elem == 4) {
    if (m.d == 64) merge_td<float, 64>(m, cfg, gamma, out, ws, base, st);
    else merge_td<float, 128>(m, cfg, gamma, out, ws, base, st);
  } else {
    if (m.d == 64) merge_td<bf16_t, 64>(m, cfg, gamma, out, ws, base, st);
    else merge_td<bf16_t, 128>(m, cfg, gamma, out, ws, base, st);
  }
  return hipGetLastError();
}

}  // namespace spla
