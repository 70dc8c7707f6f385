// Block selection for one (sequence, KV head) per workgroup (Sec. 2.1 Eq. 3
// with Select = TopK; Sec. 2.2 Eq. 6 group score; Sec. 4 forced blocks).
//
// 1. Each head's normaliser Z_m (Eq. 9) is the log-sum-exp of the tile
//    partials written by the score pass; w[tile][m] = exp(tile max - Z_m).
// 2. score(i) = sum_m e_m(i) * w[tile(i)][m]   (fp64 accumulate, fp32 key).
// 3. Forced blocks (the first n_sink, the last n_local) are always taken;
//    the rest is a most-significant-digit radix select of the top
//    (k - forced) keys over 4 passes of 8 bits, ties going to the lower
//    block id; the result is written in ascending order.
#include "spla_device.h"
#include "spla_kernels.h"

namespace spla {

constexpr int kSelThreads = 1024;
constexpr int kSelPerThread = SPLA_MAX_BLOCKS / kSelThreads;  // 32
constexpr int kSelMaxTiles = SPLA_MAX_BLOCKS / kTileBlocks;   // 512

// Block-wide exclusive prefix sum of `v`; returns the prefix, sets *total.
__device__ __forceinline__ int block_excl_scan(int v, int* lds /*[16]*/, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds[w] = x;
  __syncthreads();
  int base = 0, tot = 0;
  for (int i = 0; i < kSelThreads / 64; ++i) {
    const int t = lds[i];
    if (i < w) base += t;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return base + x - v;
}

template <typename T, bool IS_MAX>
__device__ __forceinline__ T block_reduce(T v, T* lds /*[16]*/) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = IS_MAX ? wave_max(v) : wave_sum(v);
  if (lane == 0) lds[w] = v;
  __syncthreads();
  T r = lds[0];
  for (int i = 1; i < kSelThreads / 64; ++i) r = IS_MAX ? (lds[i] > r ? lds[i] : r) : r + lds[i];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const float* __restrict__ e_vals,
    const double* __restrict__ tile_part, int32_t* __restrict__ sel_ws,
    int32_t* __restrict__ sel_out, int32_t* __restrict__ meta) {
  __shared__ float sw[kSelMaxTiles * SPLA_MAX_GROUP];  // w[tile][m]
  __shared__ double dred[16];
  __shared__ int ired[16];
  __shared__ int hist[256];
  __shared__ int s_digit, s_above;
  const int bh = blockIdx.x;
  const int b = bh / m.hkv;
  const int G = m.group, k = m.k;
  const int tid = threadIdx.x;
  const int L = seq_lens[b];
  const int nb = (L + m.B - 1) / m.B;
  int32_t* sel = sel_ws + (int64_t)bh * k;
  int32_t* so = sel_out ? sel_out + (int64_t)bh * k : nullptr;
  if (nb <= k) {  // L == 0 included: nothing or everything is selected
    for (int x = tid; x < k; x += kSelThreads) {
      const int v = x < nb ? x : -1;
      sel[x] = v;
      if (so) so[x] = v;
    }
    if (tid == 0) {
      meta[bh * 4 + 0] = nb;
      meta[bh * 4 + 1] = 1;
      meta[bh * 4 + 2] = L;
      meta[bh * 4 + 3] = 0;
    }
    return;
  }
  const int ntu = (nb + kTileBlocks - 1) / kTileBlocks;
  const int nbp = m.n_tiles * kTileBlocks;
  // --- 1. per-head normalisers and tile weights.
  const double* tp = tile_part + (int64_t)bh * m.n_tiles * G * 2;
  for (int mm = 0; mm < G; ++mm) {
    double mx = -INFINITY;
    for (int t = tid; t < ntu; t += kSelThreads) mx = fmax(mx, tp[(t * G + mm) * 2]);
    mx = block_reduce<double, true>(mx, dred);
    double sm = 0.0;
    for (int t = tid; t < ntu; t += kSelThreads)
      sm += tp[(t * G + mm) * 2 + 1] * exp(tp[(t * G + mm) * 2] - mx);
    sm = block_reduce<double, false>(sm, dred);
    for (int t = tid; t < ntu; t += kSelThreads)
      sw[t * G + mm] = (float)(exp(tp[(t * G + mm) * 2] - mx) / sm);
  }
  __syncthreads();
  // --- 2. keys. Thread t owns the contiguous blocks [t*R, t*R + R).
  const int R = (nb + kSelThreads - 1) / kSelThreads;
  const int n_sink = m.n_sink, n_local = m.n_local;
  const int kp = k - n_sink - n_local;  // blocks chosen by rank
  const float* ev = e_vals + (int64_t)bh * G * nbp;
  uint32_t key[kSelPerThread];
#pragma unroll
  for (int r = 0; r < kSelPerThread; ++r) {
    key[r] = 0u;
    const int i = tid * R + r;
    if (r < R && i < nb && i >= n_sink && i < nb - n_local) {
      const int t = i / kTileBlocks;
      double sc = 0.0;
      for (int mm = 0; mm < G; ++mm)
        sc += (double)ev[(int64_t)mm * nbp + i] * (double)sw[t * G + mm];
      key[r] = __float_as_uint((float)sc) + 1u;
    }
  }
  // --- 3. radix select of the kp-th largest key.
  uint32_t prefix = 0u, mask = 0u;
  int remaining = kp;
  if (kp == 0) prefix = 0xFFFFFFFFu;  // no block is chosen by rank
  for (int shift = 24; shift >= 0 && kp > 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSelPerThread; ++r)
      if (r < R && (key[r] & mask) == prefix) atomicAdd(&hist[(key[r] >> shift) & 255u], 1);
    __syncthreads();
    if (tid < 64) {
      // lane l owns digits 255-4l .. 252-4l (descending)
      int c[4], loc = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        c[e] = hist[255 - 4 * tid - e];
        loc += c[e];
      }
      int incl = loc;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (tid >= o) incl += y;
      }
      int above = incl - loc;  // keys with a larger digit (within prefix)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (above < remaining && above + c[e] >= remaining) {
          s_digit = 255 - 4 * tid - e;
          s_above = above;
        }
        above += c[e];
      }
    }
    __syncthreads();
    prefix |= ((uint32_t)s_digit) << shift;
    mask |= 255u << shift;
    remaining -= s_above;
    __syncthreads();
  }
  const uint32_t thr = prefix;  // kp-th largest key; take `remaining` of the ties
  // --- 4. ties in ascending block order, then ordered compaction.
  int n_eq = 0;
#pragma unroll
  for (int r = 0; r < kSelPerThread; ++r)
    if (r < R && key[r] == thr) ++n_eq;
  int tot;
  int eq_rank = block_excl_scan(n_eq, ired, &tot);
  int n_take = 0;
  uint32_t take_bits = 0u;
#pragma unroll
  for (int r = 0; r < kSelPerThread; ++r) {
    const int i = tid * R + r;
    bool t = false;
    if (r < R && i < nb) {
      if (i < n_sink || i >= nb - n_local) t = true;
      else if (key[r] > thr) t = true;
      else if (key[r] == thr) {
        t = eq_rank < remaining;
        ++eq_rank;
      }
    }
    if (t) {
      take_bits |= 1u << r;
      ++n_take;
    }
  }
  int pos = block_excl_scan(n_take, ired, &tot);
#pragma unroll
  for (int r = 0; r < kSelPerThread; ++r) {
    if (take_bits & (1u << r)) {
      const int i = tid * R + r;
      if (pos < k) {
        sel[pos] = i;
        if (so) so[pos] = i;
      }
      ++pos;
    }
  }
  if (tid == 0) {
    meta[bh * 4 + 0] = tot < k ? tot : k;
    meta[bh * 4 + 1] = 0;
    meta[bh * 4 + 2] = L;
    meta[bh * 4 + 3] = tot;
  }
  for (int x = tot + tid; x < k; x += kSelThreads) {
    sel[x] = -1;
    if (so) so[x] = -1;
  }
}

hipError_t launch_select(const Dims& m, const spla_cache& c, const DecodeWs& ws, char* base,
                         int32_t* sel_out, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(m.bh), dim3(kSelThreads), 0, st, m, c.seq_lens,
                     (const float*)(base + ws.e_vals), (const double*)(base + ws.tile_part),
                     (int32_t*)(base + ws.sel), sel_out, (int32_t*)(base + ws.meta));
  return hipGetLastError();
}

}  // namespace spla
