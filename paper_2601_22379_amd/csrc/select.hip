// Block selection, one workgroup per (sequence, KV head) (Sec. 2.1 Eq. 3 with
// Select = TopK; Sec. 2.2 Eq. 6 group score; Sec. 4 forced blocks).
//
// 1. Each head's normaliser Z_m (Eq. 9) is the log-sum-exp of the 64-block
//    tile partials of the score pass (fp64).
// 2. score(i) = sum_m e_m(i) exp(M_tile(i),m - Z_m), fp64 accumulation,
//    rounded to an fp32 key (scores are positive, so the bit patterns order
//    like the values; +1 keeps every candidate above the excluded 0). Thread
//    t owns the R consecutive blocks t*R .. t*R + R - 1.
// 3. Every wavefront picks its own best kp = k - forced keys (ties to the
//    lower block id) with a 2-bit-per-round search whose counts come from
//    ballots - no barriers. A block beaten by kp blocks of its own wavefront
//    cannot be in the global top kp, so the union of these candidates holds
//    the answer; one wavefront then runs the same search over the union.
// 4. The forced blocks (first n_sink, last n_local) and the winners are set
//    in a bitmap and written out in ascending block order.
#include "spla_device.h"
#include "spla_kernels.h"

namespace spla {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

// Largest v with #{keys >= v} >= kp over one wavefront's keys (uniform).
// Returns 0 when fewer than kp keys are non-zero.
template <int R>
__device__ __forceinline__ uint32_t wave_kth_largest(const uint32_t (&key)[R], int kp) {
  uint32_t v = 0u;
  for (int bit = 30; bit >= 0; bit -= 2) {
    const uint32_t c1 = v | (1u << bit), c2 = v | (2u << bit), c3 = v | (3u << bit);
    int n1 = 0, n2 = 0, n3 = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      n1 += __popcll(__ballot(key[r] >= c1));
      n2 += __popcll(__ballot(key[r] >= c2));
      n3 += __popcll(__ballot(key[r] >= c3));
    }
    if (n3 >= kp) v = c3;
    else if (n2 >= kp) v = c2;
    else if (n1 >= kp) v = c1;
  }
  return v;
}

// Wavefront-wide exclusive prefix sum (lane order).
__device__ __forceinline__ int wave_excl_scan(int v, int* total) {
  const int lane = threadIdx.x & 63;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  *total = __shfl(x, 63, 64);
  return x - v;
}

// Bit r of the result marks key[r] as one of this wavefront's best kp keys in
// (key, lower index) order, keys being ordered by (lane, r) = ascending block
// id. R <= 64.
template <int R>
__device__ __forceinline__ uint64_t wave_choose(const uint32_t (&key)[R], int kp) {
  uint32_t thr = wave_kth_largest<R>(key, kp);
  if (thr == 0u) thr = 1u;  // fewer than kp non-zero keys: take every one
  int n_gt = 0, n_eq = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    n_gt += __popcll(__ballot(key[r] > thr));
    n_eq += key[r] == thr ? 1 : 0;
  }
  int eq_tot;
  int eq_rank = wave_excl_scan(n_eq, &eq_tot);
  const int need = kp - n_gt;
  uint64_t take = 0ull;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    bool t = key[r] > thr;
    if (key[r] == thr) {
      t = eq_rank < need;
      ++eq_rank;
    }
    take |= (uint64_t)(t ? 1u : 0u) << r;
  }
  return take;
}

// Block-wide exclusive prefix sum of `v`; returns the prefix, sets *total.
__device__ __forceinline__ int block_excl_scan(int v, int* lds /*[kSelWaves]*/, int* total) {
  const int w = threadIdx.x >> 6;
  int wt;
  const int x = wave_excl_scan(v, &wt);
  if ((threadIdx.x & 63) == 0) lds[w] = wt;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelWaves; ++i) {
    const int t = lds[i];
    base += i < w ? t : 0;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return base + x;
}

// Wavefront 0: the global top kp among the per-wavefront candidates. Slot
// order (lane-major) is block order, so ties again go to the lower block id.
template <int RC>
__device__ __forceinline__ void final_choose(const unsigned long long* cand, const int* wave_cnt,
                                             int kp, uint32_t* bitmap) {
  const int lane = threadIdx.x & 63;
  uint32_t ck[RC];
#pragma unroll
  for (int r = 0; r < RC; ++r) {
    const int slot = lane * RC + r;
    const int sw = slot / kp, so = slot % kp;
    ck[r] = (sw < kSelWaves && so < wave_cnt[sw]) ? (uint32_t)(cand[sw * kp + so] >> 32) : 0u;
  }
  uint64_t tk = wave_choose<RC>(ck, kp);
  while (tk) {
    const int r = __ffsll((unsigned long long)tk) - 1;
    tk &= tk - 1;
    const int slot = lane * RC + r;
    const uint32_t i = (uint32_t)cand[(slot / kp) * kp + slot % kp];
    atomicOr(&bitmap[i >> 5], 1u << (i & 31));
  }
}

template <int R>
__global__ __launch_bounds__(kSelThreads) void select_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const float* __restrict__ e_vals,
    const double* __restrict__ tile_part, int32_t* __restrict__ sel_ws,
    int32_t* __restrict__ sel_out, int32_t* __restrict__ meta) {
  constexpr int kMaxTW = 8192;                       // (tile, head) weights kept in LDS
  __shared__ double sZ[SPLA_MAX_GROUP];
  __shared__ float sw[kMaxTW];
  __shared__ unsigned long long cand[kSelWaves * SPLA_MAX_TOP_K];
  __shared__ int wave_cnt[kSelWaves];
  __shared__ int scan_lds[kSelWaves];
  __shared__ uint32_t bitmap[SPLA_MAX_BLOCKS / 32];
  const int bh = blockIdx.x;
  const int b = bh / m.hkv;
  const int G = m.group, k = m.k;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nbp = m.n_tiles * kTileBlocks;
  const int i0 = tid * R;
  const int kp = k - m.n_sink - m.n_local;
  const double* tp = tile_part + (int64_t)bh * m.n_tiles * G * 2;
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
  const int n_tu = (nb + kTileBlocks - 1) / kTileBlocks;
  const int n_words = (nb + 31) / 32;
  for (int x = tid; x < n_words; x += kSelThreads) bitmap[x] = 0u;
  __syncthreads();
  if (kp > 0) {
    // --- 1. Z_m: wavefront w handles heads w, w + 16, ...
    for (int mm = w; mm < G; mm += kSelWaves) {
      double mx = -INFINITY;
      for (int t = lane; t < n_tu; t += 64) mx = fmax(mx, tp[(t * G + mm) * 2]);
      mx = wave_max(mx);
      double sm = 0.0;
      for (int t = lane; t < n_tu; t += 64) {
        const double tm = tp[(t * G + mm) * 2];
        if (tm > -INFINITY) sm += tp[(t * G + mm) * 2 + 1] * exp(tm - mx);
      }
      sm = wave_sum(sm);
      if (lane == 0) sZ[mm] = mx + log(sm);
    }
    __syncthreads();
    const bool w_lds = n_tu * G <= kMaxTW;
    if (w_lds)
      for (int x = tid; x < n_tu * G; x += kSelThreads) {
        const double tm = tp[x * 2];
        sw[x] = tm > -INFINITY ? (float)exp(tm - sZ[x % G]) : 0.f;
      }
    __syncthreads();
    // --- 2. keys
    double sc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) sc[r] = 0.0;
    for (int mm = 0; mm < G; ++mm) {
      const float* ev = e_vals + ((int64_t)bh * G + mm) * nbp + i0;
      float e[R];
#pragma unroll
      for (int r = 0; r < R; ++r) e[r] = i0 + r < nb ? ev[r] : 0.f;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int t = (i0 + r) / kTileBlocks;
        double wv;
        if (w_lds) {
          wv = t < n_tu ? (double)sw[t * G + mm] : 0.0;
        } else {
          const double tm = t < n_tu ? tp[(t * G + mm) * 2] : -INFINITY;
          wv = tm > -INFINITY ? exp(tm - sZ[mm]) : 0.0;
        }
        sc[r] = fma((double)e[r], wv, sc[r]);
      }
    }
    uint32_t key[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = i0 + r;
      key[r] = (i < nb && i >= m.n_sink && i < nb - m.n_local)
                   ? __float_as_uint((float)sc[r]) + 1u : 0u;
    }
    // --- 3a. each wavefront's own top kp, written in block order
    const uint64_t take = wave_choose<R>(key, kp);
    int wt;
    int pos = wave_excl_scan(__popcll(take), &wt);
    unsigned long long* cw = cand + w * kp;
#pragma unroll
    for (int r = 0; r < R; ++r)
      if ((take >> r) & 1ull) {
        cw[pos] = ((unsigned long long)key[r] << 32) | (uint32_t)(i0 + r);
        ++pos;
      }
    if (lane == 0) wave_cnt[w] = wt;
    __syncthreads();
    // --- 3b. wavefront 0: the global top kp among the candidates
    if (w == 0) {
      const int rc = (kSelWaves * kp + 63) / 64;
      if (rc <= 1) final_choose<1>(cand, wave_cnt, kp, bitmap);
      else if (rc <= 2) final_choose<2>(cand, wave_cnt, kp, bitmap);
      else if (rc <= 4) final_choose<4>(cand, wave_cnt, kp, bitmap);
      else if (rc <= 8) final_choose<8>(cand, wave_cnt, kp, bitmap);
      else if (rc <= 16) final_choose<16>(cand, wave_cnt, kp, bitmap);
      else if (rc <= 32) final_choose<32>(cand, wave_cnt, kp, bitmap);
      else final_choose<64>(cand, wave_cnt, kp, bitmap);
    }
  }
  for (int x = tid; x < m.n_sink; x += kSelThreads) atomicOr(&bitmap[x >> 5], 1u << (x & 31));
  for (int x = nb - m.n_local + tid; x < nb; x += kSelThreads)
    atomicOr(&bitmap[x >> 5], 1u << (x & 31));
  __syncthreads();
  // --- 4. ascending compaction: thread t owns bitmap word t
  const uint32_t word = tid < n_words ? bitmap[tid] : 0u;
  int tot;
  int opos = block_excl_scan(__popc(word), scan_lds, &tot);
  uint32_t wbits = word;
  while (wbits) {
    const int bit = __ffs(wbits) - 1;
    wbits &= wbits - 1;
    if (opos < k) {
      const int i = tid * 32 + bit;
      sel[opos] = i;
      if (so) so[opos] = i;
    }
    ++opos;
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
  const float* ev = (const float*)(base + ws.e_vals);
  const double* tp = (const double*)(base + ws.tile_part);
  int32_t* sel = (int32_t*)(base + ws.sel);
  int32_t* meta = (int32_t*)(base + ws.meta);
  const int per = (int)ceil_div(m.nb_cap, kSelThreads);
#define SPLA_R(r)                                                                              \
  hipLaunchKernelGGL(select_kernel<r>, dim3(m.bh), dim3(kSelThreads), 0, st, m, c.seq_lens, ev, \
                     tp, sel, sel_out, meta)
  if (per <= 1) SPLA_R(1);
  else if (per <= 2) SPLA_R(2);
  else if (per <= 4) SPLA_R(4);
  else if (per <= 8) SPLA_R(8);
  else if (per <= 16) SPLA_R(16);
  else SPLA_R(32);
#undef SPLA_R
  return hipGetLastError();
}

}  // namespace spla
