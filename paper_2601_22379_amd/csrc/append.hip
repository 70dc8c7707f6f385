// Append path: key/value rows into the cache, block key statistics, and the
// global linear-attention state S_bar = sum_t phi(k_t)^T v_t, z_bar =
// sum_t phi(k_t) (Sec. 3.1 statistics, Sec. 3.2 Eq. 15, phi = softmax over
// the feature dimension).
#include "spla_device.h"
#include "spla_kernels.h"

namespace spla {

// Tokens of sequence b this append really adds (clamped to the capacity).
__device__ __forceinline__ int appended_count(const Dims& m, int L0, int max_new,
                                              const int32_t* __restrict__ n_new, int b,
                                              bool* clipped) {
  int n = n_new ? n_new[b] : max_new;
  n = n < 0 ? 0 : (n > max_new ? max_new : n);
  int room = m.cap - L0;
  room = room < 0 ? 0 : room;
  *clipped = n > room;
  return n < room ? n : room;
}

// One workgroup per touched statistics unit (a block, or a strided selection
// window: unit u holds tokens u us .. u us + ul - 1): merges the new tokens
// of the unit into its statistics and copies the rows t with
// u us <= t < (u + 1) us into the caches, so that each row is copied by
// exactly one unit. The new tokens' mean and M2 are computed two-pass in fp64
// and combined with the stored ones by Chan's formula, then rounded to fp32.
// (unit ux of the units touched, of (sequence, kv head) bh; thread j handles
// coordinate j). New row r of bh is element bh * s_bh + r * s_row of k_new
// and v_new: s_bh = max_new d, s_row = d for [batch][Hkv][max_new][d]
// (spla_append), s_bh = d, s_row = batch Hkv d for position-major rows
// [max_new][batch][Hkv][d] (the chunked prefill).
template <typename T>
__device__ __forceinline__ void append_unit(
    const Dims& m, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ stats,
    const int32_t* __restrict__ seq_lens, int32_t* __restrict__ err, const T* __restrict__ k_new,
    const T* __restrict__ v_new, int max_new, const int32_t* __restrict__ n_new,
    const int32_t* __restrict__ table, int ux, int bh, int64_t s_bh, int64_t s_row) {
  const int b = bh / m.hkv;
  const int L0 = seq_lens[b];
  bool clipped;
  const int ne = appended_count(m, L0, max_new, n_new, b, &clipped);
  if (clipped && err && ux == 0 && bh % m.hkv == 0 && threadIdx.x == 0)
    atomicOr(err, (int)SPLA_DEVERR_CAPACITY);
  // first unit holding token L0: u us + ul > L0
  const int first = L0 >= m.ul ? (L0 - m.ul) / m.us + 1 : 0;
  const int i = first + ux;
  const int t_lo = max(L0, i * m.us);
  const int t_hi = min(L0 + ne, i * m.us + m.ul);
  const int t_own = min(t_hi, (i + 1) * m.us);  // rows this unit copies: t_lo .. t_own - 1
  const int j = threadIdx.x;
  if (t_hi <= t_lo || j >= m.d) return;
  const int64_t src0 = (int64_t)bh * s_bh - (int64_t)L0 * s_row + j;  // row t at src0 + t s_row

  // the slot of the block that holds the rows this unit copies (they all lie
  // in one block: a unit's first us tokens, us dividing B); -1: a paged
  // table entry out of range, the rows are not written
  int64_t slot = -1;
  if (t_own > t_lo) {
    const int blk = t_lo / m.B;
    if (!table) {
      slot = (int64_t)bh * m.nb_cap + blk;
    } else {
      const int p = block_page(m, table, bh, blk);
      slot = p < 0 ? -1 : (int64_t)p * m.hkv + bh % m.hkv;
      if (p < 0 && err && j == 0) atomicOr(err, (int)SPLA_DEVERR_PAGE);
    }
  }
  double sum = 0.0;
  for (int t = t_lo; t < t_hi; ++t) {
    const T kv = k_new[src0 + (int64_t)t * s_row];
    if (t < t_own && slot >= 0) {
      kc[k_off_slot(m, slot, t % m.B, j)] = kv;
      vc[v_off_slot(m, slot, t % m.B, j)] = v_new[src0 + (int64_t)t * s_row];
    }
    sum += (double)Elem<T>::load(&kv, 0);
  }
  const int nc = t_hi - t_lo;
  const double mean_c = sum / nc;
  double m2_c = 0.0;
  for (int t = t_lo; t < t_hi; ++t) {
    const double x = (double)Elem<T>::load(k_new, src0 + (int64_t)t * s_row) - mean_c;
    m2_c += x * x;
  }
  const int na = t_lo - i * m.us;
  const int64_t o_mean = stats_off4(m, bh, i, 0, j / 4) + (j & 3);
  const int64_t o_m2 = stats_off4(m, bh, i, 1, j / 4) + (j & 3);
  double mean = mean_c, m2 = m2_c;
  if (na > 0) {
    const double mean_a = stats[o_mean], m2_a = stats[o_m2];
    const double n = (double)(na + nc);
    const double delta = mean_c - mean_a;
    mean = mean_a + delta * (nc / n);
    m2 = m2_a + m2_c + delta * delta * ((double)na * nc / n);
  }
  stats[o_mean] = (float)mean;
  stats[o_m2] = (float)m2;
}

template <typename T>
__global__ __launch_bounds__(128) void append_blocks_kernel(
    Dims m, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ stats,
    const int32_t* __restrict__ seq_lens, int32_t* __restrict__ err, const T* __restrict__ k_new,
    const T* __restrict__ v_new, int max_new, const int32_t* __restrict__ n_new,
    const int32_t* __restrict__ table, int64_t s_bh, int64_t s_row) {
  append_unit<T>(m, kc, vc, stats, seq_lens, err, k_new, v_new, max_new, n_new, table,
                 (int)blockIdx.x, (int)blockIdx.y, s_bh, s_row);
}

// Partial linear-attention state of one chunk of new tokens:
// P[j][c] = sum_t phi(k_t)_j v_t,c and Pz[j] = sum_t phi(k_t)_j, fp32.
template <typename T, int D>
__global__ __launch_bounds__(256) void append_state_partial_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const T* __restrict__ k_new,
    const T* __restrict__ v_new, int max_new, const int32_t* __restrict__ n_new, int n_chunks,
    int chunk_tokens, float* __restrict__ part_s, float* __restrict__ part_z) {
  constexpr int R = D / 16;
  __shared__ float sE[kSubTokens][D + 1];
  __shared__ float sV[kSubTokens][D + 1];
  const int bh = blockIdx.y;
  const int b = bh / m.hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  bool clipped;
  const int ne = appended_count(m, seq_lens[b], max_new, n_new, b, &clipped);
  const int t0 = blockIdx.x * chunk_tokens;
  const int t1 = min(t0 + chunk_tokens, ne);
  const int tr = tid / 16, tc = tid % 16;
  float acc[R][R];
  float zacc[R];
#pragma unroll
  for (int a = 0; a < R; ++a) {
    zacc[a] = 0.f;
#pragma unroll
    for (int c = 0; c < R; ++c) acc[a][c] = 0.f;
  }
  for (int tt = t0; tt < t1; tt += kSubTokens) {
    const int nt = min(kSubTokens, t1 - tt);
    for (int e = tid; e < kSubTokens * D; e += 256) {
      const int row = e / D, col = e % D;
      const int64_t src = ((int64_t)bh * max_new + tt + row) * D + col;
      sE[row][col] = row < nt ? Elem<T>::load(k_new, src) : 0.f;
      sV[row][col] = row < nt ? Elem<T>::load(v_new, src) : 0.f;
    }
    __syncthreads();
    // phi(k) = softmax over the feature dimension, one row per wave step
    for (int r = 0; r < kSubTokens / 4; ++r) {
      const int row = w * (kSubTokens / 4) + r;
      float x[D / 64];
      float mx = -INFINITY;
#pragma unroll
      for (int e = 0; e < D / 64; ++e) {
        x[e] = sE[row][lane + 64 * e];
        mx = fmaxf(mx, x[e]);
      }
      mx = wave_max(mx);
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < D / 64; ++e) {
        x[e] = expf(x[e] - mx);
        s += x[e];
      }
      s = wave_sum(s);
      const float inv = row < nt ? 1.0f / s : 0.f;
#pragma unroll
      for (int e = 0; e < D / 64; ++e) sE[row][lane + 64 * e] = x[e] * inv;
    }
    __syncthreads();
    for (int t = 0; t < nt; ++t) {
      float pv[R], vv[R];
#pragma unroll
      for (int a = 0; a < R; ++a) {
        pv[a] = sE[t][tr * R + a];
        vv[a] = sV[t][tc * R + a];
      }
#pragma unroll
      for (int a = 0; a < R; ++a) {
        zacc[a] += pv[a];
#pragma unroll
        for (int c = 0; c < R; ++c) acc[a][c] = fmaf(pv[a], vv[c], acc[a][c]);
      }
    }
    __syncthreads();
  }
  float* ps = part_s + ((int64_t)bh * n_chunks + blockIdx.x) * D * D;
#pragma unroll
  for (int a = 0; a < R; ++a)
#pragma unroll
    for (int c = 0; c < R; ++c) ps[(tr * R + a) * D + tc * R + c] = acc[a][c];
  if (tc == 0) {
    float* pz = part_z + ((int64_t)bh * n_chunks + blockIdx.x) * D;
#pragma unroll
    for (int a = 0; a < R; ++a) pz[tr * R + a] = zacc[a];
  }
}

// S_bar += sum of the chunk partials, accumulated in fp64 in chunk order.
__global__ __launch_bounds__(256) void append_state_reduce_kernel(
    Dims m, int n_chunks, const float* __restrict__ part_s, const float* __restrict__ part_z,
    float* __restrict__ S, float* __restrict__ z) {
  const int bh = blockIdx.y;
  const int D = m.d;
  const int row0 = blockIdx.x * 16;
  for (int e = threadIdx.x; e < 16 * D; e += 256) {
    const int row = row0 + e / D, col = e % D;
    const int64_t o = ((int64_t)bh * D + row) * D + col;
    double s = S[o];
    for (int c = 0; c < n_chunks; ++c) s += part_s[(((int64_t)bh * n_chunks + c) * D + row) * D + col];
    S[o] = (float)s;
  }
  if (threadIdx.x < 16) {
    const int row = row0 + threadIdx.x;
    double s = z[(int64_t)bh * D + row];
    for (int c = 0; c < n_chunks; ++c) s += part_z[((int64_t)bh * n_chunks + c) * D + row];
    z[(int64_t)bh * D + row] = (float)s;
  }
}

// Single-token state update: S_bar += phi(k)^T v, z_bar += phi(k) (fp32).
// Rows rx * 16 .. rx * 16 + 15 of S_bar += phi(k)^T v (and those entries of
// z_bar += phi(k)) for the single token k, v of (sequence, kv head) bh, by the
// 256 threads of a workgroup. A sequence at capacity gets nothing.
template <typename T, int D>
__device__ __forceinline__ void append_rank1_rows(const Dims& m,
                                                  const int32_t* __restrict__ seq_lens,
                                                  const T* __restrict__ k_new,
                                                  const T* __restrict__ v_new,
                                                  float* __restrict__ S, float* __restrict__ z,
                                                  int rx, int bh) {
  __shared__ float sphi[D];
  __shared__ float sv[D];
  constexpr int PT = 16 * D / 256;  // entries of the 16 rows per thread
  const int b = bh / m.hkv;
  if (seq_lens[b] >= m.cap) return;
  const int tid = threadIdx.x;
  const int row0 = rx * 16;
  // this thread's entries of the rows, loaded before phi(k) is formed so that
  // their latency overlaps it
  float sr[PT];
#pragma unroll
  for (int u = 0; u < PT; ++u) {
    const int e = tid + 256 * u;
    sr[u] = S[((int64_t)bh * D + row0 + e / D) * D + e % D];
  }
  if (tid < 64) {
    float x[D / 64];
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      x[e] = Elem<T>::load(k_new, (int64_t)bh * D + tid + 64 * e);
      mx = fmaxf(mx, x[e]);
    }
    mx = wave_max(mx);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      x[e] = expf(x[e] - mx);
      s += x[e];
    }
    s = wave_sum(s);
#pragma unroll
    for (int e = 0; e < D / 64; ++e) sphi[tid + 64 * e] = x[e] / s;
  }
  for (int c = tid; c < D; c += 256) sv[c] = Elem<T>::load(v_new, (int64_t)bh * D + c);
  __syncthreads();
#pragma unroll
  for (int u = 0; u < PT; ++u) {
    const int e = tid + 256 * u;
    const int row = row0 + e / D, col = e % D;
    S[((int64_t)bh * D + row) * D + col] = fmaf(sphi[row], sv[col], sr[u]);
  }
  if (tid < 16) z[(int64_t)bh * D + row0 + tid] += sphi[row0 + tid];
}

// The single-token append of a decode step in one launch: workgroups
// x < D / 16 update 16 rows of S_bar each (rank one), the others the
// statistics units the token falls in (and copy its K/V rows). The two parts
// touch disjoint memory and only read seq_lens, which append_finish_kernel
// advances afterwards.
template <typename T, int D>
__global__ __launch_bounds__(256) void append_one_kernel(
    Dims m, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ stats,
    const int32_t* __restrict__ seq_lens, int32_t* __restrict__ err, const T* __restrict__ k_new,
    const T* __restrict__ v_new, const int32_t* __restrict__ table, float* __restrict__ S,
    float* __restrict__ z) {
  const int bh = (int)blockIdx.y;
  if ((int)blockIdx.x < D / 16)
    append_rank1_rows<T, D>(m, seq_lens, k_new, v_new, S, z, (int)blockIdx.x, bh);
  else
    append_unit<T>(m, kc, vc, stats, seq_lens, err, k_new, v_new, 1, nullptr, table,
                   (int)blockIdx.x - D / 16, bh, D, D);
}

__global__ void append_finish_kernel(Dims m, int32_t* __restrict__ seq_lens, int max_new,
                                     const int32_t* __restrict__ n_new) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= m.batch) return;
  bool clipped;
  const int L0 = seq_lens[b];
  seq_lens[b] = L0 + appended_count(m, L0, max_new, n_new, b, &clipped);
}

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// ------------------------------------------------------------- launchers
hipError_t launch_append_blocks(const Dims& m, const spla_cache& c, const void* k_new,
                                const void* v_new, int max_new, const int32_t* n_new,
                                hipStream_t st, bool position_major) {
  // units touched by max_new tokens from any L0 (idle workgroups return)
  const int64_t nx = windowed(m) ? ceil_div(max_new + m.ul, m.us) + 2 : ceil_div(max_new, m.B) + 1;
  dim3 grid((unsigned)nx, (unsigned)m.bh);
  const int64_t s_bh = position_major ? m.d : (int64_t)max_new * m.d;
  const int64_t s_row = position_major ? (int64_t)m.bh * m.d : m.d;
  if (m.elem == 4)
    hipLaunchKernelGGL(append_blocks_kernel<float>, grid, dim3(128), 0, st, m, (float*)c.k_cache,
                       (float*)c.v_cache, c.blk_stats, c.seq_lens, c.err_flags,
                       (const float*)k_new, (const float*)v_new, max_new, n_new,
                       m.pages > 0 ? c.block_table : nullptr, s_bh, s_row);
  else
    hipLaunchKernelGGL(append_blocks_kernel<bf16_t>, grid, dim3(128), 0, st, m,
                       (bf16_t*)c.k_cache, (bf16_t*)c.v_cache, c.blk_stats, c.seq_lens,
                       c.err_flags, (const bf16_t*)k_new, (const bf16_t*)v_new, max_new, n_new,
                       m.pages > 0 ? c.block_table : nullptr, s_bh, s_row);
  return hipGetLastError();
}

template <typename T, int D>
static void state_partial(const Dims& m, const spla_cache& c, const void* k_new, const void* v_new,
                          int max_new, const int32_t* n_new, const AppendWs& ws, char* base,
                          hipStream_t st) {
  hipLaunchKernelGGL((append_state_partial_kernel<T, D>), dim3(ws.n_chunks, m.bh), dim3(256), 0,
                     st, m, c.seq_lens, (const T*)k_new, (const T*)v_new, max_new, n_new,
                     ws.n_chunks, ws.chunk_tokens, (float*)(base + ws.part_s),
                     (float*)(base + ws.part_z));
}

hipError_t launch_append_state(const Dims& m, const spla_cache& c, const void* k_new,
                               const void* v_new, int max_new, const int32_t* n_new,
                               const AppendWs& ws, char* base, hipStream_t st) {
  if (m.elem == 4) {
    if (m.d == 64) state_partial<float, 64>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
    else state_partial<float, 128>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
  } else {
    if (m.d == 64) state_partial<bf16_t, 64>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
    else state_partial<bf16_t, 128>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(append_state_reduce_kernel, dim3(m.d / 16, m.bh), dim3(256), 0, st, m,
                     ws.n_chunks, (const float*)(base + ws.part_s),
                     (const float*)(base + ws.part_z), c.lin_state, c.lin_norm);
  return hipGetLastError();
}

// Units a single token touches: one block, or up to ul / us windows.
static int64_t units_of_one(const Dims& m) { return windowed(m) ? m.ul / m.us : 1; }

template <typename T, int D>
static void append_one_td(const Dims& m, const spla_cache& c, const void* k_new,
                          const void* v_new, hipStream_t st) {
  hipLaunchKernelGGL((append_one_kernel<T, D>), dim3((unsigned)(D / 16 + units_of_one(m)),
                     (unsigned)m.bh), dim3(256), 0, st, m, (T*)c.k_cache, (T*)c.v_cache,
                     c.blk_stats, c.seq_lens, c.err_flags, (const T*)k_new, (const T*)v_new,
                     m.pages > 0 ? c.block_table : nullptr, c.lin_state, c.lin_norm);
}

hipError_t launch_append_one(const Dims& m, const spla_cache& c, const void* k_new,
                             const void* v_new, hipStream_t st) {
  if (m.elem == 4) {
    if (m.d == 64) append_one_td<float, 64>(m, c, k_new, v_new, st);
    else append_one_td<float, 128>(m, c, k_new, v_new, st);
  } else {
    if (m.d == 64) append_one_td<bf16_t, 64>(m, c, k_new, v_new, st);
    else append_one_td<bf16_t, 128>(m, c, k_new, v_new, st);
  }
  return hipGetLastError();
}

hipError_t launch_append_finish(const Dims& m, const spla_cache& c, int max_new,
                                const int32_t* n_new, hipStream_t st) {
  hipLaunchKernelGGL(append_finish_kernel, dim3((unsigned)ceil_div(m.batch, 256)), dim3(256), 0,
                     st, m, c.seq_lens, max_new, n_new);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st) {
  const int64_t n = (int64_t)(bytes / 4);
  if (n == 0) return hipSuccess;
  int64_t blocks = ceil_div(n, 256);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, (uint32_t*)p, n);
  return hipGetLastError();
}

}  // namespace spla
