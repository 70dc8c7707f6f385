// Chunked causal prefill (Sec. 2: the decode formulation carries over to
// prefill and training). The T positions of a chunk are decoded together,
// each query exactly as a decode step at its own position would be: its own
// block selection, the statistics of the units it shares with the chunk
// taken over the tokens up to its position, and S_bar over its prefix. The
// work is split the way the paper's kernel design splits it (Sec. 3.3,
// "Kernel Design"): a linear-attention kernel for the global term and the
// fused sparse kernel for the exact branch and the selected-token linear
// term, here with the scoring and selection of every query in between:
//
//   prefill_unit_stats_kernel  running (mean, M2) of the units the chunk
//                              touches, after each of its positions
//   (append_blocks_kernel)     the chunk's K/V rows and unit statistics
//   prefill_linear_kernel      o_bar = phi(Q) S_bar(before the chunk) plus the
//                              causally masked phi(Q) phi(K)^T V inside the
//                              chunk, on matrix-core tiles; then S_bar and
//                              z_bar carried past the chunk
//   prefill_score_kernel       every query's block scores; each statistics
//                              tile is loaded once for the chunk's queries
//   prefill_select_kernel      every query's top-k
//   prefill_sparse_kernel      every query's fused exact + selected-linear
//                              pass over its own selection
//   prefill_merge_kernel       records + o_bar: residual, RMSNorm, output
//
// Query i of a chunk starting at L0 (the sequence length before it) sees
// L_i = L0 + min(i + 1, nv) tokens, nv being the chunk positions that fit
// below the capacity (a query past the capacity decodes over the full cache,
// as a decode step at capacity does).
#include "spla_kernels.h"
#include "spla_score.h"
#include "spla_select.h"
#include "spla_sparse.h"

namespace spla {

constexpr int kPrefQPW = 8;           // queries per scoring workgroup
constexpr int kPrefSelThreads = 1024;  // threads of a selection workgroup

__device__ __forceinline__ void chunk_bounds(const Dims& m, const int32_t* __restrict__ seq_lens,
                                             int b, int T, int* L0, int* nv) {
  const int l0 = min(max(seq_lens[b], 0), m.cap);
  *L0 = l0;
  *nv = min(m.cap - l0, T);
}

// first unit holding token L0 (u us + ul > L0)
__device__ __forceinline__ int first_touched_unit(const Dims& m, int L0) {
  return L0 >= m.ul ? (L0 - m.ul) / m.us + 1 : 0;
}

// ------------------------------------------------- running unit statistics
// Unit first + ur of (sequence, KV head) bh: its tokens before the chunk come
// in as the stored (mean, M2), then the chunk's tokens of the unit are added
// one at a time (Welford, fp64); after position i the running values are
// written to ustat[bh][ur][i] (fp32). Thread j: coordinate j.
template <typename T>
__global__ __launch_bounds__(128) void prefill_unit_stats_kernel(
    Dims m, int T_, const float* __restrict__ stats, const int32_t* __restrict__ seq_lens,
    const T* __restrict__ k_new, int nu_touch, float* __restrict__ ustat) {
  const int ur = blockIdx.x, bh = blockIdx.y;
  const int j = threadIdx.x;
  if (j >= m.d) return;
  int L0, nv;
  chunk_bounds(m, seq_lens, bh / m.hkv, T_, &L0, &nv);
  const int u = first_touched_unit(m, L0) + ur;
  const int64_t u0 = (int64_t)u * m.us, u1 = u0 + m.ul;
  const int na = (int)max((int64_t)0, min((int64_t)L0, u1) - u0);  // tokens before the chunk
  double n = (double)na, mean = 0.0, m2 = 0.0;
  if (na > 0) {
    mean = stats[stats_off4(m, bh, u, 0, j / 4) + (j & 3)];
    m2 = stats[stats_off4(m, bh, u, 1, j / 4) + (j & 3)];
  }
  float* out = ustat + ((int64_t)bh * nu_touch + ur) * T_ * 2 * m.d + j;
  float xs[kPrefillChunk];  // the chunk's values of coordinate j, all loads issued first
#pragma unroll
  for (int i = 0; i < kPrefillChunk; ++i)
    xs[i] = Elem<T>::load(k_new, ((int64_t)min(i, T_ - 1) * m.bh + bh) * m.d + j);
#pragma unroll
  for (int i = 0; i < kPrefillChunk; ++i) {
    if (i >= T_) break;
    const int64_t t = (int64_t)L0 + i;
    if (i < nv && t >= u0 && t < u1) {
      const double x = (double)xs[i];
      n += 1.0;
      const double delta = x - mean;
      mean += delta / n;
      m2 += delta * (x - mean);
    }
    out[(int64_t)i * 2 * m.d] = (float)mean;
    out[(int64_t)i * 2 * m.d + m.d] = (float)m2;
  }
}

// ------------------------------------------------------------- scoring
// One workgroup per (statistics tile, group of kPrefQPW queries, sequence x
// KV head): the tile is loaded once, then scored for each query with its own
// coefficient table and length (score_tile). Lanes whose unit the chunk
// touches take that query's running statistics instead of the stored ones.
// The next query's elements are loaded while the current one is scored.
template <int G, int D>
__global__ __launch_bounds__(256) void prefill_score_kernel(
    Dims m, int T_, const float* __restrict__ stats, const int32_t* __restrict__ seq_lens,
    const bf16_t* __restrict__ q, double s, int first_order, int nu_touch,
    const float* __restrict__ ustat, float* __restrict__ e_vals, double* __restrict__ tile_part) {
  constexpr int NJ = D / 16;
  __shared__ ScoreSmem<G> sm;
  const int tile = blockIdx.x, q0 = blockIdx.y * kPrefQPW, bh = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int bi = kScoreGroup * w + (lane & 15), qt = lane >> 4;
  const int t = bh * m.n_tiles + tile;
  const int64_t q_step = (int64_t)m.batch * m.hq * D;  // one position of q
  TileBuf<NJ> buf;
  load_tile<NJ>(m, stats, t, true, first_order, bi, qt, buf);
  QRegs<G, D> qr;
  load_q<G, bf16_t, D>(m, q + (int64_t)q0 * q_step, bh, qr);
  int L0, nv;
  chunk_bounds(m, seq_lens, bh / m.hkv, T_, &L0, &nv);
  const int ur = tile * kTileBlocks + bi - first_touched_unit(m, L0);
  const bool touched = ur >= 0 && ur < nu_touch;
  const int q1 = min(q0 + kPrefQPW, T_);
  for (int i = q0; i < q1; ++i) {
    if (touched) {
      const f32x4* pm = reinterpret_cast<const f32x4*>(
          ustat + (((int64_t)bh * nu_touch + ur) * T_ + i) * 2 * D) + qt * NJ;
      const f32x4* pv = first_order ? pm : pm + D / 4;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const f32x4 x = pm[j], y = pv[j];
        buf.mu[j] = make_float4(x[0], x[1], x[2], x[3]);
        buf.m2[j] = make_float4(y[0], y[1], y[2], y[3]);
      }
    }
    write_table<G, D>(qr, s, sm.sco);
    if (i + 1 < q1) load_q<G, bf16_t, D>(m, q + (int64_t)(i + 1) * q_step, bh, qr);
    __syncthreads();
    score_tile<G, D, false>(m, seq_lens, first_order, t, buf, sm.sco, sm.s_part[0], e_vals,
                            tile_part, L0 + min(i + 1, nv), bh * T_ + i);
  }
}

// ----------------------------------------------------------- selection
template <int R, bool WIN, int NT = kPrefSelThreads>
__global__ __launch_bounds__(NT) void prefill_select_kernel(
    Dims m, int T_, const int32_t* __restrict__ seq_lens, const float* __restrict__ e_vals,
    const double* __restrict__ tile_part, int32_t* __restrict__ sel_ws,
    int32_t* __restrict__ sel_out, int32_t* __restrict__ meta) {
  __shared__ SelectSmem<NT, kMaxTiles * SPLA_MAX_GROUP> sm;
  __shared__ float wsc[WIN ? kMaxWindows : 1];
  const int vh = blockIdx.x, bh = vh / T_, i = vh % T_;
  int L0, nv;
  chunk_bounds(m, seq_lens, bh / m.hkv, T_, &L0, &nv);
  select_blocks<NT, R, kMaxTiles * SPLA_MAX_GROUP, false, 0, WIN>(
      m, vh, L0 + min(i + 1, nv), e_vals, tile_part, sm, sel_ws + (int64_t)vh * m.k,
      meta + vh * 4, sel_out ? sel_out + ((int64_t)i * m.bh + bh) * m.k : nullptr, wsc);
}

// ------------------------------------------------------ fused sparse pass
// As the decode's pass, per query: its G heads' operands from its row of q,
// its selection, its length; no share of the global term.
// Workgroups are handed to the eight XCDs round-robin by index, each XCD
// with its own L2: the item of workgroup p is (p % 8) * (n / 8) + p / 8, so
// that consecutive items (the queries of one sequence x KV head, which
// largely select the same blocks) share an XCD and its L2. n_wg workgroups
// per query; the grid is n items rounded up to a multiple of 8. GC:
// accumulator columns per kind (>= G; 4 fits three workgroups per compute
// unit, 8 two).
template <int D, int BLK, int GC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(GC <= 4 ? 3 : 2)))
void prefill_sparse_kernel(
    Dims m, int T_, float s, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const bf16_t* __restrict__ q, const int32_t* __restrict__ sel,
    const int32_t* __restrict__ meta, int stride, float* __restrict__ part,
    const int32_t* __restrict__ table, int n_wg, int n_items) {
  __shared__ SparseSmem<D, GC> sm;
  const int per = (int)(gridDim.x / 8);
  const int item = ((int)blockIdx.x % 8) * per + (int)blockIdx.x / 8;
  if (item >= n_items) return;
  const int x = item % n_wg, vh = item / n_wg, bh = vh / T_, i = vh % T_;
  SparseRegs r;
  sparse_prologue<D, GC, false>(m, q + (int64_t)i * m.batch * m.hq * D, nullptr, nullptr, bh, x,
                                n_wg, r, sm);
  sparse_linear<D, GC, false>(m, nullptr, bh, r, sm);
  sparse_body_steps<D, BLK, false, GC, kPrefillStepsPerWave>(
      m, s, kc, vc, sel + (int64_t)vh * m.k, meta[vh * 4 + 2], bh, x, n_wg, r, sm, part, stride,
      table, vh);
}

// ---------------------------------------------------------------- merge
template <int D>
__global__ __launch_bounds__(512) void prefill_merge_kernel(
    Dims m, int T_, float eps, uint32_t flags, const float* __restrict__ gamma,
    const int32_t* __restrict__ meta, const float* __restrict__ part, int n_rec, int stride,
    const float* __restrict__ obar, const float* __restrict__ zq, bf16_t* __restrict__ out) {
  const int vh = blockIdx.x, bh = vh / T_, i = vh % T_;
  const int g = (int)(threadIdx.x >> 6);
  merge_head<bf16_t, D, false, true>(m, eps, flags, gamma, meta[vh * 4 + 1], meta[vh * 4 + 2],
                                     part + (int64_t)vh * n_rec * stride, n_rec, stride,
                                     out + (int64_t)i * m.batch * m.hq * D, bh, g,
                                     obar + (int64_t)vh * m.group * D, zq + (int64_t)vh * m.group);
}

// ------------------------------------------------ chunkwise linear attention
// One workgroup per (32 columns of S_bar, sequence x KV head), four
// wavefronts. With rows r = i G + g (position i, head g) of the chunk's
// queries, R = T G rows:
//   A = phi(Q) phi(K)^T, masked to key positions t <= i (and t < nv)
//   o_bar[r][c] = phi(Q)[r] . S_bar[:, c] + sum_t A[r][t] V[t][c]
//   zq[r] = phi(Q)[r] . z_bar + sum_t A[r][t]           (column block 0)
//   S_bar[:, c] += sum_t<nv phi(K)[t]^T V[t][c]; z_bar += sum_t phi(K)[t]
// All products run on v_mfma_f32_16x16x32_bf16 with fp32 accumulation; the
// fp32 operands phi(Q), phi(K), A and S_bar enter as bf16 hi + lo pairs
// (hi lo and lo hi cross terms included, about 16 mantissa bits), V exactly.
// MFMA operands of a 16 x 16 tile: lane l holds row (A) or column (B)
// l % 16 and k-elements 8 (l / 16) .. +7; the result holds column l % 16,
// rows 4 (l / 16) .. +3.
namespace pl {
constexpr int TP = kPrefillChunk;  // chunk positions (padded with zeros)
constexpr int CB = 32;             // columns of S_bar per workgroup
}  // namespace pl

template <int D>
struct alignas(16) LinearSmem {
  static constexpr int DP = D + 8;       // padded rows (bf16 elements)
  static constexpr int TPP = pl::TP + 8;
  uint16_t phk_h[pl::TP][DP], phk_l[pl::TP][DP];    // phi(K) rows
  uint16_t phkT_h[D][TPP], phkT_l[D][TPP];          // phi(K)^T
  float phk_f[pl::TP][D];                           // phi(K), fp32 (z_bar)
  uint16_t vT[pl::CB][TPP];                         // V^T of the column block
  uint16_t ST_h[pl::CB][DP], ST_l[pl::CB][DP];      // S_bar^T of the column block
  float Sf[D][pl::CB + 1];                          // S_bar of the column block
  uint16_t pq_h[4][16][DP], pq_l[4][16][DP];        // per wavefront: phi(Q) of its 16 rows
  uint16_t pa_h[4][16][TPP], pa_l[4][16][TPP];      // per wavefront: masked A of its rows
  float zb[D];
  float rsum[4][16];
};

__device__ __forceinline__ void split_bf16(float x, uint16_t& h, uint16_t& l) {
  const __bf16 hi = (__bf16)x;
  const __bf16 lo = (__bf16)(x - (float)hi);
  h = __builtin_bit_cast(uint16_t, hi);
  l = __builtin_bit_cast(uint16_t, lo);
}

__device__ __forceinline__ bf16x8 ld_op(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

__device__ __forceinline__ float row16_sum(float v) {
  v += __shfl_xor(v, 1, kWave);
  v += __shfl_xor(v, 2, kWave);
  v += __shfl_xor(v, 4, kWave);
  v += __shfl_xor(v, 8, kWave);
  return v;
}

// One row of D elements, lane holding elements lane + 64 e (row 0 when !ok,
// so that the load is issued either way).
// DE = D / 8 consecutive elements of a bf16 row (16-byte loads), as floats.
template <int DE>
__device__ __forceinline__ void load_part(const bf16_t* __restrict__ src, float (&x)[DE]) {
  static_assert(DE % 8 == 0, "whole 16-byte pieces");
#pragma unroll
  for (int u = 0; u < DE / 8; ++u) {
    const uint4 v = *reinterpret_cast<const uint4*>(src + 8 * u);
    const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e)
      x[8 * u + e] = bf16_to_f32((uint16_t)(e & 1 ? w4[e >> 1] >> 16 : w4[e >> 1] & 0xFFFFu));
  }
}

// phi of a row held by eight consecutive lanes (DE elements each): softmax
// over the row, the max and sum over the eight lanes by lane swaps; zero
// when !ok.
template <int DE>
__device__ __forceinline__ void phi_part(float (&x)[DE], bool ok) {
  float mx = -INFINITY;
#pragma unroll
  for (int e = 0; e < DE; ++e) {
    x[e] = ok ? x[e] : 0.f;
    mx = fmaxf(mx, x[e]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 4, 64));
  float sum = 0.f;
#pragma unroll
  for (int e = 0; e < DE; ++e) {
    x[e] = expf(x[e] - mx);
    sum += x[e];
  }
  sum += __shfl_xor(sum, 1, 64);
  sum += __shfl_xor(sum, 2, 64);
  sum += __shfl_xor(sum, 4, 64);
  const float inv = ok ? 1.0f / sum : 0.f;
#pragma unroll
  for (int e = 0; e < DE; ++e) x[e] *= inv;
}

template <int D>
__global__ __launch_bounds__(256) void prefill_linear_kernel(
    Dims m, int T_, const int32_t* __restrict__ seq_lens, const bf16_t* __restrict__ q,
    const bf16_t* __restrict__ k_new, const bf16_t* __restrict__ v_new, float* __restrict__ S,
    float* __restrict__ zbar, float* __restrict__ obar, float* __restrict__ zq) {
  using pl::CB;
  using pl::TP;
  constexpr int KS = D / 32;
  __shared__ LinearSmem<D> sm;
  const int cb = blockIdx.x, bh = blockIdx.y, b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group, R = T_ * G, c0 = cb * CB;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int li = lane & 15, lg = lane >> 4;
  int L0, nv;
  chunk_bounds(m, seq_lens, b, T_, &L0, &nv);

  // phi(K) of the chunk's keys (rows past nv, or past T, are zero):
  // wavefront w takes rows 8 w .. 8 w + 7 at once, eight lanes per row (lane
  // 8 r + u: coordinates u D / 8 ..)
  constexpr int DE = D / 8;
  static_assert(TP == 32, "four wavefronts of eight key rows");
  {
    const int i = 8 * w + (lane >> 3), ce = DE * (lane & 7);
    float kx[DE];
    load_part<DE>(k_new + ((int64_t)min(i, T_ - 1) * m.bh + bh) * D + ce, kx);
    phi_part<DE>(kx, i < nv);
#pragma unroll
    for (int e = 0; e < DE; ++e) {
      const int col = ce + e;
      uint16_t hh, ll;
      split_bf16(kx[e], hh, ll);
      sm.phk_h[i][col] = hh;
      sm.phk_l[i][col] = ll;
      sm.phkT_h[col][i] = hh;
      sm.phkT_l[col][i] = ll;
      sm.phk_f[i][col] = kx[e];
    }
  }
  for (int e = tid; e < TP * CB; e += 256) {
    const int i = e / CB, c = e % CB;
    sm.vT[c][i] = i < nv ? v_new[((int64_t)i * m.bh + bh) * D + c0 + c].bits : (uint16_t)0;
  }
  const float* Sb = S + (int64_t)bh * D * D;
  for (int e = tid; e < D * CB; e += 256) {
    const int jr = e / CB, c = e % CB;
    const float v = Sb[(int64_t)jr * D + c0 + c];
    sm.Sf[jr][c] = v;
    split_bf16(v, sm.ST_h[c][jr], sm.ST_l[c][jr]);
  }
  if (tid < D) sm.zb[tid] = zbar[(int64_t)bh * D + tid];
  __syncthreads();

  // the query rows, 16 per wavefront and round
  const int n_rt = (R + 15) / 16;
  for (int rt0 = 0; rt0 < n_rt; rt0 += 4) {
    const int rt = rt0 + w;
    const bool act = rt < n_rt;
    // the tile's 16 query rows, eight at a time with eight lanes per row
    // (both halves' loads issued first)
    float qx[2][DE];
    const int ce = DE * (lane & 7);
#pragma unroll
    for (int hp = 0; hp < 2; ++hp) {
      const int row = rt * 16 + 8 * hp + (lane >> 3);
      const bool ok = act && row < R;
      const int i = ok ? row / G : 0, g = ok ? row % G : 0;
      load_part<DE>(q + (((int64_t)i * m.batch + b) * m.hq + h * G + g) * D + ce, qx[hp]);
    }
#pragma unroll
    for (int hp = 0; hp < 2; ++hp) {
      const int rr = 8 * hp + (lane >> 3), row = rt * 16 + rr;
      phi_part<DE>(qx[hp], act && row < R);
#pragma unroll
      for (int e = 0; e < DE; ++e)
        split_bf16(qx[hp][e], sm.pq_h[w][rr][ce + e], sm.pq_l[w][rr][ce + e]);
    }
    __syncthreads();
    // A = phi(Q) phi(K)^T, masked, row sums
    float rs[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ct = 0; ct < TP / 16; ++ct) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 ah = ld_op(&sm.pq_h[w][li][32 * ks + 8 * lg]);
        const bf16x8 al = ld_op(&sm.pq_l[w][li][32 * ks + 8 * lg]);
        const bf16x8 bh8 = ld_op(&sm.phk_h[ct * 16 + li][32 * ks + 8 * lg]);
        const bf16x8 bl8 = ld_op(&sm.phk_l[ct * 16 + li][32 * ks + 8 * lg]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh8, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl8, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh8, acc, 0, 0, 0);
      }
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int row = rt * 16 + 4 * lg + r4;
        const int t = ct * 16 + li;
        const bool keep = act && row < R && t <= row / G && t < nv;
        const float a = keep ? acc[r4] : 0.f;
        split_bf16(a, sm.pa_h[w][4 * lg + r4][t], sm.pa_l[w][4 * lg + r4][t]);
        rs[r4] += a;
      }
    }
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const float v = row16_sum(rs[r4]);
      if (li == 0) sm.rsum[w][4 * lg + r4] = v;
    }
    __syncthreads();
    // o_bar tile: phi(Q) S_bar + A V
#pragma unroll
    for (int cc = 0; cc < CB / 16; ++cc) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 ah = ld_op(&sm.pq_h[w][li][32 * ks + 8 * lg]);
        const bf16x8 al = ld_op(&sm.pq_l[w][li][32 * ks + 8 * lg]);
        const bf16x8 bh8 = ld_op(&sm.ST_h[cc * 16 + li][32 * ks + 8 * lg]);
        const bf16x8 bl8 = ld_op(&sm.ST_l[cc * 16 + li][32 * ks + 8 * lg]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh8, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl8, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh8, acc, 0, 0, 0);
      }
#pragma unroll
      for (int kt = 0; kt < TP / 32; ++kt) {
        const bf16x8 ah = ld_op(&sm.pa_h[w][li][32 * kt + 8 * lg]);
        const bf16x8 al = ld_op(&sm.pa_l[w][li][32 * kt + 8 * lg]);
        const bf16x8 vb = ld_op(&sm.vT[cc * 16 + li][32 * kt + 8 * lg]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, vb, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, vb, acc, 0, 0, 0);
      }
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int row = rt * 16 + 4 * lg + r4;
        if (act && row < R) obar[((int64_t)bh * R + row) * D + c0 + cc * 16 + li] = acc[r4];
      }
    }
    if (cb == 0) {  // zq = phi(Q) . z_bar + the row sums of A, eight lanes per row
#pragma unroll
      for (int hp = 0; hp < 2; ++hp) {
        const int rr = 8 * hp + (lane >> 3);
        float p = 0.f;
#pragma unroll
        for (int e = 0; e < DE; ++e) {
          const int col = ce + e;
          const float ph = __builtin_bit_cast(float, (uint32_t)sm.pq_h[w][rr][col] << 16) +
                           __builtin_bit_cast(float, (uint32_t)sm.pq_l[w][rr][col] << 16);
          p = fmaf(ph, sm.zb[col], p);
        }
        p += __shfl_xor(p, 1, 64);
        p += __shfl_xor(p, 2, 64);
        p += __shfl_xor(p, 4, 64);
        const int row = rt * 16 + rr;
        if (act && row < R && (lane & 7) == 0) zq[(int64_t)bh * R + row] = p + sm.rsum[w][rr];
      }
    }
    __syncthreads();
  }

  // S_bar past the chunk: S[:, c] += phi(K)^T V[:, c] (tokens below nv)
  constexpr int NT = (D / 16) * (CB / 16);
  for (int tt = w; tt < NT; tt += 4) {
    const int rt = tt / (CB / 16), cc = tt % (CB / 16);
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < TP / 32; ++kt) {
      const bf16x8 ah = ld_op(&sm.phkT_h[rt * 16 + li][32 * kt + 8 * lg]);
      const bf16x8 al = ld_op(&sm.phkT_l[rt * 16 + li][32 * kt + 8 * lg]);
      const bf16x8 vb = ld_op(&sm.vT[cc * 16 + li][32 * kt + 8 * lg]);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, vb, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, vb, acc, 0, 0, 0);
    }
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int jr = rt * 16 + 4 * lg + r4, c = cc * 16 + li;
      S[((int64_t)bh * D + jr) * D + c0 + c] = sm.Sf[jr][c] + acc[r4];
    }
  }
  if (cb == 0 && tid < D) {
    float z = sm.zb[tid];
    for (int i = 0; i < nv; ++i) z += sm.phk_f[i][tid];
    zbar[(int64_t)bh * D + tid] = z;
  }
}

// ------------------------------------------------------------- launcher
template <int G, int D>
static void prefill_score_gd(const Dims& m, int T, const spla_cache& c, const void* q, double s,
                             int fo, const PrefillWs& ws, char* base, hipStream_t st) {
  hipLaunchKernelGGL((prefill_score_kernel<G, D>),
                     dim3((unsigned)m.n_tiles, (unsigned)ceil_div(T, kPrefQPW), (unsigned)m.bh),
                     dim3(256), 0, st, m, T, (const float*)c.blk_stats, (const int32_t*)c.seq_lens,
                     (const bf16_t*)q, s, fo, ws.nu_touch, (const float*)(base + ws.ustat),
                     (float*)(base + ws.e_vals), (double*)(base + ws.tile_part));
}

template <int D>
static void prefill_score_d(const Dims& m, int T, const spla_cache& c, const void* q, double s,
                            int fo, const PrefillWs& ws, char* base, hipStream_t st) {
  switch (m.group) {
#define SPLA_G(g) case g: prefill_score_gd<g, D>(m, T, c, q, s, fo, ws, base, st); break;
    SPLA_G(1) SPLA_G(2) SPLA_G(3) SPLA_G(4) SPLA_G(5) SPLA_G(6) SPLA_G(7) SPLA_G(8)
#undef SPLA_G
    default: break;
  }
}

template <int R, int NT = kPrefSelThreads>
static void prefill_select_r(const Dims& m, int T, const spla_cache& c, int32_t* sel_out,
                             const PrefillWs& ws, char* base, hipStream_t st) {
  const unsigned grid = (unsigned)((int64_t)m.bh * T);
  if constexpr (NT != kPrefSelThreads) {  // blocks only
    hipLaunchKernelGGL((prefill_select_kernel<R, false, NT>), dim3(grid), dim3(NT), 0, st, m, T,
                       (const int32_t*)c.seq_lens, (const float*)(base + ws.e_vals),
                       (const double*)(base + ws.tile_part), (int32_t*)(base + ws.sel), sel_out,
                       (int32_t*)(base + ws.meta));
  } else if (windowed(m))
    hipLaunchKernelGGL((prefill_select_kernel<R, true>), dim3(grid), dim3(kPrefSelThreads), 0, st,
                       m, T, (const int32_t*)c.seq_lens, (const float*)(base + ws.e_vals),
                       (const double*)(base + ws.tile_part), (int32_t*)(base + ws.sel), sel_out,
                       (int32_t*)(base + ws.meta));
  else
    hipLaunchKernelGGL((prefill_select_kernel<R, false>), dim3(grid), dim3(kPrefSelThreads), 0,
                       st, m, T, (const int32_t*)c.seq_lens, (const float*)(base + ws.e_vals),
                       (const double*)(base + ws.tile_part), (int32_t*)(base + ws.sel), sel_out,
                       (int32_t*)(base + ws.meta));
}

template <int D, int BLK>
static void prefill_sparse_db(const Dims& m, int T, float s, const spla_cache& c, const void* q,
                              const PrefillWs& ws, char* base, hipStream_t st) {
  const int64_t items = (int64_t)ws.n_wg * m.bh * T;
  auto kern = m.group <= 4 ? prefill_sparse_kernel<D, BLK, 4> : prefill_sparse_kernel<D, BLK, 8>;
  hipLaunchKernelGGL(kern, dim3((unsigned)align_up(items, 8)),
                     dim3(256), 0, st, m, T, s, (const bf16_t*)c.k_cache,
                     (const bf16_t*)c.v_cache, (const bf16_t*)q, (const int32_t*)(base + ws.sel),
                     (const int32_t*)(base + ws.meta), ws.part_stride, (float*)(base + ws.part),
                     m.pages > 0 ? c.block_table : nullptr, ws.n_wg, (int)items);
}

template <int D>
static void prefill_linear_d(const Dims& m, const spla_cache& c, int T, const void* k_new,
                             const void* v_new, const void* q, const PrefillWs& ws, char* base,
                             hipStream_t st) {
  hipLaunchKernelGGL((prefill_linear_kernel<D>), dim3(D / pl::CB, (unsigned)m.bh), dim3(256), 0,
                     st, m, T, (const int32_t*)c.seq_lens, (const bf16_t*)q,
                     (const bf16_t*)k_new, (const bf16_t*)v_new, c.lin_state, c.lin_norm,
                     (float*)(base + ws.obar), (float*)(base + ws.zq));
}

hipError_t launch_prefill_chunk(const Dims& m, const spla_config& cfg, const spla_cache& c,
                                int T, const void* k_new, const void* v_new, const void* q,
                                const float* gamma, void* out, int32_t* sel_out,
                                const PrefillWs& ws, char* base, const spla_events* ev,
                                hipStream_t st) {
  if (T < 1 || T > ws.T) return hipErrorInvalidValue;
  const double s_score =
      cfg.softmax_scale > 0.f ? (double)cfg.softmax_scale : 1.0 / sqrt((double)m.d);
  const float s = cfg.softmax_scale > 0.f ? cfg.softmax_scale : (float)(1.0 / sqrt((double)m.d));
  const int fo = (cfg.flags & SPLA_FLAG_FIRST_ORDER) ? 1 : 0;
  hipError_t e;
  // 1. running statistics of the touched units, from the statistics before the
  // chunk; then the chunk's K/V rows and the statistics of the units it touches
  mark_phase(ev, SPLA_PHASE_APPEND, false, st);
  hipLaunchKernelGGL(prefill_unit_stats_kernel<bf16_t>, dim3((unsigned)ws.nu_touch, (unsigned)m.bh),
                     dim3(128), 0, st, m, T, (const float*)c.blk_stats,
                     (const int32_t*)c.seq_lens, (const bf16_t*)k_new, ws.nu_touch,
                     (float*)(base + ws.ustat));
  if ((e = launch_append_blocks(m, c, k_new, v_new, T, nullptr, st, true)) != hipSuccess) return e;
  mark_phase(ev, SPLA_PHASE_APPEND, true, st);
  // 2. the global linear term of every query; S_bar and z_bar past the chunk
  mark_phase(ev, SPLA_PHASE_LINEAR, false, st);
  if (m.d == 64) prefill_linear_d<64>(m, c, T, k_new, v_new, q, ws, base, st);
  else prefill_linear_d<128>(m, c, T, k_new, v_new, q, ws, base, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark_phase(ev, SPLA_PHASE_LINEAR, true, st);
  // 3. block scores of every query
  mark_phase(ev, SPLA_PHASE_SCORE, false, st);
  if (m.d == 64) prefill_score_d<64>(m, T, c, q, s_score, fo, ws, base, st);
  else prefill_score_d<128>(m, T, c, q, s_score, fo, ws, base, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark_phase(ev, SPLA_PHASE_SCORE, true, st);
  // 4. selection of every query: without windows and up to 2048 blocks, 256
  // threads with up to eight blocks each (four wavefronts: cheaper barriers
  // and histogram scans; 32 positions at 128K 21.2 -> 17.5 us); otherwise
  // blocks per thread of a 1024-thread workgroup
  mark_phase(ev, SPLA_PHASE_SELECT, false, st);
  const int per = (int)ceil_div(m.nb_cap, kPrefSelThreads);
  if (!windowed(m) && m.nb_cap <= 256) prefill_select_r<1, 256>(m, T, c, sel_out, ws, base, st);
  else if (!windowed(m) && m.nb_cap <= 512) prefill_select_r<2, 256>(m, T, c, sel_out, ws, base, st);
  else if (!windowed(m) && m.nb_cap <= 1024) prefill_select_r<4, 256>(m, T, c, sel_out, ws, base, st);
  else if (!windowed(m) && m.nb_cap <= 2048) prefill_select_r<8, 256>(m, T, c, sel_out, ws, base, st);
  else if (per <= 1) prefill_select_r<1>(m, T, c, sel_out, ws, base, st);
  else if (per <= 2) prefill_select_r<2>(m, T, c, sel_out, ws, base, st);
  else if (per <= 4) prefill_select_r<4>(m, T, c, sel_out, ws, base, st);
  else if (per <= 8) prefill_select_r<8>(m, T, c, sel_out, ws, base, st);
  else if (per <= 16) prefill_select_r<16>(m, T, c, sel_out, ws, base, st);
  else prefill_select_r<32>(m, T, c, sel_out, ws, base, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark_phase(ev, SPLA_PHASE_SELECT, true, st);
  // 5. the fused sparse pass of every query
  mark_phase(ev, SPLA_PHASE_SPARSE, false, st);
  if (m.d == 64) {
    if (m.B == 32) prefill_sparse_db<64, 32>(m, T, s, c, q, ws, base, st);
    else if (m.B == 64) prefill_sparse_db<64, 64>(m, T, s, c, q, ws, base, st);
    else prefill_sparse_db<64, 128>(m, T, s, c, q, ws, base, st);
  } else {
    if (m.B == 32) prefill_sparse_db<128, 32>(m, T, s, c, q, ws, base, st);
    else if (m.B == 64) prefill_sparse_db<128, 64>(m, T, s, c, q, ws, base, st);
    else prefill_sparse_db<128, 128>(m, T, s, c, q, ws, base, st);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark_phase(ev, SPLA_PHASE_SPARSE, true, st);
  // 6. merge: records + o_bar, residual, RMSNorm, outputs
  mark_phase(ev, SPLA_PHASE_MERGE, false, st);
  const unsigned nq = (unsigned)((int64_t)m.bh * T);
  if (m.d == 64)
    hipLaunchKernelGGL((prefill_merge_kernel<64>), dim3(nq), dim3(64 * m.group), 0, st, m, T,
                       cfg.rms_eps, cfg.flags, gamma, (const int32_t*)(base + ws.meta),
                       (const float*)(base + ws.part), ws.n_wg, ws.part_stride,
                       (const float*)(base + ws.obar), (const float*)(base + ws.zq),
                       (bf16_t*)out);
  else
    hipLaunchKernelGGL((prefill_merge_kernel<128>), dim3(nq), dim3(64 * m.group), 0, st, m, T,
                       cfg.rms_eps, cfg.flags, gamma, (const int32_t*)(base + ws.meta),
                       (const float*)(base + ws.part), ws.n_wg, ws.part_stride,
                       (const float*)(base + ws.obar), (const float*)(base + ws.zq),
                       (bf16_t*)out);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark_phase(ev, SPLA_PHASE_MERGE, true, st);
  // 7. the sequences' lengths
  return launch_append_finish(m, c, T, nullptr, st);
}

}  // namespace spla
