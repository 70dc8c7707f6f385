// Fused pass over the selected blocks, and the merge (Secs. 2.2, 3.2, 3.3).
//
// Every selected block is read from HBM once. From that read the pass
// accumulates, for each of the G query heads of the KV head,
//   - the exact branch of Eq. (5): online max m, normaliser l and
//     acc = sum_t exp(s q.k_t - m) v_t over the selected tokens, and
//   - the selected-token linear term of Eq. (16):
//     accw = sum_t <phi(q), phi(k_t)> v_t and zw = sum_t <phi(q), phi(k_t)>,
//     phi being the softmax over the feature dimension.
// The global linear term o_bar = phi(q) S_bar and <phi(q), z_bar> (Eq. 15) is
// split over the same workgroups by rows of S_bar: workgroup x of a
// (sequence, KV head) owns rows x*RW .. x*RW + RW - 1 (RW = ceil(d / n_wg)),
// loads them at its start next to the key / value loads, and subtracts its
// selected-token terms from its share, so each record carries
// (m, l, zq_x - zw, acc, obar_x - accw). The merge kernel (one workgroup per
// sequence x KV head) combines the records: the sum of the last fields is
// the residual numerator o_bar - o_tilde of Eq. (14) (and its normaliser
// <phi(q), z_bar> - z_tilde); the residual is exactly 0 when every token is
// selected. It writes out = o_sparse + gamma * r / sqrt(mean(r^2) + eps)
// (Sec. 3.3).
//
// bf16 with G <= 8 runs on the matrix cores (v_mfma_f32_16x16x32_bf16, one
// 32-token step per wavefront); fp32 and larger groups use a VALU pass that
// writes the same records.
#include "spla_device.h"
#include "spla_kernels.h"
#include "spla_select.h"

namespace spla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------- merge
// Combines the n_rec records of a (sequence, KV head) and writes the output
// rows of the group's G heads: one wavefront per head, lane l owning the E
// adjacent coordinates E l .. E l + E - 1. The record headers of a batch of
// 64 records are read one record per lane; every load of a batch (and the
// gain row) is issued before any arithmetic.
template <int E>
__device__ __forceinline__ void load_vec(const float* p, float (&v)[E]) {
  if constexpr (E == 2) {
    const float2 x = *reinterpret_cast<const float2*>(p);
    v[0] = x.x;
    v[1] = x.y;
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = p[e];
  }
}

template <typename T, int D>
__global__ __launch_bounds__(1024) void merge_kernel(
    Dims m, float eps, uint32_t flags, const float* __restrict__ gamma,
    const int32_t* __restrict__ meta, const float* __restrict__ part, int n_rec, int stride,
    T* __restrict__ out) {
  constexpr int E = D / 64;  // coordinates per lane
  constexpr int NB = 16;     // record bodies per load batch
  const int bh = blockIdx.x;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group;
  const int g = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c0 = E * lane;
  const float* rec = part + (int64_t)bh * n_rec * stride;
  const int64_t orow = ((int64_t)b * m.hq + h * G + g) * D + c0;
  const bool rla = !(flags & SPLA_FLAG_NO_RLA);
  float gm[E];
  load_vec<E>(gamma + (int64_t)(h * G + g) * D + c0, gm);
  const int all_sel = meta[bh * 4 + 1];
  const int L = meta[bh * 4 + 2];
  float M = -INFINITY, l = 0.f, zt = 0.f;
  float osp[E], ot[E];
#pragma unroll
  for (int e = 0; e < E; ++e) osp[e] = ot[e] = 0.f;
  for (int x0 = 0; x0 < n_rec; x0 += 64) {
    // headers: lane u holds record x0 + u
    const bool hv = x0 + lane < n_rec;
    const float* hr = rec + (int64_t)(hv ? x0 + lane : 0) * stride;
    const float hm = hv ? hr[g] : -INFINITY;
    const float hl = hv ? hr[16 + g] : 0.f;
    const float hz = hv ? hr[32 + g] : 0.f;
    const int nb_here = n_rec - x0 < 64 ? n_rec - x0 : 64;
    // bodies, NB at a time (the first batch is issued with the headers)
    for (int u0 = 0; u0 < nb_here; u0 += NB) {
      float a[NB][E], aw[NB][E];
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int x = x0 + u0 + u < n_rec ? x0 + u0 + u : 0;
        load_vec<E>(rec + (int64_t)x * stride + kPartHead + g * D + c0, a[u]);
        load_vec<E>(rec + (int64_t)x * stride + kPartHead + (G + g) * D + c0, aw[u]);
      }
      if (u0 == 0) {  // fold this batch of headers into the running max
        const float bm = fmaxf(M, wave_max(hm));
        const float alpha = M == -INFINITY ? 0.f : __expf(M - bm);
        l *= alpha;
#pragma unroll
        for (int e = 0; e < E; ++e) osp[e] *= alpha;
        M = bm;
        l += wave_sum(hm == -INFINITY ? 0.f : hl * __expf(hm - M));
        zt += wave_sum(hz);
      }
      const float sc_l = hm == -INFINITY ? 0.f : __expf(hm - M);  // lane u: record x0 + u
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const bool ok = u0 + u < nb_here;
        const float sc = ok ? __shfl(sc_l, u0 + u, 64) : 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          osp[e] = fmaf(a[u][e], sc, osp[e]);
          ot[e] += ok ? aw[u][e] : 0.f;
        }
      }
    }
  }
  float o[E];
  if (L == 0) {
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = 0.f;
  } else {
    // residual r = o_bar - o_tilde (over its normaliser with RLA_NORMALIZE),
    // exactly 0 when every token was selected; out = o_sparse + gamma r / rms(r)
    const float den = (flags & SPLA_FLAG_RLA_NORMALIZE) ? zt : 1.f;
    float rr[E];
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      osp[e] /= l;
      rr[e] = (rla && !all_sel) ? ot[e] / den : 0.f;
      ss += rr[e] * rr[e];
    }
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / D + eps);
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = rla ? fmaf(gm[e] * rr[e], inv, osp[e]) : osp[e];
  }
#pragma unroll
  for (int e = 0; e < E; ++e) Elem<T>::store(out, orow + e, o[e]);
}

// ------------------------------------------------ global linear term
// Rows of S_bar owned by workgroup x of n_wg: row0 .. row0 + nrows - 1.
__device__ __forceinline__ void lin_rows(int D, int x, int n_wg, int* row0, int* nrows) {
  const int rw = (D + n_wg - 1) / n_wg;
  const int r0 = x * rw;
  *row0 = r0;
  *nrows = r0 >= D ? 0 : (D - r0 < rw ? D - r0 : rw);
}

// ------------------------------------------------------------ VALU pass
template <typename T, int D>
__global__ __launch_bounds__(256) void sparse_valu_kernel(
    Dims m, float s, float eps, uint32_t flags, const T* __restrict__ kc,
    const T* __restrict__ vc, const T* __restrict__ q, const float* __restrict__ gamma,
    const float* __restrict__ S, const float* __restrict__ zbar,
    const int32_t* __restrict__ sel, const int32_t* __restrict__ meta, int bps, int stride,
    float* __restrict__ part) {
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
  const int nb = (L + m.B - 1) / m.B;
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
    int blk = sel[(int64_t)bh * m.k + p];
    blk = blk < 0 ? 0 : (blk >= nb ? nb - 1 : blk);
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
  // this workgroup's rows of the global linear term, minus its selected terms
  int row0, nrows;
  lin_rows(D, split, gridDim.x, &row0, &nrows);
  const float* Sb = S + (int64_t)bh * D * D;
  float* rec = part + ((int64_t)bh * gridDim.x + split) * stride;
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int idx = tid + 256 * r;
    if (idx < G * D) {
      const int mm = idx / D, c = idx % D;
      float ob = 0.f;
      for (int j = row0; j < row0 + nrows; ++j) ob = fmaf(sphq[mm][j], Sb[j * D + c], ob);
      rec[kPartHead + mm * D + c] = acc[r];
      rec[kPartHead + (G + mm) * D + c] = ob - accw[r];
    }
  }
  if (tid < G) {
    float zq = 0.f;
    for (int j = row0; j < row0 + nrows; ++j) zq = fmaf(sphq[tid][j], zbar[(int64_t)bh * D + j], zq);
    rec[tid] = s_m[tid];
    rec[16 + tid] = s_l[tid];
    rec[32 + tid] = zq - s_zw[tid];
  }
}

// ------------------------------------------------------------ MFMA pass
// One 32-token step of one selected block per wavefront (the workgroup's
// four wavefronts take consecutive steps). With g = lane / 16 and
// j = lane % 16 (the MFMA column), for the two 16-row tiles of a step the key
// row loaded by lane l is token 8 (i / 4) + 4 tile + (i % 4), i = l % 16, so
// that after S = K [Q | phi(Q)]^T the accumulator rows held by lane l are
// exactly the tokens 8 g .. 8 g + 7 of the step, in order - the layout the
// second product needs for its B operand. Columns 0..7 carry the exact-branch
// logits of heads 0..G-1, columns 8..15 the linear weights
// <phi(q), phi(k)> of the same heads; one accumulator holds both. phi(k) and
// the probabilities enter the products as bf16 hi + lo pairs (about 16
// mantissa bits); accumulation is fp32.
//
// R > 0: the workgroup first selects the blocks of its (sequence, KV head)
// itself (select_blocks with 256 threads, R blocks per thread; every
// workgroup of the pair computes the same selection), so no selection kernel
// runs; workgroup 0 publishes the selection and the meta words. R = 0: the
// selection comes from the selection kernel.
template <int D, int BLK, int R>
__global__ __launch_bounds__(256) void sparse_mfma_kernel(
    Dims m, float s, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const uint4* __restrict__ qprep, const float* __restrict__ S, const float* __restrict__ zbar,
    const int32_t* __restrict__ sel, int32_t* __restrict__ meta, int stride,
    float* __restrict__ part, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ e_vals, const double* __restrict__ tile_part,
    int32_t* __restrict__ sel_out) {
  constexpr int KS = D / 32;   // k-steps of the first product
  constexpr int MT = D / 16;   // coordinate tiles of the second product
  constexpr int CPB = BLK / 32;  // steps per block
  constexpr int SPRE = 8;        // S_bar entries per thread loaded up front
  constexpr int SWN = R > 0 ? kTileBlocks * 8 : 4;  // tile weights: <= 64 tiles x 8 heads
  __shared__ SelectSmem<256, SWN> ssm;
  __shared__ int32_t s_sel[R > 0 ? SPLA_MAX_TOP_K : 1];
  __shared__ int32_t s_meta[4];
  __shared__ float s_o[kSparseWaves][D][17];
  __shared__ float s_m[kSparseWaves][16], s_l[kSparseWaves][16];
  __shared__ float s_phq[8][D];          // phi(q) of the group's heads
  __shared__ float s_S[SPRE * 256];      // this workgroup's rows of S_bar
  __shared__ float s_zb[D];
  const int bh = blockIdx.y;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int j = lane & 15, g = lane >> 4, i = lane & 15;
  const int item = blockIdx.x * kSparseWaves + w;
  const int p = item / CPB, ch = item % CPB;
  const bool exact_col = j < 8;
  const int head = exact_col ? j : j - 8;
  const bool live = head < G;
  // B operands, laid out per lane by the scoring pass: [q | 0] for the
  // logits, [0 | phi(q)_hi] and [0 | phi(q)_lo] for the linear weights
  bf16x8 qb[KS], pqh[KS], pql[KS];
  {
    const uint4* qp = qprep + (int64_t)bh * 3 * KS * 64 + lane;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qb[ks] = __builtin_bit_cast(bf16x8, qp[(0 * KS + ks) * 64]);
      pqh[ks] = __builtin_bit_cast(bf16x8, qp[(1 * KS + ks) * 64]);
      pql[ks] = __builtin_bit_cast(bf16x8, qp[(2 * KS + ks) * 64]);
    }
  }
  // this workgroup's rows of S_bar and z_bar (read here, used in the epilogue)
  int row0, nrows;
  lin_rows(D, blockIdx.x, gridDim.x, &row0, &nrows);
  const bool s_pre = nrows * D <= SPRE * 256;
  float spre[SPRE];
  {
    const float* Sb = S + ((int64_t)bh * D + row0) * D;
#pragma unroll
    for (int u = 0; u < SPRE; ++u) {
      const int e = tid + 256 * u;
      spre[u] = (s_pre && e < nrows * D) ? Sb[e] : 0.f;
    }
  }
  const float zbv = tid < nrows ? zbar[(int64_t)bh * D + row0 + tid] : 0.f;
  // this wavefront's block id (entries past the selection are -1) and the
  // sequence length
  int blk_sel, L;
  if constexpr (R > 0) {
    select_blocks<256, R, SWN>(m, bh, seq_lens, e_vals, tile_part, ssm, s_sel, s_meta,
                               blockIdx.x == 0 && sel_out ? sel_out + (int64_t)bh * m.k : nullptr);
    __syncthreads();
    if (blockIdx.x == 0 && tid < 4) meta[bh * 4 + tid] = s_meta[tid];
    blk_sel = p < m.k ? s_sel[p] : -1;
    L = s_meta[2];
  } else {
    blk_sel = p < m.k ? sel[(int64_t)bh * m.k + p] : -1;
    L = meta[bh * 4 + 2];
  }
  const int nb = (L + BLK - 1) / BLK;
  int n_valid = 0;  // tokens of this step that exist
  bf16x8 ka[2][KS];
  bf16x8 va[MT];
  if (blk_sel >= 0) {
    const int blk = blk_sel >= nb ? nb - 1 : blk_sel;
    n_valid = min(32, block_count(L, BLK, blk) - ch * 32);
    if (n_valid > 0) {
      const bf16_t* kblk = kc + ((int64_t)bh * m.cap + (int64_t)blk * BLK + ch * 32) * D;
      const bf16_t* vblk = vc + ((int64_t)bh * m.nb_cap + blk) * D * BLK + ch * 32;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const int row = 8 * (i >> 2) + 4 * mt + (i & 3);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          ka[mt][ks] = *reinterpret_cast<const bf16x8*>(kblk + (int64_t)row * D + 32 * ks + 8 * g);
      }
#pragma unroll
      for (int t = 0; t < MT; ++t)
        va[t] = *reinterpret_cast<const bf16x8*>(vblk + (int64_t)(16 * t + i) * BLK + 8 * g);
    }
  }
  floatx4 acc_o[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc_o[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;  // exact columns: max / sum; linear columns: sum
  // wavefront 0 leaves phi(q) (hi + lo) in LDS for the global linear term
  if (w == 0 && !exact_col && live) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        s_phq[head][32 * ks + 8 * g + e] = (float)pqh[ks][e] + (float)pql[ks][e];
  }
  if (n_valid > 0) {
    floatx4 sw[2];
    float zinv[2];  // 1 / sum exp(k - max k) of this lane's key row, per tile
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      sw[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[mt][ks], qb[ks], sw[mt], 0, 0, 0);
      // exp(k - max k) of this lane's key row (row i of the tile), spread over
      // lanes i + 16 g'; the 1 / sum of phi(k) is applied to the result rows
      float kx[KS][8];
      float mx = -INFINITY;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          kx[ks][e] = (float)ka[mt][ks][e];
          mx = fmaxf(mx, kx[ks][e]);
        }
      mx = fmaxf(mx, xor16(mx));
      mx = fmaxf(mx, xor32(mx));
      const float mxl = mx * kLog2e;
      float sum = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          kx[ks][e] = __builtin_amdgcn_exp2f(fmaf(kx[ks][e], kLog2e, -mxl));
          sum += kx[ks][e];
        }
      sum += xor16(sum);
      sum += xor32(sum);
      zinv[mt] = 1.0f / sum;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        bf16x8 fh, fl;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float f = kx[ks][e];
          const __bf16 hi = (__bf16)f;
          fh[e] = hi;
          fl[e] = (__bf16)(f - (float)hi);
        }
        sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh, pqh[ks], sw[mt], 0, 0, 0);
        sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh, pql[ks], sw[mt], 0, 0, 0);
        sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fl, pqh[ks], sw[mt], 0, 0, 0);
      }
    }
    // tokens 8g .. 8g+7 of this step: tile 0 rows 4g..4g+3, tile 1 rows 4g..4g+3
    // (result row 4g + r of tile t is token 8g + 4t + r; its 1 / Z sits in
    // lane 4g + r)
    float val[8];
    float cmax = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool ok = 8 * g + e < n_valid;
      const float zi = __shfl(zinv[e >> 2], 4 * g + (e & 3), kWave);
      const float x = sw[e >> 2][e & 3];
      val[e] = exact_col ? (ok ? x * s : -INFINITY) : (ok ? x * zi : 0.f);
      cmax = fmaxf(cmax, val[e]);
    }
    cmax = fmaxf(cmax, xor16(cmax));
    cmax = fmaxf(cmax, xor32(cmax));
    float psum = 0.f;
    bf16x8 bh8, bl8;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pv = exact_col ? __builtin_amdgcn_exp2f((val[e] - cmax) * kLog2e) : val[e];
      psum += pv;
      const __bf16 hi = (__bf16)pv;
      bh8[e] = hi;
      bl8[e] = (__bf16)(pv - (float)hi);
    }
    psum += xor16(psum);
    psum += xor32(psum);
    m_run = exact_col ? cmax : -INFINITY;
    l_run = psum;
    if (n_valid < 32) {  // rows past the sequence end may hold anything: zero them
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (8 * g + e >= n_valid) va[t][e] = (__bf16)0.f;
    }
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[t], bh8, acc_o[t], 0, 0, 0);
      acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[t], bl8, acc_o[t], 0, 0, 0);
    }
  }
  // ---- merge the four wavefronts of the workgroup into one record
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) s_o[w][16 * t + 4 * g + r][j] = acc_o[t][r];
  if (lane < 16) {
    s_m[w][lane] = m_run;
    s_l[w][lane] = l_run;
  }
#pragma unroll
  for (int u = 0; u < SPRE; ++u) s_S[tid + 256 * u] = spre[u];
  if (tid < D) s_zb[tid] = zbv;
  __syncthreads();
  float* rec = part + ((int64_t)bh * gridDim.x + blockIdx.x) * stride;
  for (int e = tid; e < G * D; e += 256) {
    const int hh = e / D, c = e % D;
    float M = -INFINITY;
#pragma unroll
    for (int x = 0; x < kSparseWaves; ++x) M = fmaxf(M, s_m[x][hh]);
    float a = 0.f, aw = 0.f;
#pragma unroll
    for (int x = 0; x < kSparseWaves; ++x) {
      const float sc = s_m[x][hh] == -INFINITY ? 0.f : __expf(s_m[x][hh] - M);
      a = fmaf(s_o[x][c][hh], sc, a);
      aw += s_o[x][c][8 + hh];
    }
    float ob = 0.f;  // this workgroup's rows of phi(q) S_bar
    if (s_pre) {
      for (int r = 0; r < nrows; ++r) ob = fmaf(s_phq[hh][row0 + r], s_S[r * D + c], ob);
    } else {
      const float* Sb = S + (int64_t)bh * D * D;
      for (int r = row0; r < row0 + nrows; ++r) ob = fmaf(s_phq[hh][r], Sb[r * D + c], ob);
    }
    rec[kPartHead + hh * D + c] = a;
    rec[kPartHead + (G + hh) * D + c] = ob - aw;
  }
  if (tid < G) {
    float M = -INFINITY;
#pragma unroll
    for (int x = 0; x < kSparseWaves; ++x) M = fmaxf(M, s_m[x][tid]);
    float l = 0.f, zw = 0.f;
#pragma unroll
    for (int x = 0; x < kSparseWaves; ++x) {
      l += s_m[x][tid] == -INFINITY ? 0.f : s_l[x][tid] * __expf(s_m[x][tid] - M);
      zw += s_l[x][8 + tid];
    }
    float zq = 0.f;
    for (int r = 0; r < nrows; ++r) zq = fmaf(s_phq[tid][row0 + r], s_zb[r], zq);
    rec[tid] = M;
    rec[16 + tid] = l;
    rec[32 + tid] = zq - zw;
  }
}

// ------------------------------------------------------------- launchers
template <typename T, int D>
static void valu_td(const Dims& m, const spla_config& cfg, float s, const spla_cache& c,
                    const void* q, const float* gamma, void* out, const DecodeWs& ws, char* base,
                    hipStream_t st) {
  hipLaunchKernelGGL((sparse_valu_kernel<T, D>), dim3(ws.n_wg, m.bh), dim3(256), 0, st, m, s,
                     cfg.rms_eps, cfg.flags, (const T*)c.k_cache, (const T*)c.v_cache,
                     (const T*)q, gamma, (const float*)c.lin_state, (const float*)c.lin_norm,
                     (const int32_t*)(base + ws.sel), (const int32_t*)(base + ws.meta),
                     ws.blocks_per_wg, ws.part_stride, (float*)(base + ws.part));
}

// Blocks per thread of the in-workgroup selection (0: use the selection
// kernel). Every workgroup repeats the selection of its (sequence, KV head),
// which pays only while the grid is small (about two workgroups per compute
// unit) and the block count is at most 4096.
static int sparse_select_r(const Dims& m) {
  if (!use_mfma_sparse(m) || m.nb_cap > 256 * 16) return 0;
  const DecodeWs ws = decode_ws_layout(m);
  if ((int64_t)ws.n_wg * m.bh > 2 * (int64_t)compute_units()) return 0;
  const int per = (int)ceil_div(m.nb_cap, 256);
  return per <= 2 ? 2 : (per <= 4 ? 4 : (per <= 8 ? 8 : 16));
}

bool sparse_selects(const Dims& m) { return sparse_select_r(m) > 0; }

template <int D, int BLK, int R>
static void mfma_dbr(const Dims& m, float s, const spla_cache& c, int32_t* sel_out,
                     const DecodeWs& ws, char* base, hipStream_t st) {
  hipLaunchKernelGGL((sparse_mfma_kernel<D, BLK, R>), dim3(ws.n_wg, m.bh), dim3(256), 0, st, m, s,
                     (const bf16_t*)c.k_cache, (const bf16_t*)c.v_cache,
                     (const uint4*)(base + ws.qprep), (const float*)c.lin_state,
                     (const float*)c.lin_norm, (const int32_t*)(base + ws.sel),
                     (int32_t*)(base + ws.meta), ws.part_stride, (float*)(base + ws.part),
                     c.seq_lens, (const float*)(base + ws.e_vals),
                     (const double*)(base + ws.tile_part), sel_out);
}

template <int D, int BLK>
static void mfma_db(const Dims& m, float s, const spla_cache& c, int32_t* sel_out,
                    const DecodeWs& ws, char* base, hipStream_t st) {
  switch (sparse_select_r(m)) {
    case 2: mfma_dbr<D, BLK, 2>(m, s, c, sel_out, ws, base, st); break;
    case 4: mfma_dbr<D, BLK, 4>(m, s, c, sel_out, ws, base, st); break;
    case 8: mfma_dbr<D, BLK, 8>(m, s, c, sel_out, ws, base, st); break;
    case 16: mfma_dbr<D, BLK, 16>(m, s, c, sel_out, ws, base, st); break;
    default: mfma_dbr<D, BLK, 0>(m, s, c, sel_out, ws, base, st); break;
  }
}

template <int D>
static void mfma_d(const Dims& m, float s, const spla_cache& c, int32_t* sel_out,
                   const DecodeWs& ws, char* base, hipStream_t st) {
  if (m.B == 32) mfma_db<D, 32>(m, s, c, sel_out, ws, base, st);
  else if (m.B == 64) mfma_db<D, 64>(m, s, c, sel_out, ws, base, st);
  else mfma_db<D, 128>(m, s, c, sel_out, ws, base, st);
}

template <typename T, int D>
static void merge_td(const Dims& m, const spla_config& cfg, const float* gamma, void* out,
                     const DecodeWs& ws, char* base, hipStream_t st) {
  hipLaunchKernelGGL((merge_kernel<T, D>), dim3(m.bh), dim3(64 * m.group), 0, st, m, cfg.rms_eps,
                     cfg.flags, gamma, (const int32_t*)(base + ws.meta),
                     (const float*)(base + ws.part), ws.n_wg, ws.part_stride, (T*)out);
}

hipError_t launch_sparse(const Dims& m, const spla_config& cfg, const spla_cache& c,
                         const void* q, const float* gamma, void* out, int32_t* sel_out,
                         const DecodeWs& ws, char* base, hipStream_t st) {
  const float s = cfg.softmax_scale > 0.f ? cfg.softmax_scale : (float)(1.0 / sqrt((double)m.d));
  if (use_mfma_sparse(m)) {
    if (m.d == 64) mfma_d<64>(m, s, c, sel_out, ws, base, st);
    else mfma_d<128>(m, s, c, sel_out, ws, base, st);
  } else if (m.elem == 4) {
    if (m.d == 64) valu_td<float, 64>(m, cfg, s, c, q, gamma, out, ws, base, st);
    else valu_td<float, 128>(m, cfg, s, c, q, gamma, out, ws, base, st);
  } else {
    if (m.d == 64) valu_td<bf16_t, 64>(m, cfg, s, c, q, gamma, out, ws, base, st);
    else valu_td<bf16_t, 128>(m, cfg, s, c, q, gamma, out, ws, base, st);
  }
  return hipGetLastError();
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
