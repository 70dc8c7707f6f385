// The fused pass over the selected blocks and the merge (Secs. 2.2, 3.2,
// 3.3), as device functions shared by the separate sparse / merge kernels and
// the single-launch decode kernel.
//
// Every selected block is read from HBM once. From that read the pass
// accumulates, for each of the G query heads of the KV head,
//   - the exact branch of Eq. (5): online max m, normaliser l and
//     acc = sum_t exp(s q.k_t - m) v_t over the selected tokens, and
//   - the selected-token linear term of Eq. (16):
//     accw = sum_t <phi(q), phi(k_t)> v_t and zw = sum_t <phi(q), phi(k_t)>,
//     phi being the softmax over the feature dimension.
// The global linear term o_bar = phi(q) S_bar and <phi(q), z_bar> (Eq. 15) is
// split over the same workgroups by rows of S_bar: workgroup x of the n_wg of
// a (sequence, KV head) owns rows x*RW .. x*RW + RW - 1 (RW = ceil(d / n_wg)),
// loads them at its start next to the key / value loads, and subtracts its
// selected-token terms from its share, so each record carries
// (m, l, zq_x - zw, acc, obar_x - accw). The merge combines the records: the
// sum of the last fields is the residual numerator o_bar - o_tilde of
// Eq. (14) (and its normaliser <phi(q), z_bar> - z_tilde); the residual is
// exactly 0 when every token is selected. It writes
// out = o_sparse + gamma * r / sqrt(mean(r^2) + eps) (Sec. 3.3).
//
// The matrix-core pass (bf16, G <= 8) runs one 32-token step of one selected
// block per wavefront on v_mfma_f32_16x16x32_bf16; the workgroup's four
// wavefronts take consecutive steps.
#pragma once

#include "spla_device.h"

namespace spla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));


typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// x = hi + lo as bf16 pairs (about 16 mantissa bits): hi = bf16(x), lo =
// bf16(x - hi), both rounded to nearest. Each pair of hi is converted once
// and read back from the packed bits (element 0 in the low half).
__device__ __forceinline__ void split_bf16x8(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
  uint32_t hp[4], lp[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const uint32_t u =
        __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x[2 * p], x[2 * p + 1]}, bf16x2));
    const float h0 = __uint_as_float(u << 16), h1 = __uint_as_float(u & 0xFFFF0000u);
    hp[p] = u;
    lp[p] = __builtin_bit_cast(
        uint32_t, __builtin_convertvector(f32x2{x[2 * p] - h0, x[2 * p + 1] - h1}, bf16x2));
  }
  hi = __builtin_bit_cast(bf16x8, make_uint4(hp[0], hp[1], hp[2], hp[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(lp[0], lp[1], lp[2], lp[3]));
}

// Rows of S_bar owned by workgroup x of n_wg: row0 .. row0 + nrows - 1.
__device__ __forceinline__ void lin_rows(int D, int x, int n_wg, int* row0, int* nrows) {
  const int rw = (D + n_wg - 1) / n_wg;
  const int r0 = x * rw;
  *row0 = r0;
  *nrows = r0 >= D ? 0 : (D - r0 < rw ? D - r0 : rw);
}

// ------------------------------------------------------------------ merge
// E consecutive floats at byte offset off of the wave-uniform base.
template <int E, bool CO>
__device__ __forceinline__ void load_vec(const float* base, uint32_t off, float (&v)[E]) {
  static_assert(E == 2 || E == 4, "two or four floats per lane");
  if constexpr (E == 4) {
    const uint4 x = Mem<CO>::ld16(base, off);
    v[0] = __uint_as_float(x.x);
    v[1] = __uint_as_float(x.y);
    v[2] = __uint_as_float(x.z);
    v[3] = __uint_as_float(x.w);
  } else {
    const float2 x = Mem<CO>::ld2(base + off / 4);
    v[0] = x.x;
    v[1] = x.y;
  }
}

// Combines the n_rec records `rec` (wave-uniform) of sequence x KV head bh
// for query head g of the group and writes its output row; one wavefront.
// Each half-wavefront takes every other record, lane l owning the E = D / 32
// adjacent coordinates E (l % 32) .. +E-1, so that one load instruction
// fetches two record rows (16 bytes per lane for D = 128); the halves are
// added at the end. The record headers of a batch of 64 records are read
// one record per lane; every load of a batch (and the gain row) is issued
// before any arithmetic. CO: the records are read with Mem<true> (written
// by other workgroups of the same launch).
// HALF: each half-wavefront merges a query head of its own, g + (lane / 32)
// (none past G), over every record, with headers in batches of 32: a
// wavefront then merges two heads at once (groups of 5 or 6 heads; the
// single-launch kernel and the separate merge use the same form, so their
// outputs agree bit for bit).
// ADD: the records carry no share of the global term (the chunked prefill
// computes o_bar and <phi(q), z_bar> for every query in a kernel of its own);
// obar_add (this query's G x D rows) and zq_add (its G values) are added to
// the sums of the records' linear fields instead.
template <typename T, int D, bool CO, bool ADD = false, bool HALF = false, int NP = 8>
__device__ __forceinline__ void merge_head(const Dims& m, float eps, uint32_t flags,
                                           const float* __restrict__ gamma, int all_sel, int L,
                                           const float* rec, int n_rec, int stride,
                                           T* __restrict__ out, int bh, int g,
                                           const float* __restrict__ obar_add = nullptr,
                                           const float* __restrict__ zq_add = nullptr) {
  static_assert(!(ADD && HALF), "one head per wavefront with ADD");
  constexpr int E = D / 32;            // coordinates per lane
  // NP: record pairs (HALF: records) per load batch
  constexpr int HB = HALF ? 32 : 64;   // records per batch of headers
  constexpr int RS = HALF ? NP : 2 * NP;  // records per batch of bodies
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group;
  const int lane = threadIdx.x & 63, hf = lane >> 5;
  const int gh = HALF ? g + hf : g;       // this lane's head
  const bool gon = gh < G;                // HALF with odd G: the last half idles
  const int gg = gon ? gh : g;            // its row in the records
  const int c0 = E * (lane & 31);
  const int64_t orow = ((int64_t)b * m.hq + h * G + gg) * D + c0;
  const bool rla = !(flags & SPLA_FLAG_NO_RLA);
  float gm[E];
#pragma unroll
  for (int e = 0; e < E; ++e) gm[e] = gamma[(int64_t)(h * G + gg) * D + c0 + e];
  float M = -INFINITY, l = 0.f, zt = 0.f;
  float osp[E], ot[E];
#pragma unroll
  for (int e = 0; e < E; ++e) osp[e] = ot[e] = 0.f;
  if constexpr (ADD) {  // once per coordinate: the halves are added at the end
#pragma unroll
    for (int e = 0; e < E; ++e) ot[e] = hf ? 0.f : obar_add[g * D + c0 + e];
  }
  auto red_max = [](float v) { return HALF ? half_wave_max(v) : wave_max(v); };
  auto red_sum = [](float v) { return HALF ? half_wave_sum(v) : wave_sum(v); };
  for (int x0 = 0; x0 < n_rec; x0 += HB) {
    // headers: lane u holds record x0 + u (HALF: lane u of each half)
    const int ul = HALF ? (lane & 31) : lane;
    const bool hv = x0 + ul < n_rec;
    const float* hr = rec + (int64_t)(hv ? x0 + ul : 0) * stride;
    // loaded whether or not hv (no branch), selected after the first bodies
    // are issued, so that no wait for them comes before those loads
    const float hm0 = Mem<CO>::ld(hr + gg), hl0 = Mem<CO>::ld(hr + 16 + gg);
    const float hz0 = Mem<CO>::ld(hr + 32 + gg);
    const int nb_here = n_rec - x0 < HB ? n_rec - x0 : HB;
    float sc_l = 0.f;  // lane u: weight exp(m - M) of record x0 + u
    // bodies, RS records at a time (the first batch is issued with the headers)
    for (int u0 = 0; u0 < nb_here; u0 += RS) {
      float a[NP][E], aw[NP][E];
#pragma unroll
      for (int u = 0; u < NP; ++u) {
        const int xr = HALF ? x0 + u0 + u : x0 + u0 + 2 * u + hf;
        const uint32_t o = (uint32_t)((int64_t)(xr < n_rec ? xr : 0) * stride + kPartHead + c0) * 4u;
        load_vec<E, CO>(rec, o + (uint32_t)(gg * D) * 4u, a[u]);
        load_vec<E, CO>(rec, o + (uint32_t)((G + gg) * D) * 4u, aw[u]);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (u0 == 0) {  // fold this batch of headers into the running max
        const float hm = hv ? hm0 : -INFINITY, hl = hv ? hl0 : 0.f, hz = hv ? hz0 : 0.f;
        const float bm = fmaxf(M, red_max(hm));
        const float alpha = M == -INFINITY ? 0.f : __expf(M - bm);
        l *= alpha;
#pragma unroll
        for (int e = 0; e < E; ++e) osp[e] *= alpha;
        M = bm;
        l += red_sum(hm == -INFINITY ? 0.f : hl * __expf(hm - M));
        zt += red_sum(hz);
        sc_l = hm == -INFINITY ? 0.f : __expf(hm - M);
      }
#pragma unroll
      for (int u = 0; u < NP; ++u) {
        float sc;
        bool ok;
        if constexpr (HALF) {
          const int r = u0 + u;  // this record within the batch, in each half
          const float s0 = r < nb_here ? lane_f32(sc_l, r) : 0.f;
          const float s1 = r < nb_here ? lane_f32(sc_l, 32 + r) : 0.f;
          ok = r < nb_here;
          sc = hf ? s1 : s0;
        } else {
          const int r0 = u0 + 2 * u;  // this pair's records within the batch: r0, r0 + 1
          const float s0 = r0 < nb_here ? lane_f32(sc_l, r0) : 0.f;
          const float s1 = r0 + 1 < nb_here ? lane_f32(sc_l, r0 + 1) : 0.f;
          ok = r0 + hf < nb_here;
          sc = hf ? s1 : s0;
        }
#pragma unroll
        for (int e = 0; e < E; ++e) {
          osp[e] = fmaf(a[u][e], sc, osp[e]);
          ot[e] += ok ? aw[u][e] : 0.f;
        }
      }
    }
  }
  if constexpr (!HALF) {
#pragma unroll
    for (int e = 0; e < E; ++e) {  // the two halves' records
      osp[e] += xor32(osp[e]);
      ot[e] += xor32(ot[e]);
    }
  }
  if constexpr (ADD) zt += zq_add[g];
  float o[E];
  if (L == 0) {
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = 0.f;
  } else {
    // residual r = o_bar - o_tilde (over its normaliser with RLA_NORMALIZE);
    // out = o_sparse + gamma r / rms(r). When every token was selected there
    // is no residual branch and out = o_sparse (also at eps = 0)
    const bool res = rla && !all_sel;
    const float den = (flags & SPLA_FLAG_RLA_NORMALIZE) ? zt : 1.f;
    float rr[E];
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      osp[e] /= l;
      rr[e] = res ? ot[e] / den : 0.f;
      ss += rr[e] * rr[e];
    }
    ss = HALF ? half_wave_sum(ss) : wave_sum(hf ? 0.f : ss);  // each coordinate once
    const float inv = 1.0f / sqrtf(ss / D + eps);
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = res ? fmaf(gm[e] * rr[e], inv, osp[e]) : osp[e];
  }
  if (HALF ? gon : hf == 0) {
    if constexpr (E == 4) {
      Elem<T>::store4(out, orow, o);
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) Elem<T>::store(out, orow + e, o[e]);
    }
  }
}

// Whether a group's merge takes two query heads per wavefront (HALF): the
// groups above four heads that the single-launch kernel also runs.
SPLA_HD bool merge_halves(int G) { return G > 4 && G <= kFusedMaxGroup; }

// ------------------------------------------------------ matrix-core pass

// LDS of one sparse workgroup for groups of at most GC heads: the B
// operands of the first products (q, phi(q) hi, phi(q) lo per k-step, in
// lane order), the four wavefronts' accumulators (exact columns 0 .. GC-1,
// linear columns GC .. 2 GC-1), phi(q) and this workgroup's rows of S_bar.
// The accumulators come last and are written only at the end of sparse_body,
// so a kernel may lay other LDS over them until then (kOverlay).
template <int D, int GC>
struct SparseSmem {
  uint4 qops[3][D / 32][64];
  float m[kSparseWaves][16], l[kSparseWaves][16];
  float phq[GC][D];
  float S[kSparsePre * 256];
  float zb[D];
  float o[kSparseWaves][D][2 * GC + 1];
  static constexpr size_t kOverlay = sizeof(qops) + sizeof(m) + sizeof(l) + sizeof(phq) +
                                     sizeof(S) + sizeof(zb);  // offset of o
};

// What a workgroup loads and computes before it knows its blocks: its rows
// of S_bar and z_bar (the query operands go to LDS), then its share of
// phi(q) S_bar (ob: output e = tid + 256 i is head e / D, coordinate e % D)
// and of <phi(q), z_bar> (zq, thread g < G for head g).
struct SparseRegs {
  float spre[kSparsePre];
  float zbv;
  int row0, nrows;
  float ob[4];
  float zq;
};

// The loads of sparse_prologue: this lane's query elements (raw) and this
// workgroup's rows of S_bar and z_bar (into r).
template <int D, int GC, bool LIN = true>
__device__ __forceinline__ void sparse_prologue_load(const Dims& m, const bf16_t* __restrict__ q,
                                                     const float* __restrict__ S,
                                                     const float* __restrict__ zbar, int bh,
                                                     int x, int n_wg, SparseRegs& r,
                                                     uint4 (&raw)[D / 32]) {
  constexpr int KS = D / 32;
  const int b = bh / m.hkv, h = bh % m.hkv;
  const int G = m.group;
  const int tid = threadIdx.x, lane = tid & 63;
  const int j = lane & 15, g = lane >> 4;
  const bool exact_col = j < 8;
  const int head = exact_col ? j : j - 8;
  const bool live = head < G;
  const bf16_t* qrow = q + ((int64_t)b * m.hq + h * G + (live ? head : 0)) * D + 8 * g;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) raw[ks] = *reinterpret_cast<const uint4*>(qrow + 32 * ks);
  lin_rows(D, x, n_wg, &r.row0, &r.nrows);
  if constexpr (!LIN) {
#pragma unroll
    for (int u = 0; u < kSparsePre; ++u) r.spre[u] = 0.f;
    r.zbv = 0.f;
    r.nrows = 0;
  } else {
    // the first kSparsePre * 256 / D rows (sparse_linear reads any further
    // ones itself); loads issued whether or not in range (from row 0 when
    // not): no branch
    const float* Sh = S + (int64_t)bh * D * D;
#pragma unroll
    for (int u = 0; u < kSparsePre; ++u) {
      const int e = tid + 256 * u;
      const bool ok = e < r.nrows * D;
      const float v = Sh[ok ? r.row0 * D + e : 0];
      r.spre[u] = ok ? v : 0.f;
    }
  }
  if constexpr (LIN) {
    const bool ok = tid < r.nrows;
    const float v = zbar[(int64_t)bh * D + (ok ? r.row0 + tid : 0)];
    r.zbv = ok ? v : 0.f;
  }
}

// The arithmetic of the prologue, from the query elements raw.
template <int D, int GC>
__device__ __forceinline__ void sparse_prologue_finish(const Dims& m, const uint4 (&raw)[D / 32],
                                                       SparseSmem<D, GC>& sm) {
  constexpr int KS = D / 32;
  const int G = m.group;
  const int tid = threadIdx.x, lane = tid & 63;
  const int j = lane & 15, g = lane >> 4;
  const bool exact_col = j < 8;
  const int head = exact_col ? j : j - 8;
  const bool live = head < G;
  // phi(q) of this lane's head (every lane computes it; columns 0..7 discard it)
  float xv[KS][8];
  float mx = -INFINITY;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const bf16x8 v = __builtin_bit_cast(bf16x8, raw[ks]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xv[ks][e] = (float)v[e];
      mx = fmaxf(mx, xv[ks][e]);
    }
  }
  mx = fmaxf(mx, xor16(mx));
  mx = fmaxf(mx, xor32(mx));
  float sum = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xv[ks][e] = __expf(xv[ks][e] - mx);
      sum += xv[ks][e];
    }
  sum += xor16(sum);
  sum += xor32(sum);
  const float inv = 1.0f / sum;
  // wavefront 0 leaves the operands and phi(q) (hi + lo) in LDS; absent
  // operands are masked to zero (bit masks, not selects between arrays)
  const bool lin = !exact_col && live;
  const uint32_t mq = (exact_col && live) ? 0xFFFFFFFFu : 0u, ml = lin ? 0xFFFFFFFFu : 0u;
  auto masked = [](uint4 v, uint32_t k) { return make_uint4(v.x & k, v.y & k, v.z & k, v.w & k); };
  if ((tid >> 6) == 0) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 hi8, lo8;
      float ph[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float pq = xv[ks][e] * inv;
        const __bf16 hi = (__bf16)pq;
        const __bf16 lo = (__bf16)(pq - (float)hi);
        hi8[e] = hi;
        lo8[e] = lo;
        ph[e] = (float)hi + (float)lo;
      }
      sm.qops[0][ks][lane] = masked(raw[ks], mq);
      sm.qops[1][ks][lane] = masked(__builtin_bit_cast(uint4, hi8), ml);
      sm.qops[2][ks][lane] = masked(__builtin_bit_cast(uint4, lo8), ml);
      if (lin) {
        float4* dst = reinterpret_cast<float4*>(&sm.phq[head][32 * ks + 8 * g]);
        dst[0] = make_float4(ph[0], ph[1], ph[2], ph[3]);
        dst[1] = make_float4(ph[4], ph[5], ph[6], ph[7]);
      }
    }
  }
}

// With g = lane / 16 and j = lane % 16 (the MFMA column), the B operands of
// the first product hold coordinates 32 ks + 8 g .. +7 of head j (columns
// 0..7: q itself, for the exact-branch logits) or of head j - 8 (columns
// 8..15: phi(q) as a bf16 hi + lo pair, for the linear weights); absent heads
// are zero. The four lanes of a column (g = 0..3) hold all d coordinates of
// its head, so the softmax of phi(q) needs only the two lane swaps. Also
// issues the loads of this workgroup's rows of S_bar and z_bar (x of n_wg).
// LIN = false: no share of the global term (no S_bar rows are loaded; ob and
// zq stay zero), for the chunked prefill.
template <int D, int GC, bool LIN = true>
__device__ __forceinline__ void sparse_prologue(const Dims& m, const bf16_t* __restrict__ q,
                                                const float* __restrict__ S,
                                                const float* __restrict__ zbar, int bh, int x,
                                                int n_wg, SparseRegs& r, SparseSmem<D, GC>& sm) {
  uint4 raw[D / 32];
  sparse_prologue_load<D, GC, LIN>(m, q, S, zbar, bh, x, n_wg, r, raw);
  sparse_prologue_finish<D, GC>(m, raw, sm);
}

// This workgroup's rows x of the global linear term (Eq. 15): ob and zq of r,
// from the S_bar rows of r and phi(q) (LDS). Needs nothing from the
// selection, so it runs while the workgroup would otherwise wait for it.
template <int D, int GC, bool LIN = true>
__device__ __forceinline__ void sparse_linear(const Dims& m, const float* __restrict__ S, int bh,
                                              SparseRegs& r, SparseSmem<D, GC>& sm) {
  if constexpr (!LIN) {
    __syncthreads();  // the query operands and phi(q) are in LDS
#pragma unroll
    for (int i = 0; i < 4; ++i) r.ob[i] = 0.f;
    r.zq = 0.f;
    return;
  }
  constexpr int NO = (GC * D + 255) / 256;  // outputs (head, coordinate) per thread
  constexpr int RMAX = kSparsePre * 256 / D;  // rows held in LDS
  static_assert(NO <= 4, "ob holds four outputs");
  const int G = m.group, tid = threadIdx.x;
  const int row0 = r.row0, nrows = r.nrows;
#pragma unroll
  for (int u = 0; u < kSparsePre; ++u) sm.S[tid + 256 * u] = r.spre[u];
  if (tid < D) sm.zb[tid] = r.zbv;
  __syncthreads();  // the query operands, phi(q) and the S_bar rows are in LDS
  // the first RMAX rows from LDS (rows past nrows are zero there; their
  // phi(q) index is clamped), in row order
  const int c = tid % D;  // the coordinate of every output of this thread
  float acc[NO];
#pragma unroll
  for (int i = 0; i < NO; ++i) {
    const int hh = (tid + 256 * i) / D;
    acc[i] = 0.f;
#pragma unroll
    for (int rr = 0; rr < RMAX; ++rr)
      acc[i] = fmaf(sm.phq[hh < G ? hh : 0][min(row0 + rr, D - 1)], sm.S[rr * D + c], acc[i]);
  }
  // a workgroup with more rows (few sparse workgroups per head) reads the
  // rest from global memory, eight rows per batch of loads, in row order
  if (nrows > RMAX) {  // uniform over the workgroup
    const float* Sb = S + (int64_t)bh * D * D + c;
    const int rend = row0 + nrows;
    for (int r0 = row0 + RMAX; r0 < rend; r0 += 8) {
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = Sb[(int64_t)(r0 + j < rend ? r0 + j : row0) * D];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float vj = r0 + j < rend ? v[j] : 0.f;
#pragma unroll
        for (int i = 0; i < NO; ++i) {
          const int hh = (tid + 256 * i) / D;
          acc[i] = fmaf(sm.phq[hh < G ? hh : 0][min(r0 + j, D - 1)], vj, acc[i]);
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < NO; ++i) r.ob[i] = tid + 256 * i < G * D ? acc[i] : 0.f;
  float zq = 0.f;
  if (tid < G) {
    for (int rr = 0; rr < nrows; ++rr) zq = fmaf(sm.phq[tid][row0 + rr], sm.zb[rr], zq);
  }
  r.zq = zq;
}

// The rank-one update of a step (spla_step) for the rows of S_bar (and z_bar)
// a sparse workgroup holds (its lin_rows, all in r.spre / r.zbv, loaded by
// sparse_prologue): S_bar[j][c] += phi(k)_j v_c, z_bar[j] += phi(k)_j, with
// phi(k) the softmax of the appended key over d computed exactly as the
// single-token append does; the updated rows are written back. Nothing
// happens for a sequence that received no token (at capacity).
// The inputs of step_rank1, loaded ahead of their use by step_load: this
// lane's key elements, this thread's value element, the tokens appended.
template <int D>
struct StepIn {
  float x[D / 64];
  float vc;
  int app;
};

template <int D>
__device__ __forceinline__ void step_load(const Dims& m, const bf16_t* __restrict__ k_step,
                                          const bf16_t* __restrict__ v_step,
                                          const int32_t* __restrict__ appended, int bh,
                                          StepIn<D>& in) {
  const int tid = threadIdx.x, lane = tid & 63;
  in.app = appended[bh / m.hkv];
#pragma unroll
  for (int e = 0; e < D / 64; ++e)
    in.x[e] = bf16_to_f32(k_step[(int64_t)bh * D + lane + 64 * e].bits);
  in.vc = bf16_to_f32(v_step[(int64_t)bh * D + tid % D].bits);
}

template <int D>
__device__ __forceinline__ void step_apply(const Dims& m, StepIn<D>& in, float* S, float* zbar,
                                           int bh, SparseRegs& r) {
  const int tid = threadIdx.x;
  if (in.app <= 0) return;  // uniform over the workgroup
  float mx = -INFINITY;
#pragma unroll
  for (int e = 0; e < D / 64; ++e) mx = fmaxf(mx, in.x[e]);
  mx = wave_max(mx);
  float sum = 0.f;
#pragma unroll
  for (int e = 0; e < D / 64; ++e) {
    in.x[e] = expf(in.x[e] - mx);
    sum += in.x[e];
  }
  sum = wave_sum(sum);
  float ph[D / 64];
#pragma unroll
  for (int e = 0; e < D / 64; ++e) ph[e] = in.x[e] / sum;
  float* Sh = S + (int64_t)bh * D * D;
#pragma unroll
  for (int u = 0; u < kSparsePre; ++u) {
    const int e = tid + 256 * u;
    const int row = r.row0 + e / D;  // uniform over the wavefront
    const float pr = lane_f32(ph[(row % D) / 64], row % 64);
    if (e < r.nrows * D) {
      r.spre[u] = fmaf(pr, in.vc, r.spre[u]);
      Sh[r.row0 * D + e] = r.spre[u];
    }
  }
  const int row = r.row0 + tid;
  float pz = __shfl(ph[0], row % 64, kWave);
  if constexpr (D / 64 > 1) {
    const float p1 = __shfl(ph[1], row % 64, kWave);
    pz = (row % D) / 64 ? p1 : pz;
  }
  if (tid < r.nrows) {
    r.zbv += pz;
    zbar[(int64_t)bh * D + row] = r.zbv;
  }
}

template <int D>
__device__ __forceinline__ void step_rank1(const Dims& m, const bf16_t* __restrict__ k_step,
                                           const bf16_t* __restrict__ v_step,
                                           const int32_t* __restrict__ appended, float* S,
                                           float* zbar, int bh, SparseRegs& r) {
  StepIn<D> in;
  step_load<D>(m, k_step, v_step, appended, bh, in);
  step_apply<D>(m, in, S, zbar, bh, r);
}

// Selected block of this wavefront's step: entry p of the selection, where
// workgroup x's wavefront w takes step 4 x + w and a block has BLK / 32 steps.
template <int BLK>
__device__ __forceinline__ int sparse_step_entry(int x) {
  return (x * kSparseWaves + (int)(threadIdx.x >> 6)) / (BLK / 32);
}

// One 32-token step of one selected block per wavefront, then the record of
// workgroup x (of n_wg) of sequence x KV head bh. blk_sel: this wavefront's
// block (entry sparse_step_entry of the selection; -1 for none); L: the
// sequence length. For the two 16-row tiles of a step the key row loaded by
// lane l is token 8 (i / 4) + 4 tile + (i % 4), i = l % 16 (the bf16 cache
// stores each step in exactly this order: k_off, v_off), so that after
// S = K [Q | phi(Q)]^T the accumulator rows held by lane l are exactly the
// tokens 8 g .. 8 g + 7 of the step, in order - the layout the second product
// needs for its B operand. Columns 0..7 carry the exact-branch logits of heads
// 0..G-1, columns 8..15 the linear weights <phi(q), phi(k)> of the same heads;
// one accumulator holds both. phi(k) and the probabilities enter the products
// as bf16 hi + lo pairs (about 16 mantissa bits); accumulation is fp32. CO:
// the record is written with Mem<true> (merged by another workgroup of the
// same launch).
// The keys and values of one wavefront's step, as loaded (k_off / v_off
// order: chunk (mt KS + ks) 64 + lane and t 64 + lane), and how many of its
// 32 tokens exist.
template <int D>
struct SparseKV {
  bf16x8 ka[2][D / 32];
  bf16x8 va[D / 16];
  int n_valid;
};

// This wavefront's block and step: the block selected for it (blk_sel, -1 for
// none; clipped to the last block) and its valid token count (0: nothing).
template <int BLK>
__device__ __forceinline__ int sparse_step_block(const Dims& m, int blk_sel, int& L, int x,
                                                 int* n_valid, int ch_in = -1) {
  const int ch = ch_in >= 0 ? ch_in : (x * kSparseWaves + (int)(threadIdx.x >> 6)) % (BLK / 32);
  L = min(max(L, 0), m.cap);
  const int nb = (L + BLK - 1) / BLK;
  const int blk = blk_sel >= nb ? nb - 1 : blk_sel;
  *n_valid = (blk_sel >= 0 && nb > 0) ? min(32, block_count(L, BLK, blk) - ch * 32) : 0;
  return blk;
}

// Issues the loads of step ch of block blk of (sequence, KV head) bh: from the
// per-sequence cache, or from the block's page of a paged pool (table given;
// an entry out of range reads page 0). blk >= 0.
template <int D, int BLK>
__device__ __forceinline__ void sparse_load(const Dims& m, const bf16_t* __restrict__ kc,
                                            const bf16_t* __restrict__ vc, int blk, int bh,
                                            int x, const int32_t* __restrict__ table,
                                            SparseKV<D>& kv, int ch_in = -1) {
  constexpr int KS = D / 32, MT = D / 16;
  const int lane = threadIdx.x & 63;
  const int ch = ch_in >= 0 ? ch_in : (x * kSparseWaves + (int)(threadIdx.x >> 6)) % (BLK / 32);
  int64_t step0;
  if (table) {
    const int p = block_page(m, table, bh, blk);
    step0 = (((int64_t)(p < 0 ? 0 : p) * m.hkv + bh % m.hkv) * BLK + ch * 32) * D;
  } else {
    step0 = ((int64_t)bh * m.cap + (int64_t)blk * BLK + ch * 32) * D;
  }
  const bf16x8* kst = reinterpret_cast<const bf16x8*>(kc + step0) + lane;
  const bf16x8* vst = reinterpret_cast<const bf16x8*>(vc + step0) + lane;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kv.ka[mt][ks] = kst[(mt * KS + ks) * 64];
#pragma unroll
  for (int t = 0; t < MT; ++t) kv.va[t] = vst[t * 64];
}

// The two products of one step (n_valid > 0): S = K [q | phi(q)]^T, the
// step's softmax over the exact columns, and acc_o = V^T P; m_run / l_run get
// the step's max and sum (exact columns) or the sum of the linear weights.
// ONLINE: acc_o, m_run and l_run already hold earlier steps of this
// wavefront; the exact columns are rescaled to the running max first.
template <int D, int GC, bool ONLINE = false>
__device__ __forceinline__ void sparse_mma(float s, SparseKV<D>& kv, SparseSmem<D, GC>& sm,
                                           floatx4 (&acc_o)[D / 16], float& m_run,
                                           float& l_run) {
  constexpr int KS = D / 32;     // k-steps of the first product
  constexpr int MT = D / 16;     // coordinate tiles of the second product
  const int lane = threadIdx.x & 63;
  const int j = lane & 15, g = lane >> 4;
  const bool exact_col = j < 8;
  const int n_valid = kv.n_valid;
  floatx4 sw[2];
  float zinv[2];  // 1 / sum exp(k - max k) of this lane's key row, per tile
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    sw[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          kv.ka[mt][ks], __builtin_bit_cast(bf16x8, sm.qops[0][ks][lane]), sw[mt], 0, 0, 0);
    // exp(k - max k) of this lane's key row (row i of the tile), spread over
    // lanes i + 16 g'; the 1 / sum of phi(k) is applied to the result rows
    float mx = -INFINITY;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) mx = fmaxf(mx, (float)kv.ka[mt][ks][e]);
    mx = fmaxf(mx, xor16(mx));
    mx = fmaxf(mx, xor32(mx));
    const float mxl = mx * kLog2e;
    // exp(k - max k) k-step by k-step, each step straight into its products
    float sum = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 fh, fl;
      float f[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        f[e] = __builtin_amdgcn_exp2f(fmaf((float)kv.ka[mt][ks][e], kLog2e, -mxl));
        sum += f[e];
      }
      split_bf16x8(f, fh, fl);
      const bf16x8 ph = __builtin_bit_cast(bf16x8, sm.qops[1][ks][lane]);
      const bf16x8 pl = __builtin_bit_cast(bf16x8, sm.qops[2][ks][lane]);
      sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh, ph, sw[mt], 0, 0, 0);
      sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh, pl, sw[mt], 0, 0, 0);
      sw[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fl, ph, sw[mt], 0, 0, 0);
    }
    sum += xor16(sum);
    sum += xor32(sum);
    zinv[mt] = 1.0f / sum;
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
    const float xx = sw[e >> 2][e & 3];
    val[e] = exact_col ? (ok ? xx * s : -INFINITY) : (ok ? xx * zi : 0.f);
    cmax = fmaxf(cmax, val[e]);
  }
  cmax = fmaxf(cmax, xor16(cmax));
  cmax = fmaxf(cmax, xor32(cmax));
  float alpha = 1.f;  // ONLINE: the earlier steps' scale (exact columns)
  if constexpr (ONLINE) {
    if (exact_col) {
      const float mn = fmaxf(m_run, cmax);
      alpha = m_run == -INFINITY ? 0.f : __expf(m_run - mn);
      cmax = mn;
    }
  }
  float psum = 0.f;
  bf16x8 bh8, bl8;
  float pv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    pv[e] = exact_col ? __builtin_amdgcn_exp2f((val[e] - cmax) * kLog2e) : val[e];
    psum += pv[e];
  }
  split_bf16x8(pv, bh8, bl8);
  psum += xor16(psum);
  psum += xor32(psum);
  if constexpr (ONLINE) {
#pragma unroll
    for (int t = 0; t < MT; ++t) acc_o[t] = acc_o[t] * alpha;
    l_run = fmaf(l_run, alpha, psum);
  } else {
    l_run = psum;
  }
  m_run = exact_col ? cmax : -INFINITY;
  if (n_valid < 32) {  // rows past the sequence end may hold anything: zero them
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (8 * g + e >= n_valid) kv.va[t][e] = (__bf16)0.f;
  }
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv.va[t], bh8, acc_o[t], 0, 0, 0);
    acc_o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv.va[t], bl8, acc_o[t], 0, 0, 0);
  }
}

// Merges the four wavefronts' accumulators into the record of workgroup x:
// row bh of the records, or rec_row (the chunked prefill keeps one row per
// (sequence, KV head, position)).
template <int D, bool CO, int GC>
__device__ __forceinline__ void sparse_record(const Dims& m, const floatx4 (&acc_o)[D / 16],
                                              float m_run, float l_run, int bh, int x, int n_wg,
                                              const SparseRegs& r, SparseSmem<D, GC>& sm,
                                              float* __restrict__ part, int stride,
                                              int64_t rec_row) {
  constexpr int MT = D / 16;
  constexpr int NO = (GC * D + 255) / 256;  // outputs (head, coordinate) per thread
  const int G = m.group;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int j = lane & 15, g = lane >> 4;
  const bool exact_col = j < 8;
  const int head = exact_col ? j : j - 8;
  const bool live = head < G;
  if (live) {  // only the live columns: exact heads to 0 .., linear heads to GC ..
    const int cj = exact_col ? head : GC + head;
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) sm.o[w][16 * t + 4 * g + rr][cj] = acc_o[t][rr];
  }
  if (lane < 16) {
    sm.m[w][lane] = m_run;
    sm.l[w][lane] = l_run;
  }
  __syncthreads();
  float* rec = part + ((rec_row >= 0 ? rec_row : (int64_t)bh) * n_wg + x) * stride;
#pragma unroll
  for (int i = 0; i < NO; ++i) {
    const int e = tid + 256 * i;
    if (e >= G * D) break;
    const int hh = e / D, c = e % D;
    float M = -INFINITY;
#pragma unroll
    for (int xx = 0; xx < kSparseWaves; ++xx) M = fmaxf(M, sm.m[xx][hh]);
    float a = 0.f, aw = 0.f;
#pragma unroll
    for (int xx = 0; xx < kSparseWaves; ++xx) {
      const float sc = sm.m[xx][hh] == -INFINITY ? 0.f : __expf(sm.m[xx][hh] - M);
      a = fmaf(sm.o[xx][c][hh], sc, a);
      aw += sm.o[xx][c][GC + hh];
    }
    Mem<CO>::st(rec + kPartHead + hh * D + c, a);
    Mem<CO>::st(rec + kPartHead + (G + hh) * D + c, r.ob[i] - aw);
  }
  if (tid < G) {
    float M = -INFINITY;
#pragma unroll
    for (int xx = 0; xx < kSparseWaves; ++xx) M = fmaxf(M, sm.m[xx][tid]);
    float l = 0.f, zw = 0.f;
#pragma unroll
    for (int xx = 0; xx < kSparseWaves; ++xx) {
      l += sm.m[xx][tid] == -INFINITY ? 0.f : sm.l[xx][tid] * __expf(sm.m[xx][tid] - M);
      zw += sm.l[xx][8 + tid];
    }
    Mem<CO>::st(rec + tid, M);
    Mem<CO>::st(rec + 16 + tid, l);
    Mem<CO>::st(rec + 32 + tid, r.zq - zw);
  }
}

// One 32-token step of one selected block per wavefront, then the record of
// workgroup x (of n_wg) of sequence x KV head bh. blk_sel: this wavefront's
// block (entry sparse_step_entry of the selection; -1 for none); L: the
// sequence length. For the two 16-row tiles of a step the key row loaded by
// lane l is token 8 (i / 4) + 4 tile + (i % 4), i = l % 16 (the bf16 cache
// stores each step in exactly this order: k_off, v_off), so that after
// S = K [Q | phi(Q)]^T the accumulator rows held by lane l are exactly the
// tokens 8 g .. 8 g + 7 of the step, in order - the layout the second product
// needs for its B operand. Columns 0..7 carry the exact-branch logits of heads
// 0..G-1, columns 8..15 the linear weights <phi(q), phi(k)> of the same heads;
// one accumulator holds both. phi(k) and the probabilities enter the products
// as bf16 hi + lo pairs (about 16 mantissa bits); accumulation is fp32. CO:
// the record is written with Mem<true> (merged by another workgroup of the
// same launch).
template <int D, int BLK, bool CO, int GC>
__device__ __forceinline__ void sparse_body(const Dims& m, float s,
                                            const bf16_t* __restrict__ kc,
                                            const bf16_t* __restrict__ vc,
                                            int blk_sel, int L,
                                            int bh, int x, int n_wg, const SparseRegs& r,
                                            SparseSmem<D, GC>& sm, float* __restrict__ part,
                                            int stride,
                                            const int32_t* __restrict__ table = nullptr,
                                            int64_t rec_row = -1) {
  constexpr int MT = D / 16;
  SparseKV<D> kv;
  const int blk = sparse_step_block<BLK>(m, blk_sel, L, x, &kv.n_valid);
  floatx4 acc_o[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc_o[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;  // exact columns: max / sum; linear columns: sum
  // loads and their use in one branch: a load issued in one branch and used
  // in another leaves the compiler assuming it may still be in flight after
  // them, and it then waits for every store before the record's next ones
  if (kv.n_valid > 0) {
    sparse_load<D, BLK>(m, kc, vc, blk, bh, x, table, kv);
    sparse_mma<D, GC>(s, kv, sm, acc_o, m_run, l_run);
  }
  sparse_record<D, CO, GC>(m, acc_o, m_run, l_run, bh, x, n_wg, r, sm, part, stride, rec_row);
}

// sparse_body with SPW consecutive 32-token steps per wavefront: step
// (x kSparseWaves + w) SPW + j of the selection (B / 32 steps per selected
// block, entries of sel_row), accumulated online, then one record per
// workgroup (n_wg = k B / (32 kSparseWaves SPW) records per query).
template <int D, int BLK, bool CO, int GC, int SPW>
__device__ __forceinline__ void sparse_body_steps(const Dims& m, float s,
                                                  const bf16_t* __restrict__ kc,
                                                  const bf16_t* __restrict__ vc,
                                                  const int32_t* __restrict__ sel_row, int L,
                                                  int bh, int x, int n_wg, const SparseRegs& r,
                                                  SparseSmem<D, GC>& sm, float* __restrict__ part,
                                                  int stride,
                                                  const int32_t* __restrict__ table,
                                                  int64_t rec_row) {
  constexpr int MT = D / 16, CPB = BLK / 32;
  floatx4 acc_o[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc_o[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const int g0 = (x * kSparseWaves + (int)(threadIdx.x >> 6)) * SPW;
#pragma unroll
  for (int j = 0; j < SPW; ++j) {
    const int gs = g0 + j, e = gs / CPB, ch = gs % CPB;
    const int v = e < m.k ? sel_row[e] : -1;
    const int blk_sel = __builtin_amdgcn_readfirstlane(v);
    SparseKV<D> kv;
    int Lj = L;
    const int blk = sparse_step_block<BLK>(m, blk_sel, Lj, x, &kv.n_valid, ch);
    if (kv.n_valid > 0) {
      sparse_load<D, BLK>(m, kc, vc, blk, bh, x, table, kv, ch);
      if (j == 0) sparse_mma<D, GC>(s, kv, sm, acc_o, m_run, l_run);
      else sparse_mma<D, GC, true>(s, kv, sm, acc_o, m_run, l_run);
    }
  }
  sparse_record<D, CO, GC>(m, acc_o, m_run, l_run, bh, x, n_wg, r, sm, part, stride, rec_row);
}

}  // namespace spla
