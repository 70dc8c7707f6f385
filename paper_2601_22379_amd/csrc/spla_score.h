// Block scoring of one tile of 64 blocks of one (sequence, KV head)
// (Sec. 3.1), shared by the scoring kernel and the single-launch decode
// kernel. Within a tile each wavefront takes 16 blocks, lane = (block,
// quarter of the head dimension); every 16-byte load of the tile-interleaved
// statistics is a contiguous 256 B run per 16 lanes, and the loads are
// nontemporal (each byte is read once per step). For head m of the group the
// log block mass is
//   ell_m(i) = s q_m.mu_i + ln n_i + ln(1 + 1/2 s^2 sum_j q_mj^2 M2_ij / n_i)
// (Eqs. 8 and 10, diagonal covariance M2/n): eight coordinates at a time in
// fp32 (the query coefficients reach the lanes by DPP row broadcasts, not
// LDS reads), those partial sums accumulated in fp64 and summed over the four
// quarters with a cross-lane reduce-scatter; lane (block, quarter) then
// finishes heads quarter, quarter+4, ... Each tile yields exp(ell - tile max)
// per head and block and the (max, sum) of its 64 blocks per head, from
// which the selection forms each head's normaliser Z (Eq. 9) without another
// pass over the statistics.
#pragma once

#include "spla_device.h"

namespace spla {

constexpr int kScoreGroup = 16;  // blocks per wavefront
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int NJ>
struct TileBuf {
  float4 mu[NJ], m2[NJ];
};

// Issues the statistics loads of item t (sequence x KV head x tile) for this
// lane; an item past the run (valid = false) re-reads the first 16 bytes of
// the buffer, so every path issues the same loads and no wait depends on the
// branch taken.
template <int NJ>
__device__ __forceinline__ void load_tile(const Dims& m, const float* __restrict__ stats, int t,
                                          bool valid, int first_order, int bi, int qt,
                                          TileBuf<NJ>& buf) {
  const int bh = t / m.n_tiles, tile = t % m.n_tiles;
  const int64_t blk = (int64_t)tile * kTileBlocks + bi;
  // first order: the second-moment loads re-read the means (same lines)
  const f32x4* pm = reinterpret_cast<const f32x4*>(
      valid ? stats + stats_off4(m, bh, blk, 0, qt * NJ) : stats);
  const f32x4* pv = reinterpret_cast<const f32x4*>(
      valid ? stats + stats_off4(m, bh, blk, first_order ? 0 : 1, qt * NJ) : stats);
  const int stride = valid ? kTileBlocks : 0;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {  // interleaved: group j is usable once its two loads land
    const f32x4 x = __builtin_nontemporal_load(pm + j * stride);
    const f32x4 y = __builtin_nontemporal_load(pv + j * stride);
    buf.mu[j] = make_float4(x[0], x[1], x[2], x[3]);
    buf.m2[j] = make_float4(y[0], y[1], y[2], y[3]);
  }
}

// Coefficient table of sequence x KV head bh: s q (table 0) and s^2 q^2 / 2
// (table 1) per head, laid out [quarter][(table * G + head) * 32 + c] for
// coordinate 32 quarter + c (D = 128; D = 64 uses c < 16). load_q issues the
// query loads, write_table fills the table; clamped entries rewrite the last
// element's value.
template <int G, int D>
struct QRegs {
  float x[(G * D + 255) / 256];
};

template <int G, typename T, int D>
__device__ __forceinline__ void load_q(const Dims& m, const T* __restrict__ q, int bh,
                                       QRegs<G, D>& r) {
  constexpr int QE = (G * D + 255) / 256;
  const int b = bh / m.hkv, h = bh % m.hkv;
#pragma unroll
  for (int i = 0; i < QE; ++i) {
    const int e = min((int)threadIdx.x + 256 * i, G * D - 1);
    r.x[i] = Elem<T>::load(q, ((int64_t)b * m.hq + h * G + e / D) * D + e % D);
  }
}

template <int G, int D>
__device__ __forceinline__ void write_table(const QRegs<G, D>& r, double s, float (*sco)[2 * G * 32]) {
  constexpr int Q = D / 4;
  constexpr int QE = (G * D + 255) / 256;
#pragma unroll
  for (int i = 0; i < QE; ++i) {
    const int e = min((int)threadIdx.x + 256 * i, G * D - 1);
    const int mm = e / D, j = e % D;
    const int qq = j / Q, c = j % Q;
    const double x = (double)r.x[i];
    sco[qq][mm * 32 + c] = (float)(s * x);
    sco[qq][(G + mm) * 32 + c] = (float)(0.5 * s * s * x * x);
  }
}

// acc (+)= c[lane N of this lane's 16-lane row] * x: the coefficient reaches
// every lane of the row through a DPP row broadcast, so the products need no
// LDS traffic. Callers keep at least two other VALU instructions between two
// updates of one accumulator and never follow a VALU write of c directly.
template <bool FIRST, int N>
__device__ __forceinline__ void row_bcast_fma(float& acc, float c, float x) {
  if constexpr (FIRST)
    asm volatile("v_mul_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
                 : "=v"(acc) : "v"(c), "v"(x), "i"(N));
  else
    asm volatile("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
                 : "+v"(acc) : "v"(c), "v"(x), "i"(N));
}

template <int E>
__device__ __forceinline__ float f4_at(const float4& v) {
  static_assert(E >= 0 && E < 4, "float4 element");
  if constexpr (E == 0) return v.x;
  else if constexpr (E == 1) return v.y;
  else if constexpr (E == 2) return v.z;
  else return v.w;
}

// f(Idx<I>{}) for I = B, ..., E - 1: the index is a constant expression in
// every call, whatever the size of the body.
template <int I>
struct Idx {
  static constexpr int v = I;
};
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(Idx<B>{});
    static_for<B + 1, E>(f);
  }
}

// Scores one tile from buf; s_part is this tile's half of the double-buffered
// cross-wavefront scratch. L_arg >= 0 replaces the sequence length and
// out_row >= 0 the row of e_vals / tile_part (the chunked prefill scores
// every query of a chunk, each with its own length, from one load of a tile).
template <int G, int D, bool CO>
__device__ __forceinline__ void score_tile(const Dims& m, const int32_t* __restrict__ seq_lens,
                                           int first_order, int t, const TileBuf<D / 16>& buf,
                                           const float (*sco)[2 * G * 32],
                                           double (*s_part)[G][2], float* __restrict__ e_vals,
                                           double* __restrict__ tile_part, int L_arg = -1,
                                           int out_row = -1) {
  constexpr int NJ = D / 16;
  constexpr int U = (G + 3) / 4;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int qt = lane >> 4;
  const int bh = t / m.n_tiles, tile = t % m.n_tiles;
  const int blk = tile * kTileBlocks + kScoreGroup * w + (lane & 15);
  const int L = L_arg >= 0 ? L_arg : seq_lens[bh / m.hkv];
  const int orow = out_row >= 0 ? out_row : bh;
  const int nb = (L + m.us - 1) / m.us;  // units (blocks or windows) present
  // this lane's coefficients: cf[k] holds entry 16 k + (lane % 16) of its
  // quarter's table, read once per tile
  constexpr int NK = (2 * G * 32) / 16;
  float cf[NK];
#pragma unroll
  for (int k = 0; k < NK; ++k) cf[k] = sco[qt][16 * k + (lane & 15)];
  double am[G], av[G];
#pragma unroll
  for (int mm = 0; mm < G; ++mm) am[mm] = av[mm] = 0.0;
  // eight coordinates at a time in fp32, those partials added in fp64. The
  // 2G partials of a step are updated round-robin, so one accumulator's
  // updates are 2G instructions apart (plus a nop for G = 1).
  asm volatile("s_nop 4");  // spacing after any earlier EXEC / VGPR write
  static_for<0, NJ / 2>([&](auto jpi) {
    constexpr int jp = decltype(jpi)::v;
    float pa[G], pb[G];
    static_for<0, 8>([&](auto ei) {
      constexpr int e8 = decltype(ei)::v;
      constexpr int c = 8 * jp + e8;  // coordinate within the quarter
      const float xm = f4_at<e8 & 3>(buf.mu[2 * jp + (e8 >> 2)]);
      const float xv = f4_at<e8 & 3>(buf.m2[2 * jp + (e8 >> 2)]);
      static_for<0, G>([&](auto mi) {
        constexpr int mm = decltype(mi)::v;
        row_bcast_fma<e8 == 0, c & 15>(pa[mm], cf[mm * 2 + (c >> 4)], xm);
      });
      static_for<0, G>([&](auto mi) {
        constexpr int mm = decltype(mi)::v;
        row_bcast_fma<e8 == 0, c & 15>(pb[mm], cf[(G + mm) * 2 + (c >> 4)], xv);
      });
      if constexpr (G == 1) asm volatile("s_nop 0");
    });
#pragma unroll
    for (int mm = 0; mm < G; ++mm) {
      am[mm] += (double)pa[mm];
      av[mm] += (double)pb[mm];
    }
  });
  // reduce-scatter over the four quarters (qt = lane / 16): lane (block, qt)
  // ends with the sums of heads qt + 4u, u < U (zero past G). Quarters 0, 1
  // keep heads 4u, 4u + 1 and quarters 2, 3 heads 4u + 2, 4u + 3 (half_sum),
  // then even quarters keep the first of those, odd ones the second
  // (row_pair_sum).
  double ra[U], rv[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    double ta[2], tv[2];
#pragma unroll
    for (int r0 = 0; r0 < 2; ++r0) {
      const int hl = 4 * u + r0, hh = hl + 2;
      const double al = hl < G ? am[hl < G ? hl : 0] : 0.0, ah = hh < G ? am[hh < G ? hh : 0] : 0.0;
      const double vl = hl < G ? av[hl < G ? hl : 0] : 0.0, vh = hh < G ? av[hh < G ? hh : 0] : 0.0;
      ta[r0] = half_sum(al, ah);
      tv[r0] = half_sum(vl, vh);
    }
    ra[u] = row_pair_sum(ta[0], ta[1]);
    rv[u] = row_pair_sum(tv[0], tv[1]);
  }
  // lane (block, qt) finishes heads qt + 4u. ln n and ln(1 + x) are O(1)
  // and taken in fp32 from the hardware log2 (about one ulp of log2, so an
  // absolute error ~1e-7 on ell; ln n is the same for every full block);
  // x = rv / n uses the hardware reciprocal. ell itself is fp64.
  constexpr float kLn2f = 0.69314718055994531f;
  const bool valid = blk < nb;
  const int n_i = valid ? min(m.ul, L - blk * m.us) : 1;  // tokens of the unit
  const float rcp_n = __builtin_amdgcn_rcpf((float)n_i);
  const double ln_n = (double)(__builtin_amdgcn_logf((float)n_i) * kLn2f);
  const int nbp = m.n_tiles * kTileBlocks;
  float* ev = e_vals + (int64_t)orow * G * nbp;
  double ell[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int mm = qt + 4 * u;
    double x = ra[u] + ln_n;
    if (!first_order)
      x += (double)(__builtin_amdgcn_logf(1.0f + (float)rv[u] * rcp_n) * kLn2f);
    ell[u] = valid ? x : -INFINITY;
    // the tile offset is the max of the fp32-rounded ell (any common offset
    // works; this one is exact in both precisions)
    const float mx = row_max_to15((float)ell[u]);
    if ((lane & 15) == 15 && mm < G) s_part[w][mm][0] = (double)mx;
  }
  __syncthreads();
  // exp(ell - tile max) = 2^t, t = (ell - tile max) log2(e) in fp64: the
  // tile's 64 blocks share one offset per head; 2^t is the hardware exp2 of
  // t's fp32 head times 1 + (the rest of t) ln 2
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int mm = qt + 4 * u;
    if (mm < G) {
      double tmx = -INFINITY;
#pragma unroll
      for (int x = 0; x < 4; ++x) tmx = fmax(tmx, s_part[x][mm][0]);
      const double t = (ell[u] - tmx) * 1.4426950408889634;
      const float th = (float)t;
      const float tl = (float)(t - (double)th);
      const float eh = __builtin_amdgcn_exp2f(th);
      const float e = valid ? fmaf(eh, tl * kLn2f, eh) : 0.f;
      Mem<CO>::st(ev + (int64_t)mm * nbp + blk, e);
      const double sum = row_sum_to15((double)e);
      if ((lane & 15) == 15) s_part[w][mm][1] = sum;
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
    double* tp = tile_part + (((int64_t)orow * G + tid) * m.n_tiles + tile) * 2;
    Mem<CO>::st(tp, mx);
    Mem<CO>::st(tp + 1, sum);
  }
}


// LDS of the scoring of up to two tiles (one cross-wavefront scratch each).
template <int G>
struct ScoreSmem {
  float sco[4][2 * G * 32];
  double s_part[2][4][G][2];
};

// Scores tiles t, ..., t + NT - 1 of one sequence x KV head (t = item index
// (sequence x KV head) * n_tiles + tile; tiles past the sequence's n_tiles
// are skipped) with the 256 threads of a workgroup; CO: store the results
// with Mem<true> (read by another workgroup of the same launch). Load order:
// the query elements of the coefficient table, then the statistics of every
// tile (16 x 16 B per lane and tile); the table is built while they are in
// flight. Blocks past the sequence end are scored and masked: an early exit
// would let the compiler sink the loads below the barrier.
template <int G, typename T, int D, bool CO, int NT>
__device__ __forceinline__ void score_items(const Dims& m, const float* __restrict__ stats,
                                            const int32_t* __restrict__ seq_lens,
                                            const T* __restrict__ q, double s, int first_order,
                                            int t, float* __restrict__ e_vals,
                                            double* __restrict__ tile_part, ScoreSmem<G>& sm) {
  static_assert(NT == 1 || NT == 2, "one or two tiles per item");
  constexpr int NJ = D / 16;  // float4 loads per lane and statistics part
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int bi = kScoreGroup * w + (lane & 15), qt = lane >> 4;
  const bool second = NT == 2 && (t % m.n_tiles) + 1 < m.n_tiles;
  QRegs<G, D> qr;
  load_q<G, T, D>(m, q, t / m.n_tiles, qr);
  TileBuf<NJ> A, B;
  load_tile<NJ>(m, stats, t, true, first_order, bi, qt, A);
  if constexpr (NT == 2) load_tile<NJ>(m, stats, t + 1, second, first_order, bi, qt, B);
  __builtin_amdgcn_sched_barrier(0);
  write_table<G, D>(qr, s, sm.sco);
  __syncthreads();
  score_tile<G, D, CO>(m, seq_lens, first_order, t, A, sm.sco, sm.s_part[0], e_vals, tile_part);
  if constexpr (NT == 2) {
    if (second)
      score_tile<G, D, CO>(m, seq_lens, first_order, t + 1, B, sm.sco, sm.s_part[1], e_vals,
                           tile_part);
  }
}

}  // namespace spla
