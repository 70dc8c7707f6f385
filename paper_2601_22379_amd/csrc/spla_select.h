// Block selection of one (sequence, KV head) by the threads of one
// workgroup (Sec. 2.1 Eq. 3 with Select = TopK; Sec. 2.2 Eq. 6 group score;
// Sec. 4 forced blocks). The selection kernel runs it with 1024 threads per
// (sequence, KV head); the sparse pass runs it inside each of its workgroups
// (256 threads) when the block count is small enough, which saves a launch.
//
// 1. Each head's normaliser Z_m (Eq. 9) is the log-sum-exp of the 64-block
//    tile partials of the score pass; wavefront w handles heads w, w + NW, ...
//    and leaves the tile weights exp(M_tile,m - Z_m) in LDS (computed as
//    exp(M_tile,m - max) / sum, fp64 sum).
// 2. score(i) = sum_m e_m(i) exp(M_tile(i),m - Z_m), fp64 accumulation,
//    rounded to an fp32 key (scores are positive, so the bit patterns order
//    like the values; +1 keeps every candidate above the excluded 0). Thread
//    t owns the R consecutive blocks t*R .. t*R + R - 1.
// 3. The kp-th largest key (kp = k - forced blocks) is found digit by digit
//    (bits 30..20, 19..10, 9..0; bit 31 is clear): one LDS histogram per
//    digit, each wavefront then reads the whole histogram and finds the digit
//    itself, so a digit costs one barrier. The search stops as soon as the
//    bin holding the kp-th key is taken whole.
// 4. Keys above the threshold, the first `need` keys equal to it (ties go to
//    the lower block id) and the forced blocks (first n_sink, last n_local)
//    are placed in ascending block order by one block-wide prefix sum,
//    staged in LDS and written out by the first k threads.
// The per-key logic is written with bitwise tests and selects: with one
// wavefront per SIMD, branch and exec-mask bookkeeping would dominate.
#pragma once

#include "spla_device.h"

namespace spla {

constexpr int kMaxTiles = SPLA_MAX_BLOCKS / kTileBlocks;  // tiles per sequence

// Block-wide exclusive prefix sum over NW wavefronts (thread order); one barrier.
template <int NW>
__device__ __forceinline__ uint32_t block_excl_scan_u32(uint32_t v, uint32_t* lds, uint32_t* total) {
  const int w = threadIdx.x >> 6;
  const uint32_t x = wave_incl_scan_u32(v);
  if ((threadIdx.x & 63) == 63) lds[w] = x;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t t = lds[i];
    base += i < w ? t : 0u;
    tot += t;
  }
  *total = tot;
  return base + x - v;
}

// R consecutive floats at base + off (4R-byte aligned; zeros when !ok, or
// whatever base holds when !MASK); base is wave-uniform. The loads are issued
// whether or not ok (from base when not): a load under a branch makes the
// compiler wait for it inside the branch, before the loads after it are
// issued.
template <int R, bool CO, bool MASK = true>
__device__ __forceinline__ void load_run(const float* base, int64_t off, bool ok,
                                         float (&out)[R]) {
  const int64_t o = ok ? off : 0;
  if constexpr (R == 1) {
    out[0] = Mem<CO>::ld(base + o);
  } else if constexpr (R == 2) {
    const float2 v = Mem<CO>::ld2(base + o);
    out[0] = v.x;
    out[1] = v.y;
  } else {
#pragma unroll
    for (int j = 0; j < R / 4; ++j) {
      const uint4 v = Mem<CO>::ld16(base, (uint32_t)(o + 4 * j) * 4u);
      out[4 * j] = __uint_as_float(v.x);
      out[4 * j + 1] = __uint_as_float(v.y);
      out[4 * j + 2] = __uint_as_float(v.z);
      out[4 * j + 3] = __uint_as_float(v.w);
    }
  }
  if constexpr (MASK) {
#pragma unroll
    for (int r = 0; r < R; ++r) out[r] = ok ? out[r] : 0.f;
  }
}

// The (max, sum) partial of tile t of the head whose partials start at tp
// (wave-uniform), as one 16-byte load; (-inf, 0) when !ok.
template <bool CO>
__device__ __forceinline__ void load_tile_part(const double* tp, int t, bool ok, double& mx,
                                               double& sum) {
  const uint4 v = Mem<CO>::ld16(tp, (uint32_t)(ok ? t : 0) * 16u);
  const double a = __hiloint2double((int)v.y, (int)v.x), b = __hiloint2double((int)v.w, (int)v.z);
  mx = ok ? a : -INFINITY;
  sum = ok ? b : 0.0;
}

struct RadixPick {
  uint32_t digit;  // bin holding the need-th largest key
  uint32_t above;  // keys in higher bins
  uint32_t cnt;    // keys in that bin
  uint32_t total;  // keys in the histogram
};

// Finds, from a histogram of 64 * BPL bins, the bin holding the need-th
// largest key. Every wavefront computes the same (wave-uniform) answer: lane
// l first sums bins BPL l .. BPL l + BPL - 1 (reading its run from a rotated
// start so that the lanes spread over the LDS banks), then the BPL bins of the
// lane that holds the key are spread one per lane.
template <int BPL>
__device__ __forceinline__ RadixPick radix_pick(const uint32_t* hist, uint32_t need) {
  constexpr int NV = BPL / 4;
  const int lane = threadIdx.x & 63;
  uint32_t c = 0u;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int jj = (j + lane) & (NV - 1);
    const uint4 v = *reinterpret_cast<const uint4*>(hist + BPL * lane + 4 * jj);
    c += v.x + v.y + v.z + v.w;
  }
  const uint32_t pre = wave_incl_scan_u32(c);
  const uint32_t total = lane_u32(pre, 63);
  const uint32_t above_l = total - pre;  // keys in the bins of lanes > l
  const uint64_t here = __ballot(above_l < need && need <= above_l + c);
  const int src = here ? __ffsll((unsigned long long)here) - 1 : 0;
  const uint32_t above_src = lane_u32(above_l, src);
  const uint32_t v = lane < BPL ? hist[BPL * src + lane] : 0u;
  const uint32_t p2 = wave_incl_scan_u32(v);
  const uint32_t a2 = above_src + lane_u32(p2, 63) - p2;  // keys in bins above this one
  const uint64_t here2 = __ballot(lane < BPL && a2 < need && need <= a2 + v);
  const int d = here2 ? __ffsll((unsigned long long)here2) - 1 : 0;
  RadixPick p;
  p.digit = (uint32_t)(BPL * src + d);
  p.above = lane_u32(a2, d);
  p.cnt = lane_u32(v, d);
  p.total = total;
  return p;
}

// LDS of one selection: tile weights [tile][head] (SWN >= n_tiles * G), the
// digit histograms (2048 + 1024 + 1024 bins), each thread's taken and tie
// bits (one word per thread and kind) and the staging of the k output slots.
template <int NT, int SWN>
struct SelectSmem {
  float sw[SWN];
  __align__(16) uint32_t hist[4096];
  uint32_t bits[2][NT];
  int32_t out[SPLA_MAX_TOP_K + 1];
};

// The selection of sequence x KV head bh (length seq_len, clipped to the
// capacity) by the NT threads of a workgroup, thread t owning blocks
// t R .. t R + R - 1 (NT R >= blocks of the capacity). The length is an
// argument so that no load of it sits in front of the first loads here.
// Writes sel[0 .. k) (ascending block ids, -1 padded), meta4 = (selected,
// all selected, length, candidates) and, if so is not NULL, the ids to so as
// well. sel, meta4 and so may point to global memory or to LDS; the caller
// synchronises before reading them. CO: e_vals and tile_part are read, and
// sel and meta4 (then global) written, with Mem<true> (another workgroup of
// the same launch produced / consumes them). SEL_OFF is added to every id
// written to sel (not to so): with SEL_OFF = 2 an entry is never 0, so a
// consumer can poll sel itself for the selection (meta4 may then be NULL).
// WIN: the scoring units are strided selection windows (unit u: tokens
// u us .. u us + ul - 1, Sec. 3.1) and a block's score is the largest group
// score among the windows that share a token with it (max-pooling); wsc is
// LDS for kMaxWindows window scores. GMAX >= G (known at compile time): with
// at most eight heads and eight blocks per thread every head's masses load
// in one batch, and a wavefront that takes a second head's tile partials
// loads them with the first head's. GEX: the group is GMAX exactly.
template <int NT, int R, int SWN, bool CO, int SEL_OFF = 0, bool WIN = false,
          int GMAX = SPLA_MAX_GROUP, bool GEX = false>
__device__ void select_blocks(const Dims& m, int bh, int seq_len,
                              const float* __restrict__ e_vals,
                              const double* __restrict__ tile_part, SelectSmem<NT, SWN>& sm,
                              int32_t* sel, int32_t* meta4, int32_t* so,
                              float* wsc = nullptr) {
  constexpr int NW = NT / 64;
  constexpr int HC0 = R <= 2 ? 16 / R : (R <= 8 ? 4 : 32 / R);
  constexpr int HC = (R <= 8 && GMAX <= 8 && GMAX > HC0) ? GMAX : HC0;  // heads per load batch
  constexpr bool PRE2 = !WIN && GMAX > NW && GMAX <= 2 * NW;  // heads w and w + NW preloaded
  // tiles per lane: n_tiles <= NT R / 64 blocks, or <= kMaxWindows / 64 windows
  constexpr int TJ = WIN ? kMaxWindows / 4096 : (NT * R + 4095) / 4096;
  float* sw = sm.sw;
  uint32_t* hist = sm.hist;
  const int G = GEX ? GMAX : m.group, k = m.k;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nbp = m.n_tiles * kTileBlocks;
  const int i0 = tid * R;
  const int kp = k - m.n_sink - m.n_local;
  const double* tp = tile_part + (int64_t)bh * m.n_tiles * G * 2;
  const float* ev = e_vals + (int64_t)bh * G * nbp;  // this thread's run: + h nbp + i0

  const int L = min(max(seq_len, 0), m.cap);  // a length past the capacity is clipped
  double tm[TJ], ts[TJ];
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    const int t = lane + 64 * j;
    load_tile_part<CO>(tp + (int64_t)(w < G ? w : 0) * m.n_tiles * 2, t, w < G && t < m.n_tiles,
                       tm[j], ts[j]);
  }
  double tm2[PRE2 ? TJ : 1], ts2[PRE2 ? TJ : 1];  // head w + NW
  if constexpr (PRE2) {
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int t = lane + 64 * j, w2 = w + NW;
      load_tile_part<CO>(tp + (int64_t)(w2 < G ? w2 : 0) * m.n_tiles * 2, t,
                         w2 < G && t < m.n_tiles, tm2[j], ts2[j]);
    }
  }
  // nbp is a multiple of 64 >= R: a thread's run is all in or all out; the
  // masses of a run past nbp, or of a head past G, are never used (the keys
  // of blocks past the sequence are 0 whatever they hold)
  float e[HC][R];
  if constexpr (!WIN) {
#pragma unroll
    for (int h = 0; h < HC; ++h)
      load_run<R, CO, false>(ev, (int64_t)h * nbp + i0, h < G && i0 < nbp, e[h]);
  }
  // WIN: the window masses of the first four heads, as runs of four windows
  // starting at 4 (t + j NT) (16-byte loads; a run holding a window below nu
  // lies inside the row), issued here so that they overlap the tile weights
  constexpr int J4 = WIN ? kMaxWindows / (4 * NT) : 1;
  static_assert(!WIN || kMaxWindows % (4 * NT) == 0, "window staging");
  const int nu = WIN ? (L + m.us - 1) / m.us : 0;  // windows present
  uint4 wv[4][J4];
  if constexpr (WIN) {
#pragma unroll
    for (int hh = 0; hh < 4; ++hh)
#pragma unroll
      for (int j = 0; j < J4; ++j) {
        const int u = 4 * (tid + j * NT);
        wv[hh][j] = Mem<CO>::ld16(ev + (int64_t)min(hh, G - 1) * nbp,
                                  (uint32_t)(u < nu ? u : 0) * 4u);
      }
  }

  const int nb = (L + m.B - 1) / m.B;
  if (nb <= k) {  // L == 0 included: nothing or everything is selected
    for (int x = tid; x < k; x += NT) {
      const int v = x < nb ? x : -1;
      Mem<CO>::st(sel + x, v + SEL_OFF);
      if (so) so[x] = v;
    }
    if (tid == 0 && meta4) {
      Mem<CO>::st(meta4 + 0, nb);
      Mem<CO>::st(meta4 + 1, 1);
      Mem<CO>::st(meta4 + 2, L);
      Mem<CO>::st(meta4 + 3, 0);
    }
    return;
  }
  const int n_tu = ((WIN ? nu : nb) + kTileBlocks - 1) / kTileBlocks;  // unit tiles present
  for (int x = tid; x < 1024; x += NT) reinterpret_cast<uint4*>(hist)[x] = make_uint4(0u, 0u, 0u, 0u);
  // --- 1. Z_m and the tile weights of heads m = w, w + NW, ...
  for (int mm = w; kp > 0 && mm < G; mm += NW) {
    if (mm != w) {  // the first head's partials were loaded above
      if constexpr (PRE2) {  // and so were the second's
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          tm[j] = tm2[j];
          ts[j] = ts2[j];
        }
      } else {
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          const int t = lane + 64 * j;
          load_tile_part<CO>(tp + (int64_t)mm * m.n_tiles * 2, t, t < m.n_tiles, tm[j], ts[j]);
        }
      }
    }
    double mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < TJ; ++j)
      if (lane + 64 * j < n_tu) mx = fmax(mx, tm[j]);
    mx = wave_max_u(mx);
    // tile weight exp(M - Z) = exp(M - max) / sum_t S_t exp(M_t - max), S_t
    // being tile t's sum of exp(ell - M_t) (Eq. 9 with Z = max + log sum: no
    // logarithm is needed). exp(M - max) <= 1 is taken in fp32 from an fp64
    // hi + lo argument; the sum and the division stay fp64.
    float et[TJ];
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const bool on = lane + 64 * j < n_tu && tm[j] > -INFINITY;
      const double d = on ? tm[j] - mx : 0.0;
      const float dh = (float)d, dl = (float)(d - (double)dh);
      const float eh = expf(dh);
      et[j] = on ? fmaf(eh, dl, eh) : 0.f;
      s += ts[j] * (double)et[j];
    }
    s = wave_sum_u(s);
    const double inv = 1.0 / s;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int t = lane + 64 * j;
      if (t < n_tu) sw[t * G + mm] = (float)((double)et[j] * inv);
    }
  }
  __syncthreads();

  uint32_t gt = 0xFFFFFFFFu;  // keys above gt are taken
  uint32_t eqv = 0u;          // of the keys equal to eqv, the first eq_need are taken
  uint32_t eq_need = 0u;
  uint32_t key[R];
#pragma unroll
  for (int r = 0; r < R; ++r) key[r] = 0u;
  if (kp > 0) {
    // --- 2. keys
    float best[R];  // the block's score, rounded to fp32
    if constexpr (WIN) {
      // every window's group score (fp64 sum over the heads, rounded to
      // fp32) into LDS, four heads at a time: the first four heads' masses
      // were loaded at the start, later ones are loaded per batch
      double g[J4][4];
#pragma unroll
      for (int j = 0; j < J4; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) g[j][c] = 0.0;
      for (int h0 = 0; h0 < G; h0 += 4) {
        if (h0 > 0) {
#pragma unroll
          for (int hh = 0; hh < 4; ++hh)
#pragma unroll
            for (int j = 0; j < J4; ++j) {
              const int u = 4 * (tid + j * NT);
              wv[hh][j] = Mem<CO>::ld16(ev + (int64_t)min(h0 + hh, G - 1) * nbp,
                                        (uint32_t)(u < nu ? u : 0) * 4u);
            }
        }
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
          if (h0 + hh < G) {
#pragma unroll
            for (int j = 0; j < J4; ++j) {
              const int u = 4 * (tid + j * NT);
              const double wt = (double)sw[((u < nu ? u : 0) / kTileBlocks) * G + h0 + hh];
              g[j][0] = fma((double)__uint_as_float(wv[hh][j].x), wt, g[j][0]);
              g[j][1] = fma((double)__uint_as_float(wv[hh][j].y), wt, g[j][1]);
              g[j][2] = fma((double)__uint_as_float(wv[hh][j].z), wt, g[j][2]);
              g[j][3] = fma((double)__uint_as_float(wv[hh][j].w), wt, g[j][3]);
            }
          }
        }
      }
#pragma unroll
      for (int j = 0; j < J4; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int u = 4 * (tid + j * NT) + c;
          if (u < nu) wsc[u] = (float)g[j][c];
        }
      __syncthreads();
      // the windows sharing a token with block i (s divides B and C) are
      // i B / s - (C / s - 1) .. (i + 1) B / s - 1: a run of B / s + C / s - 1
      const int bpw = m.B / m.us, wpb = m.ul / m.us, nvb = bpw + wpb - 1;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int u0 = (i0 + r) * bpw - (wpb - 1);
        float bst = 0.f;
        for (int v = 0; v < nvb; ++v) {
          const int u = u0 + v;
          if (u >= 0 && u < nu) bst = fmaxf(bst, wsc[u]);
        }
        best[r] = bst;
      }
    } else {
    const int t = i0 / kTileBlocks;  // R <= 64: one tile per thread
    double sc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) sc[r] = 0.0;
    for (int h0 = 0; h0 < G; h0 += HC) {
      if (h0 > 0) {
#pragma unroll
        for (int h = 0; h < HC; ++h)
          load_run<R, CO, false>(ev, (int64_t)(h0 + h) * nbp + i0, h0 + h < G && i0 < nbp,
                                 e[h]);
      }
#pragma unroll
      for (int h = 0; h < HC; ++h) {
        if (h0 + h < G) {
          const double wv = t < n_tu ? (double)sw[t * G + h0 + h] : 0.0;
#pragma unroll
          for (int r = 0; r < R; ++r) sc[r] = fma((double)e[h][r], wv, sc[r]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) best[r] = (float)sc[r];
    }
    // candidates: real blocks that are not forced (bitwise tests: no branches)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = i0 + r;
      const bool cand = (i < nb) & (i >= m.n_sink) & (i < nb - m.n_local);
      key[r] = cand ? __float_as_uint(best[r]) + 1u : 0u;
    }
    // --- 3. the kp-th largest key, one digit per barrier. Every key is added
    // to its digit's bin (adding 0 when it is not in the running), so the
    // atomics need no per-lane branches; a wavefront none of whose keys is in
    // the running skips them.
    uint32_t prefix = 0u, need = (uint32_t)kp;
#pragma unroll
    for (int rd = 0; rd < 3; ++rd) {
      const int sh = 20 - 10 * rd;  // digits: bits 30..20, 19..10, 9..0
      const uint32_t msk = rd == 0 ? 0x7FFu : 0x3FFu;
      uint32_t* H = hist + (rd == 0 ? 0 : 1024 + 1024 * rd);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const bool in = (key[r] != 0u) & ((rd == 0) | ((key[r] >> (sh + 10)) == prefix));
        if (__ballot(in) != 0ull) atomicAdd(&H[(key[r] >> sh) & msk], in ? 1u : 0u);
      }
      __syncthreads();
      const RadixPick p = rd == 0 ? radix_pick<32>(H, need) : radix_pick<16>(H, need);
      if (rd == 0 && p.total < need) {  // fewer candidates than kp: take all
        gt = 0u;
        break;
      }
      need -= p.above;
      prefix = (prefix << 10) | p.digit;
      if (need == p.cnt) {  // the bin is taken whole
        const uint32_t lo = prefix << sh;
        gt = lo == 0u ? 0u : lo - 1u;
        break;
      }
      if (rd == 2) {  // prefix is now the kp-th key itself
        gt = prefix;
        eqv = prefix;
        eq_need = need;
      }
    }
  }

  // --- 4. ascending output. Each thread leaves one word of taken bits (keys
  // above the threshold, forced blocks) and one of tie bits (keys equal to
  // it) for its R blocks; wavefront 0 then reads them NT / 64 threads per
  // lane (lane order is block order), keeps the first eq_need ties in block
  // order, places every taken block by one wave-wide prefix sum and writes
  // the k entries out.
  uint32_t tkb = 0u, tqb = 0u;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = i0 + r;
    const bool forced = (i < nb) & ((i < m.n_sink) | (i >= nb - m.n_local));
    const bool tk = forced | ((key[r] != 0u) & (key[r] > gt));
    const bool tq = !tk & (eq_need > 0u) & (key[r] == eqv);
    tkb |= (tk ? 1u : 0u) << r;
    tqb |= (tq ? 1u : 0u) << r;
  }
  sm.bits[0][tid] = tkb;
  sm.bits[1][tid] = tqb;
  __syncthreads();
  if (w != 0) return;
  // lane l covers blocks l TPL R .. (l + 1) TPL R - 1 as LW words (thread
  // q of the lane at bit q R: R divides 32, so no thread straddles a word)
  constexpr int TPL = NT / 64;  // threads per lane
  constexpr int LW = (TPL * R + 31) / 32;
  uint32_t tkw[LW], tqw[LW];
#pragma unroll
  for (int u = 0; u < LW; ++u) tkw[u] = tqw[u] = 0u;
#pragma unroll
  for (int q = 0; q < TPL; ++q) {
    tkw[q * R / 32] |= sm.bits[0][lane * TPL + q] << (q * R % 32);
    tqw[q * R / 32] |= sm.bits[1][lane * TPL + q] << (q * R % 32);
  }
  uint32_t ct = 0u, cq = 0u;
#pragma unroll
  for (int u = 0; u < LW; ++u) {
    ct += (uint32_t)__builtin_popcount(tkw[u]);
    cq += (uint32_t)__builtin_popcount(tqw[u]);
  }
  if (eq_need > 0u) {  // the first eq_need ties, in block order
    const uint32_t before = wave_incl_scan_u32(cq) - cq;
    uint32_t left = eq_need > before ? eq_need - before : 0u;
#pragma unroll
    for (int u = 0; u < LW; ++u) {
      uint32_t x = tqw[u];
      while (x != 0u && left > 0u) {
        const uint32_t bit = x & (0u - x);
        tkw[u] |= bit;
        x ^= bit;
        --left;
        ++ct;
      }
    }
  }
  const uint32_t incl = wave_incl_scan_u32(ct);
  const int tot = (int)lane_u32(incl, 63);
  int pos = (int)(incl - ct);
#pragma unroll
  for (int u = 0; u < LW; ++u) {
    const int id0 = lane * TPL * R + 32 * u;
    for (uint32_t x = tkw[u]; x != 0u; x &= x - 1u) {
      sm.out[pos < k ? pos : SPLA_MAX_TOP_K] = id0 + __builtin_ctz(x);  // never past k
      ++pos;
    }
  }
  // (one wavefront's LDS accesses complete in order)
  for (int x = lane; x < k; x += 64) {
    const int v = x < tot ? sm.out[x] : -1;
    Mem<CO>::st(sel + x, v + SEL_OFF);
    if (so) so[x] = v;
  }
  if (lane == 0 && meta4) {
    Mem<CO>::st(meta4 + 0, tot < k ? tot : k);
    Mem<CO>::st(meta4 + 1, 0);
    Mem<CO>::st(meta4 + 2, L);
    Mem<CO>::st(meta4 + 3, tot);
  }
}

// ------------------------------------------------------------------------
// Two-stage selection for long sequences. One workgroup per (sequence, KV
// head) leaves most of the GPU idle when a head has tens of thousands of
// blocks and there are few heads (one sequence of 1M tokens: 8 workgroups).
// Instead, slices of kSliceBlocks blocks each take their own top-kp
// candidates (kp = k - forced blocks) under the same order as select_blocks
// (score descending, lower block id first), then the last slice of each
// head to finish picks the top kp among the candidates (the same launch:
// one kernel boundary less). Every block of the global top kp
// has fewer than kp blocks ahead of it in its own slice, so the candidates
// hold the whole top set and the result is select_blocks' exactly: the keys
// are computed with the same arithmetic in the same order.

constexpr int kSliceThreads = 256;
constexpr int kSliceR = kSliceBlocks / kSliceThreads;     // blocks per thread
constexpr int kSliceTiles = kSliceBlocks / kTileBlocks;   // 16 statistics tiles

// The kp-th largest of the keys held R per thread by the NT threads (0: not
// a candidate), found digit by digit as in select_blocks: keys above gt are
// taken and, of the keys equal to eqv, the first eq_need in thread order.
// Fewer than kp candidates: every candidate (gt = 0). hist: 4096 words,
// zeroed by the caller before a barrier.
template <int NT, int R>
__device__ __forceinline__ void radix_cut(const uint32_t (&key)[R], uint32_t kp, uint32_t* hist,
                                          uint32_t& gt, uint32_t& eqv, uint32_t& eq_need) {
  gt = 0xFFFFFFFFu;
  eqv = 0u;
  eq_need = 0u;
  uint32_t prefix = 0u, need = kp;
#pragma unroll
  for (int rd = 0; rd < 3; ++rd) {
    const int sh = 20 - 10 * rd;
    const uint32_t msk = rd == 0 ? 0x7FFu : 0x3FFu;
    uint32_t* H = hist + (rd == 0 ? 0 : 1024 + 1024 * rd);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const bool in = (key[r] != 0u) & ((rd == 0) | ((key[r] >> (sh + 10)) == prefix));
      if (__ballot(in) != 0ull) atomicAdd(&H[(key[r] >> sh) & msk], in ? 1u : 0u);
    }
    __syncthreads();
    const RadixPick p = rd == 0 ? radix_pick<32>(H, need) : radix_pick<16>(H, need);
    if (rd == 0 && p.total < need) {
      gt = 0u;
      return;
    }
    need -= p.above;
    prefix = (prefix << 10) | p.digit;
    if (need == p.cnt) {
      const uint32_t lo = prefix << sh;
      gt = lo == 0u ? 0u : lo - 1u;
      return;
    }
    if (rd == 2) {
      gt = prefix;
      eqv = prefix;
      eq_need = need;
    }
  }
}

// Slice sl (blocks sl kSliceBlocks ..) of sequence x KV head bh: the
// candidates' keys and ids, ascending by id, to ck / ci (k slots) and their
// count to *cn, written device-coherent (the pick runs in another workgroup
// of the same launch). Z_m comes from every tile partial of the head (TJ
// tiles per lane), exactly as select_blocks forms it; a wavefront with two
// heads loads the second head's partials with the first's. Nothing for a
// head whose blocks all fit in k (the pick selects them all). GM >= G: heads
// loaded.
template <int TJ, int GM>
__device__ void select_slice(const Dims& m, int bh, int sl, const int32_t* __restrict__ seq_lens,
                             const float* __restrict__ e_vals,
                             const double* __restrict__ tile_part, uint32_t* __restrict__ ck,
                             int32_t* __restrict__ ci, int32_t* __restrict__ cn, float* sw,
                             uint32_t* hist, uint32_t* scan) {
  constexpr int R = kSliceR, NW = kSliceThreads / 64;
  constexpr bool PRE2 = GM > NW && GM <= 2 * NW;  // heads w and w + NW preloaded
  const int G = m.group, k = m.k;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nbp = m.n_tiles * kTileBlocks;
  const int kp = k - m.n_sink - m.n_local;
  const int i0 = sl * kSliceBlocks + tid * R;
  const double* tp = tile_part + (int64_t)bh * m.n_tiles * G * 2;
  const float* ev = e_vals + (int64_t)bh * G * nbp;
  // loads first: this wave's first head's tile partials, this thread's masses
  double tm[TJ], ts[TJ];
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    const int t = lane + 64 * j;
    load_tile_part<false>(tp + (int64_t)(w < G ? w : 0) * m.n_tiles * 2, t,
                          w < G && t < m.n_tiles, tm[j], ts[j]);
  }
  double tm2[PRE2 ? TJ : 1], ts2[PRE2 ? TJ : 1];  // head w + NW
  if constexpr (PRE2) {
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int t = lane + 64 * j, w2 = w + NW;
      load_tile_part<false>(tp + (int64_t)(w2 < G ? w2 : 0) * m.n_tiles * 2, t,
                            w2 < G && t < m.n_tiles, tm2[j], ts2[j]);
    }
  }
  float e[GM][R];
#pragma unroll
  for (int h = 0; h < GM; ++h)
    load_run<R, false>(ev, (int64_t)(h < G ? h : 0) * nbp + i0, h < G && i0 < nbp, e[h]);
  const int L = min(max(seq_lens[bh / m.hkv], 0), m.cap);
  const int nb = (L + m.B - 1) / m.B;
  if (nb <= k || kp <= 0 || sl * kSliceBlocks >= nb) {  // uniform over the workgroup
    if (tid == 0) Mem<true>::st(cn, 0);
    return;
  }
  const int n_tu = (nb + kTileBlocks - 1) / kTileBlocks;
  for (int x = tid; x < 1024; x += kSliceThreads)
    reinterpret_cast<uint4*>(hist)[x] = make_uint4(0u, 0u, 0u, 0u);
  // --- Z_m of heads m = w, w + NW, ... and the weights of this slice's tiles
  const int jt = (sl * kSliceTiles) / 64, lt = (sl * kSliceTiles) % 64;  // slice tiles' lanes
  for (int mm = w; mm < G; mm += NW) {
    if (mm != w) {
      if constexpr (PRE2) {  // loaded at the start
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          tm[j] = tm2[j];
          ts[j] = ts2[j];
        }
      } else {
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          const int t = lane + 64 * j;
          load_tile_part<false>(tp + (int64_t)mm * m.n_tiles * 2, t, t < m.n_tiles, tm[j],
                                ts[j]);
        }
      }
    }
    double mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < TJ; ++j)
      if (lane + 64 * j < n_tu) mx = fmax(mx, tm[j]);
    mx = wave_max_u(mx);
    float et[TJ];
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const bool on = lane + 64 * j < n_tu && tm[j] > -INFINITY;
      const double d = on ? tm[j] - mx : 0.0;
      const float dh = (float)d, dl = (float)(d - (double)dh);
      const float eh = expf(dh);
      et[j] = on ? fmaf(eh, dl, eh) : 0.f;
      s += ts[j] * (double)et[j];
    }
    s = wave_sum_u(s);
    const double inv = 1.0 / s;
    float mine = 0.f;  // this lane's entry of register jt
#pragma unroll
    for (int j = 0; j < TJ; ++j) mine = j == jt ? et[j] : mine;
    const float etv = __shfl(mine, lt + (lane & (kSliceTiles - 1)), kWave);
    const int t = sl * kSliceTiles + lane;
    if (lane < kSliceTiles && t < n_tu) sw[lane * G + mm] = (float)((double)etv * inv);
  }
  __syncthreads();
  // --- keys (as select_blocks: fp64 sum over the heads in order)
  const int tt = (i0 - sl * kSliceBlocks) / kTileBlocks;  // this thread's tile in the slice
  const bool tile_on = sl * kSliceTiles + tt < n_tu;
  double sc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) sc[r] = 0.0;
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    if (h < G) {
      const double wv = tile_on ? (double)sw[tt * G + h] : 0.0;
#pragma unroll
      for (int r = 0; r < R; ++r) sc[r] = fma((double)e[h][r], wv, sc[r]);
    }
  }
  uint32_t key[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = i0 + r;
    const bool cand = (i < nb) & (i >= m.n_sink) & (i < nb - m.n_local);
    key[r] = cand ? __float_as_uint((float)sc[r]) + 1u : 0u;
  }
  uint32_t gt, eqv, eq_need;
  radix_cut<kSliceThreads, R>(key, (uint32_t)kp, hist, gt, eqv, eq_need);
  // --- the candidates, ascending by id: (taken above) | (ties) << 16, one scan
  bool tk[R], tq[R];
  uint32_t na = 0u, ne = 0u;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    tk[r] = (key[r] != 0u) & (key[r] > gt);
    tq[r] = !tk[r] & (eq_need > 0u) & (key[r] == eqv);
    na += tk[r] ? 1u : 0u;
    ne += tq[r] ? 1u : 0u;
  }
  uint32_t tot_p;
  const uint32_t before = block_excl_scan_u32<NW>(na | (ne << 16), scan, &tot_p);
  uint32_t a_run = before & 0xFFFFu, e_run = before >> 16;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t pg = a_run + (e_run < eq_need ? e_run : eq_need);
    const uint32_t pq = e_run < eq_need ? a_run + e_run : 0xFFFFFFFFu;
    const uint32_t pos = tk[r] ? pg : (tq[r] ? pq : 0xFFFFFFFFu);
    a_run += tk[r] ? 1u : 0u;
    e_run += tq[r] ? 1u : 0u;
    if (pos < (uint32_t)k) {
      Mem<true>::st(ck + pos, key[r]);
      Mem<true>::st(ci + pos, i0 + r);
    }
  }
  const uint32_t ta = tot_p & 0xFFFFu, te = tot_p >> 16;
  if (tid == 0) Mem<true>::st(cn, (int)(ta + (te < eq_need ? te : eq_need)));
}

// The pick of sequence x KV head bh from the candidates of its n_sl slices
// (k slots each, ck / ci / cn as select_slice wrote them): the kp largest,
// ties to the lower id, and the forced blocks, ascending, to sel[0 .. k)
// (-1 padded) and so (if not NULL); meta4 as select_blocks writes it. NT
// threads, R2 candidate slots per thread (NT R2 >= n_sl k); the slots in
// thread order are ascending by id. The candidates are read device-coherent
// (other workgroups of the same launch wrote them).
template <int R2, int NT>
__device__ void select_pick(const Dims& m, int bh, int n_sl, const int32_t* __restrict__ seq_lens,
                            const uint32_t* __restrict__ ck, const int32_t* __restrict__ ci,
                            const int32_t* __restrict__ cn, int32_t* __restrict__ sel,
                            int32_t* __restrict__ meta4, int32_t* __restrict__ so,
                            uint32_t* hist, uint32_t* scan, int32_t* out) {
  constexpr int NW = NT / 64;
  const int k = m.k, tid = threadIdx.x;
  const int kp = k - m.n_sink - m.n_local;
  uint32_t key[R2];
  int32_t id[R2];
#pragma unroll
  for (int r = 0; r < R2; ++r) {
    const int q = tid * R2 + r, s = q / k, j = q % k;
    const bool ok = s < n_sl;
    const int qq = ok ? q : 0;
    const int n = Mem<true>::ld(cn + (ok ? s : 0));
    const uint32_t kv = Mem<true>::ld(ck + qq);
    const int32_t iv = Mem<true>::ld(ci + qq);
    key[r] = ok && j < n ? kv : 0u;
    id[r] = iv;
  }
  const int L = min(max(seq_lens[bh / m.hkv], 0), m.cap);
  const int nb = (L + m.B - 1) / m.B;
  if (nb <= k) {  // every block (or none) is selected
    for (int x = tid; x < k; x += NT) {
      const int v = x < nb ? x : -1;
      sel[x] = v;
      if (so) so[x] = v;
    }
    if (tid == 0 && meta4) {
      meta4[0] = nb;
      meta4[1] = 1;
      meta4[2] = L;
      meta4[3] = 0;
    }
    return;
  }
  for (int x = tid; x < 1024; x += NT) reinterpret_cast<uint4*>(hist)[x] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  uint32_t gt = 0u, eqv = 0u, eq_need = 0u;
  if (kp > 0) radix_cut<NT, R2>(key, (uint32_t)kp, hist, gt, eqv, eq_need);
  bool tk[R2], tq[R2];
  uint32_t na = 0u, ne = 0u;
#pragma unroll
  for (int r = 0; r < R2; ++r) {
    tk[r] = (key[r] != 0u) & (key[r] > gt);
    tq[r] = !tk[r] & (eq_need > 0u) & (key[r] == eqv);
    na += tk[r] ? 1u : 0u;
    ne += tq[r] ? 1u : 0u;
  }
  uint32_t tot_p;
  const uint32_t before = block_excl_scan_u32<NW>(na | (ne << 16), scan, &tot_p);
  uint32_t a_run = before & 0xFFFFu, e_run = before >> 16;
  const int ns = m.n_sink;
#pragma unroll
  for (int r = 0; r < R2; ++r) {
    const uint32_t pg = a_run + (e_run < eq_need ? e_run : eq_need);
    const uint32_t pq = e_run < eq_need ? a_run + e_run : 0xFFFFFFFFu;
    const uint32_t pos = tk[r] ? pg : (tq[r] ? pq : 0xFFFFFFFFu);
    a_run += tk[r] ? 1u : 0u;
    e_run += tq[r] ? 1u : 0u;
    if (pos < (uint32_t)kp) out[ns + (int)pos] = id[r];
  }
  const uint32_t ta = tot_p & 0xFFFFu, te = tot_p >> 16;
  const int taken = (int)(ta + (te < eq_need ? te : eq_need));
  const int tot = ns + taken + m.n_local;  // <= k: taken <= kp
  if (tid < ns) out[tid] = tid;
  if (tid < m.n_local) out[ns + taken + tid] = nb - m.n_local + tid;
  __syncthreads();
  for (int x = tid; x < k; x += NT) {
    const int v = x < tot ? out[x] : -1;
    sel[x] = v;
    if (so) so[x] = v;
  }
  if (tid == 0 && meta4) {
    meta4[0] = tot;
    meta4[1] = 0;
    meta4[2] = L;
    meta4[3] = tot;
  }
}

}  // namespace spla
