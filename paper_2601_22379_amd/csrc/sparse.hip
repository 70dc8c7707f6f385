// Separate-kernel form of the fused pass over the selected blocks and of the
// merge (Secs. 2.2, 3.2, 3.3; the arithmetic is described in
// spla_sparse.h). bf16 with G <= 8 runs the matrix-core pass of
// spla_sparse.h; fp32 and larger groups use a VALU pass that writes the same
// records. The single-launch decode kernel (decode.hip) runs the same
// device functions.
#include "spla_device.h"
#include "spla_kernels.h"
#include "spla_select.h"
#include "spla_sparse.h"

namespace spla {

// ---------------------------------------------------------------- merge
// One single-wavefront workgroup per (sequence, KV head, query head), or per
// pair of query heads for groups of 5 or 6 (merge_halves): the records of a
// head are read by several compute units rather than one.
template <typename T, int D>
__global__ __launch_bounds__(64) void merge_kernel(
    Dims m, float eps, uint32_t flags, const float* __restrict__ gamma,
    const int32_t* __restrict__ meta, const float* __restrict__ part, int n_rec, int stride,
    T* __restrict__ out) {
  const int bh = blockIdx.x;
  if (merge_halves(m.group))  // uniform: two query heads per workgroup
    merge_head<T, D, false, false, true>(m, eps, flags, gamma, meta[bh * 4 + 1],
                                         meta[bh * 4 + 2], part + (int64_t)bh * n_rec * stride,
                                         n_rec, stride, out, bh, 2 * (int)blockIdx.y);
  else if (n_rec > 16)  // uniform: every record's loads in one batch (32 records)
    merge_head<T, D, false, false, false, 16>(m, eps, flags, gamma, meta[bh * 4 + 1],
                                              meta[bh * 4 + 2], part + (int64_t)bh * n_rec * stride,
                                              n_rec, stride, out, bh, (int)blockIdx.y);
  else
    merge_head<T, D, false>(m, eps, flags, gamma, meta[bh * 4 + 1], meta[bh * 4 + 2],
                            part + (int64_t)bh * n_rec * stride, n_rec, stride, out, bh,
                            (int)blockIdx.y);
}

// ------------------------------------------------------------ VALU pass
template <typename T, int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void sparse_valu_kernel(
    Dims m, float s, float eps, uint32_t flags, const T* __restrict__ kc,
    const T* __restrict__ vc, const T* __restrict__ q, const float* __restrict__ gamma,
    const float* __restrict__ S, const float* __restrict__ zbar,
    const int32_t* __restrict__ sel, const int32_t* __restrict__ meta, int stride,
    float* __restrict__ part, const int32_t* __restrict__ table) {
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
  const int nsel = min(max(meta[bh * 4 + 0], 0), m.k);
  const int L = min(max(meta[bh * 4 + 2], 0), m.cap);  // as the matrix-core pass clips it
  const int nb = (L + m.B - 1) / m.B;
  // workgroup split: sub-tile sub0 of selection entry p0 (B / 32 sub-tiles
  // per block), so a block's sub-tiles run side by side
  const int spb = m.B / kSubTokens;
  const int p0 = split / spb, sub0 = split % spb, p1 = min(p0 + 1, nsel);
  // this workgroup's rows of S_bar and z_bar for the global linear term: the
  // first kLinPre rows loaded now (they land while the blocks are processed),
  // any further ones at the end, kLinPre rows per batch of loads
  constexpr int kLinPre = 8;
  int row0, nrows;
  lin_rows(D, split, gridDim.x, &row0, &nrows);
  const int rend = row0 + nrows;
  const int cS = tid % D;  // the coordinate of every (head, coordinate) output of this thread
  const float* Sb = S + (int64_t)bh * D * D + cS;
  const float* zb = zbar + (int64_t)bh * D;
  float sv[kLinPre], zv[kLinPre];
#pragma unroll
  for (int u = 0; u < kLinPre; ++u) {
    const int j = row0 + u < rend ? row0 + u : 0;
    sv[u] = Sb[(int64_t)j * D];
    zv[u] = zb[j];
  }

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
    // the block's slot: per-sequence cache, or its page of a paged pool (an
    // entry out of range reads page 0)
    int64_t slot = (int64_t)bh * m.nb_cap + blk;
    if (table) {
      const int pg = block_page(m, table, bh, blk);
      slot = (int64_t)(pg < 0 ? 0 : pg) * m.hkv + h;
    }
    for (int sub = sub0; sub == sub0 && sub * kSubTokens < n_i; ++sub) {
      const int tb0 = sub * kSubTokens;
      const int nt = min(kSubTokens, n_i - sub * kSubTokens);
      // every load of the sub-tile issued before any is used (rows past nt
      // read the sub-tile's first row and are masked)
      constexpr int NE = kSubTokens * D / 256;
      float kx[NE], vx[NE];
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        const int e = tid + 256 * i;
        const int row = e / D, col = e % D, c2 = e / kSubTokens, r2 = e % kSubTokens;
        kx[i] = Elem<T>::load(kc, k_off_slot(m, slot, tb0 + (row < nt ? row : 0), col));
        vx[i] = Elem<T>::load(vc, v_off_slot(m, slot, tb0 + (r2 < nt ? r2 : 0), c2));
      }
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        const int e = tid + 256 * i;
        const int row = e / D, col = e % D, c2 = e / kSubTokens, r2 = e % kSubTokens;
        sK[row][col] = row < nt ? kx[i] : 0.f;
        sV[c2][r2] = r2 < nt ? vx[i] : 0.f;
      }
      __syncthreads();
      // phi(k) rows: wavefront w takes rows 8 w .. 8 w + 7 at once, eight
      // lanes per row (lane 8 r + u: coordinates u D / 8 ..), the softmax's
      // max and sum over the row's lanes by lane swaps
      {
        static_assert(kSubTokens == 32, "four wavefronts of eight rows");
        constexpr int DE = D / 8;
        const int row = 8 * w + (lane >> 3), c0 = DE * (lane & 7);
        float x[DE];
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < DE; ++e) {
          x[e] = sK[row][c0 + e];
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
        const float inv = row < nt ? 1.0f / sum : 0.f;
#pragma unroll
        for (int e = 0; e < DE; ++e) sE[row][c0 + e] = x[e] * inv;
      }
      __syncthreads();
      // logits and linear weights: eight lanes per (head, token), each over
      // D / 8 coordinates, added by lane swaps; G passes of 32 products
      for (int e0 = 0; e0 < G * kSubTokens; e0 += 32) {
        constexpr int DE = D / 8;
        const int e = e0 + (tid >> 3), c0 = DE * (tid & 7);
        const int mm = e / kSubTokens, t = e % kSubTokens;
        float a = 0.f, wl = 0.f;
#pragma unroll 8
        for (int j = 0; j < DE; ++j) {
          a = fmaf(sq[mm][c0 + j], sK[t][c0 + j], a);
          wl = fmaf(sphq[mm][c0 + j], sE[t][c0 + j], wl);
        }
        a += __shfl_xor(a, 1, 64);
        wl += __shfl_xor(wl, 1, 64);
        a += __shfl_xor(a, 2, 64);
        wl += __shfl_xor(wl, 2, 64);
        a += __shfl_xor(a, 4, 64);
        wl += __shfl_xor(wl, 4, 64);
        if ((tid & 7) == 0) {
          sP[mm][t] = t < nt ? a : -INFINITY;
          sW[mm][t] = t < nt ? wl : 0.f;
        }
      }
      __syncthreads();
      // online softmax bookkeeping: wavefront w takes heads w, w + 4, ..., lane
      // t < kSubTokens token t
      static_assert(kSubTokens <= 64, "one token per lane");
      for (int mm = w; mm < G; mm += 4) {
        const bool on = lane < nt;
        const float lg = on ? sP[mm][lane] : -INFINITY;
        const float mx = fmaxf(s_m[mm], wave_max(lg));
        const float alpha = expf(s_m[mm] - mx);
        const float pv = on ? expf(lg - mx) : 0.f;
        const float l = s_l[mm] * alpha + wave_sum(pv);
        const float zw = s_zw[mm] + wave_sum(lane < kSubTokens ? sW[mm][lane] : 0.f);
        if (lane < kSubTokens) sP[mm][lane] = pv;
        if (lane == 0) {
          s_m[mm] = mx;
          s_l[mm] = l;
          s_alpha[mm] = alpha;
          s_zw[mm] = zw;
        }
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < PER; ++r) {
        const int idx = tid + 256 * r;
        if (idx < G * D) {
          const int mm = idx / D, c = idx % D;
          float a = acc[r] * s_alpha[mm], aw = accw[r];
          // tokens past nt add exact zeros (p, w and v are 0 there)
#pragma unroll 8
          for (int t = 0; t < kSubTokens; ++t) {
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
  // this workgroup's rows of the global linear term, minus its selected
  // terms (rows in ascending order)
  float ob[PER], zq = 0.f;
#pragma unroll
  for (int r = 0; r < PER; ++r) ob[r] = 0.f;
  const int gz = tid < G ? tid : 0;
  auto add_rows = [&](int j0, const float (&v)[kLinPre], const float (&z)[kLinPre]) {
#pragma unroll
    for (int u = 0; u < kLinPre; ++u) {
      const bool ok = j0 + u < rend;
      const int jc = ok ? j0 + u : 0;
#pragma unroll
      for (int r = 0; r < PER; ++r) {
        const int mm = (tid + 256 * r) / D;
        ob[r] = fmaf(sphq[mm < MG ? mm : 0][jc], ok ? v[u] : 0.f, ob[r]);
      }
      zq = fmaf(sphq[gz][jc], ok ? z[u] : 0.f, zq);
    }
  };
  add_rows(row0, sv, zv);
  for (int j0 = row0 + kLinPre; j0 < rend; j0 += kLinPre) {
#pragma unroll
    for (int u = 0; u < kLinPre; ++u) {
      const int j = j0 + u < rend ? j0 + u : row0;
      sv[u] = Sb[(int64_t)j * D];
      zv[u] = zb[j];
    }
    add_rows(j0, sv, zv);
  }
  float* rec = part + ((int64_t)bh * gridDim.x + split) * stride;
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int idx = tid + 256 * r;
    if (idx < G * D) {
      const int mm = idx / D, c = idx % D;
      rec[kPartHead + mm * D + c] = acc[r];
      rec[kPartHead + (G + mm) * D + c] = ob[r] - accw[r];
    }
  }
  if (tid < G) {
    rec[tid] = s_m[tid];
    rec[16 + tid] = s_l[tid];
    rec[32 + tid] = zq - s_zw[tid];
  }
}

// ------------------------------------------------------------ MFMA pass
// R > 0: the workgroup first selects the blocks of its (sequence, KV head)
// itself (select_blocks with 256 threads, R blocks per thread; every
// workgroup of the pair computes the same selection), so no selection kernel
// runs; workgroup 0 publishes the selection and the meta words. R = 0: the
// selection comes from the selection kernel.
// STEP (R = 0 only): first apply the step's rank-one update to this
// workgroup's rows of S_bar (step_rank1), as the single-launch step does.
// GC: accumulator columns per kind (>= G). The selection's LDS (R > 0) lies
// over the accumulators, which sparse_body writes only after the selection.
template <int D, int BLK, int R, int GC, bool STEP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(GC <= 4 ? 3 : 2)))
void sparse_mfma_kernel(
    Dims m, float s, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const bf16_t* __restrict__ q, float* __restrict__ S, float* __restrict__ zbar,
    const int32_t* __restrict__ sel, int32_t* __restrict__ meta, int stride,
    float* __restrict__ part, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ e_vals, const double* __restrict__ tile_part,
    int32_t* __restrict__ sel_out, const int32_t* __restrict__ table,
    const bf16_t* __restrict__ k_step = nullptr, const bf16_t* __restrict__ v_step = nullptr,
    const int32_t* __restrict__ appended = nullptr) {
  constexpr int SWN = R > 0 ? kTileBlocks * 8 : 4;  // tile weights: <= 64 tiles x 8 heads
  using SpSm = SparseSmem<D, GC>;
  using SeSm = SelectSmem<256, SWN>;
  constexpr size_t kLds = R > 0 && SpSm::kOverlay + sizeof(SeSm) > sizeof(SpSm)
                              ? SpSm::kOverlay + sizeof(SeSm) : sizeof(SpSm);
  static_assert(SpSm::kOverlay % 16 == 0, "overlay alignment");
  __shared__ __align__(16) unsigned char lds[kLds];
  SpSm& sm = *reinterpret_cast<SpSm*>(lds);
  SeSm& ssm = *reinterpret_cast<SeSm*>(lds + SpSm::kOverlay);
  __shared__ int32_t s_sel[R > 0 ? SPLA_MAX_TOP_K : 1];
  __shared__ int32_t s_meta[4];
  const int bh = blockIdx.y;
  const int x = (int)blockIdx.x;
  SparseRegs r;
  if constexpr (R == 0) {
    // the selection is known at the start: the step's keys and values are
    // loaded first, behind only the query and S_bar loads, so that their
    // latency overlaps the prologue's arithmetic (loads complete in order)
    const int e = sparse_step_entry<BLK>(x);
    const int blk_sel = e < m.k ? sel[(int64_t)bh * m.k + e] : -1;
    int L = meta[bh * 4 + 2];
    uint4 raw[D / 32];
    sparse_prologue_load<D, GC>(m, q, S, zbar, bh, x, (int)gridDim.x, r, raw);
    StepIn<D> sin;
    if constexpr (STEP) step_load<D>(m, k_step, v_step, appended, bh, sin);
    SparseKV<D> kv;
    const int blk = sparse_step_block<BLK>(m, blk_sel, L, x, &kv.n_valid);
    sparse_load<D, BLK>(m, kc, vc, blk < 0 ? 0 : blk, bh, x, table, kv);
    sparse_prologue_finish<D, GC>(m, raw, sm);
    if constexpr (STEP) step_apply<D>(m, sin, S, zbar, bh, r);
    sparse_linear<D, GC>(m, S, bh, r, sm);
    floatx4 acc_o[D / 16];
#pragma unroll
    for (int t = 0; t < D / 16; ++t) acc_o[t] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    if (kv.n_valid > 0) sparse_mma<D, GC>(s, kv, sm, acc_o, m_run, l_run);
    sparse_record<D, false, GC>(m, acc_o, m_run, l_run, bh, x, (int)gridDim.x, r, sm, part,
                                stride, -1);
  } else {  // every workgroup makes its head's selection itself
    sparse_prologue<D, GC>(m, q, S, zbar, bh, x, (int)gridDim.x, r, sm);
    sparse_linear<D, GC>(m, S, bh, r, sm);
    select_blocks<256, R, SWN, false, 0, false, GC>(
        m, bh, seq_lens[bh / m.hkv], e_vals, tile_part, ssm, s_sel, s_meta,
        x == 0 && sel_out ? sel_out + (int64_t)bh * m.k : nullptr);
    __syncthreads();
    if (x == 0 && threadIdx.x < 4) meta[bh * 4 + threadIdx.x] = s_meta[threadIdx.x];
    const int e = sparse_step_entry<BLK>(x);
    sparse_body<D, BLK, false, GC>(m, s, kc, vc, e < m.k ? s_sel[e] : -1, s_meta[2], bh, x,
                                   (int)gridDim.x, r, sm, part, stride, table);
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
                     ws.part_stride, (float*)(base + ws.part),
                     m.pages > 0 ? c.block_table : nullptr);
}

// Blocks per thread of the in-workgroup selection (0: use the selection
// kernel). Every workgroup repeats the selection of its (sequence, KV head),
// which pays only while the grid is small (about two workgroups per compute
// unit) and the block count is at most 4096.
static int sparse_select_r(const Dims& m, bool step) {
  if (step || !use_mfma_sparse(m) || m.nb_cap > 256 * 16 || windowed(m)) return 0;
  const DecodeWs ws = decode_ws_layout(m);
  if ((int64_t)ws.n_wg * m.bh > 2 * (int64_t)compute_units()) return 0;
  const int per = (int)ceil_div(m.nb_cap, 256);
  return per <= 2 ? 2 : (per <= 4 ? 4 : (per <= 8 ? 8 : 16));
}

bool sparse_selects(const Dims& m, bool step) { return sparse_select_r(m, step) > 0; }

template <int D, int BLK, int R, bool STEP>
static void mfma_dbr(const Dims& m, float s, const spla_cache& c, const void* q,
                     int32_t* sel_out, const DecodeWs& ws, char* base, hipStream_t st,
                     const void* k_step, const void* v_step) {
  auto kern = m.group <= 4 ? sparse_mfma_kernel<D, BLK, R, 4, STEP>
                           : sparse_mfma_kernel<D, BLK, R, 8, STEP>;
  hipLaunchKernelGGL(kern, dim3(ws.n_wg, m.bh), dim3(256), 0, st,
                     m, s, (const bf16_t*)c.k_cache, (const bf16_t*)c.v_cache, (const bf16_t*)q,
                     c.lin_state, c.lin_norm, (const int32_t*)(base + ws.sel),
                     (int32_t*)(base + ws.meta), ws.part_stride, (float*)(base + ws.part),
                     c.seq_lens, (const float*)(base + ws.e_vals),
                     (const double*)(base + ws.tile_part), sel_out,
                     m.pages > 0 ? c.block_table : nullptr, (const bf16_t*)k_step,
                     (const bf16_t*)v_step, (const int32_t*)(base + ws.appended));
}

template <int D, int BLK>
static void mfma_db(const Dims& m, float s, const spla_cache& c, const void* q, int32_t* sel_out,
                    const DecodeWs& ws, char* base, hipStream_t st, const void* k_step,
                    const void* v_step) {
  if (k_step) {
    mfma_dbr<D, BLK, 0, true>(m, s, c, q, sel_out, ws, base, st, k_step, v_step);
    return;
  }
  switch (sparse_select_r(m, false)) {
    case 2: mfma_dbr<D, BLK, 2, false>(m, s, c, q, sel_out, ws, base, st, nullptr, nullptr); break;
    case 4: mfma_dbr<D, BLK, 4, false>(m, s, c, q, sel_out, ws, base, st, nullptr, nullptr); break;
    case 8: mfma_dbr<D, BLK, 8, false>(m, s, c, q, sel_out, ws, base, st, nullptr, nullptr); break;
    case 16: mfma_dbr<D, BLK, 16, false>(m, s, c, q, sel_out, ws, base, st, nullptr, nullptr); break;
    default: mfma_dbr<D, BLK, 0, false>(m, s, c, q, sel_out, ws, base, st, nullptr, nullptr); break;
  }
}

template <int D>
static void mfma_d(const Dims& m, float s, const spla_cache& c, const void* q, int32_t* sel_out,
                   const DecodeWs& ws, char* base, hipStream_t st, const void* k_step,
                   const void* v_step) {
  if (m.B == 32) mfma_db<D, 32>(m, s, c, q, sel_out, ws, base, st, k_step, v_step);
  else if (m.B == 64) mfma_db<D, 64>(m, s, c, q, sel_out, ws, base, st, k_step, v_step);
  else mfma_db<D, 128>(m, s, c, q, sel_out, ws, base, st, k_step, v_step);
}

template <typename T, int D>
static void merge_td(const Dims& m, const spla_config& cfg, const float* gamma, void* out,
                     const DecodeWs& ws, char* base, hipStream_t st) {
  const int gy = merge_halves(m.group) ? (m.group + 1) / 2 : m.group;
  hipLaunchKernelGGL((merge_kernel<T, D>), dim3(m.bh, gy), dim3(64), 0, st, m, cfg.rms_eps,
                     cfg.flags, gamma, (const int32_t*)(base + ws.meta),
                     (const float*)(base + ws.part), ws.n_wg, ws.part_stride, (T*)out);
}

hipError_t launch_sparse(const Dims& m, const spla_config& cfg, const spla_cache& c,
                         const void* q, const float* gamma, void* out, int32_t* sel_out,
                         const DecodeWs& ws, char* base, hipStream_t st, const void* k_step,
                         const void* v_step) {
  const float s = cfg.softmax_scale > 0.f ? cfg.softmax_scale : (float)(1.0 / sqrt((double)m.d));
  if (k_step && !step_fusable(m)) return hipErrorInvalidValue;
  if (use_mfma_sparse(m)) {
    if (m.d == 64) mfma_d<64>(m, s, c, q, sel_out, ws, base, st, k_step, v_step);
    else mfma_d<128>(m, s, c, q, sel_out, ws, base, st, k_step, v_step);
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
