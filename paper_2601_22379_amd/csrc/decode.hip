// Single-launch decode step: block scoring, selection, the fused pass over
// the selected blocks and the merge of every (sequence, KV head) in one
// kernel, so that selections and the reads of the selected keys and values of
// the heads scored first overlap the statistics stream of the others.
//
// One workgroup per item, in workgroup-index order:
//   score items   kTilesPerItem 64-block statistics tiles of one (sequence,
//                 KV head) (score_items), in (sequence, KV head) order. The
//                 workgroup that finishes a head's last item runs the head's
//                 selection (select_blocks), which publishes every selected
//                 block as its own word (block + 2, never 0).
//   sparse items  one per share x of the fused pass (sparse_body) of each
//                 (sequence, KV head), in (sequence, KV head) order rotated
//                 to start with the heads scored last (sparse_rotation): one
//                 lane polls the words of the workgroup's blocks (one 16-byte
//                 chunk), and clears them once read. The workgroup that
//                 writes a head's last record merges the head's records into
//                 its output rows.
// Only sparse items wait (for their head's selection), and only for score
// items, which have smaller indices and never wait; workgroups start in index
// order on each XCD, so every score item starts, and every wait ends. Waits
// are bounded all the same (kSpinLimit polls); a wait that gives up sets
// SPLA_DEVERR_SYNC.
//
// Data published by one workgroup and read by another (e_vals, tile_part,
// the selection words, the records) is written and read with
// device-coherent accesses (Mem<true>: agent-scope atomic loads and stores,
// and sc1 buffer loads, which bypass the per-XCD L2 caches); the producer
// waits for its stores to complete before the word that announces them is
// updated. No cache-wide writeback or invalidation (agent-scope fences) is
// used: on this GPU they act on a whole L2 and cost far more than the
// kilobytes moved. The counters are agent-scope atomics, each alone in a
// 128-byte line; the selection words of a head share lines (sync_layout). Each call leaves them all at zero: a head's selecting
// workgroup resets its item counter, its sparse workgroups their selection
// words, and its merging workgroup its record counter.
#include "spla_kernels.h"
#include "spla_score.h"
#include "spla_select.h"
#include "spla_sparse.h"

namespace spla {

constexpr int kSpinLimit = 1 << 20;  // polls of a wait (about a second)
constexpr int kTilesPerItem = 1;  // statistics tiles per score item (two measured slower)

struct FusedArgs {
  Dims m;
  const float* stats;
  const int32_t* seq_lens;
  const bf16_t* q;
  const bf16_t* kc;
  const bf16_t* vc;
  const float* S;
  const float* zbar;
  const float* gamma;
  bf16_t* out;
  int32_t* sel_out;    // caller's selection output or NULL
  int32_t* err_flags;  // caller's error word or NULL
  float* e_vals;
  double* tile_part;
  int32_t* sel;
  int32_t* meta;
  float* part;
  int32_t* sync;
  SyncLayout y;
  double s_score;
  float s;
  float eps;
  uint32_t flags;
  int first_order;
  int n_si;     // score items per (sequence, KV head)
  int n_wg;     // sparse items per (sequence, KV head)
  int rot;      // the sparse items start with (sequence, KV head) rot (sparse_rotation)
  int stride;   // floats per record
  const int32_t* table;  // block table of a paged K/V pool, or NULL
  // fused step: the token appended to each (sequence, KV head) and how many
  // tokens each sequence received (0 at capacity), or NULL
  const bf16_t* k_step;
  const bf16_t* v_step;
  const int32_t* appended;
};


__device__ __forceinline__ void report_sync_error(const FusedArgs& a) {
  atomic_add_agent(a.sync + a.y.err, 1);
  if (a.err_flags) atomicOr(a.err_flags, (int)SPLA_DEVERR_SYNC);
}


// Built for three waves per SIMD (at most 168 registers per lane; measured
// faster than two, and than four with its 128-register budget, at the 128K
// workload). A launch whose items would not all be resident at three but are
// at four (32K: 1024 items) takes the four-wave build: then no sparse item
// starts after its selection (27.3 -> 25.2 us).
constexpr int kDecodeWaves = 3;

// R: blocks per thread of the selection (256 R >= blocks per sequence).
// STEP: the sparse items first apply the step's rank-one update (step_rank1).
// WAVES: waves per SIMD the kernel is built for (3 or 4).
template <int G, int BLK, int R, bool STEP, int WAVES>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WAVES, WAVES)))
void decode_kernel(FusedArgs a) {
  constexpr int D = 128;
  constexpr int SWN = 4 * R * G;  // tile weights: n_tiles <= 4 R
  constexpr int GC = G <= 4 ? 4 : (G <= 6 ? 6 : 8);  // accumulator columns per kind
  __shared__ union {
    ScoreSmem<G> sc;
    SelectSmem<256, SWN> se;
    SparseSmem<D, GC> sp;
  } sm;
  __shared__ int s_flag;
  __shared__ int s_words[4];
  const Dims& m = a.m;
  const SyncLayout& y = a.y;
  int32_t* sy = a.sync;
  const int tid = threadIdx.x;
  const int n_score = m.bh * a.n_si;
  if ((int)blockIdx.x < n_score) {
    // ---------------------------------------------------------- score item
    const int t = (int)blockIdx.x;
    const int bh = t / a.n_si, i = t % a.n_si;
    const int L = a.seq_lens[bh / m.hkv];  // for the selection; loaded long before it is used
    score_items<G, bf16_t, D, true, kTilesPerItem>(
        m, a.stats, a.seq_lens, a.q, a.s_score, a.first_order,
        bh * m.n_tiles + i * kTilesPerItem, a.e_vals, a.tile_part, sm.sc);
    int32_t* done = sy + y.items_done + (int64_t)bh * kSyncLine;
    if (!arrive_last(done, a.n_si, &s_flag)) return;
    // the selection is on the path to the head's output: its wavefronts go
    // ahead of the score items that share their SIMDs
    __builtin_amdgcn_s_setprio(3);
    select_blocks<256, R, SWN, true, 2, false, G, true>(m, bh, L, a.e_vals, a.tile_part, sm.se,
                                        sy + y.sel_ready + (int64_t)bh * m.k, nullptr,
                                        a.sel_out ? a.sel_out + (int64_t)bh * m.k : nullptr);
    // reset last: vmcnt counts stores, so an earlier store would hold up
    // every wait on the selection's loads until it completed
    if (tid == 0) store_agent(done, 0);
    return;
  }
  // ------------------------------------------------------------ sparse item
  const int j = (int)blockIdx.x - n_score;
  const int bh = (j / a.n_wg + a.rot) % m.bh, x = j % a.n_wg;
  // the workgroup's selection entries (one per step: 4x / (BLK/32) .. of its
  // four steps, 4 / (BLK/32) of them) are polled by lane 0 of wavefront 0
  // alone, as the 16-byte chunk holding them, the first time before the
  // prologue's loads (a workgroup that starts after its selection then has
  // them when the prologue is done); one poller per workgroup keeps the
  // polling traffic on the line the selection writes low
  constexpr int CPB = BLK / 32;
  constexpr int NE = CPB >= 4 ? 1 : 4 / CPB;  // entries of one workgroup
  const int e0 = (x * kSparseWaves) / CPB;
  const int32_t* words = sy + y.sel_ready + (int64_t)bh * m.k;
  const uint32_t chunk = (uint32_t)(e0 / 4) * 16u;  // the area is padded for the last row
  const bool poller = tid == 0;
  auto ready = [&](const uint4& c) {
    bool ok = true;
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int e = e0 + i, c4 = e & 3;
      const uint32_t v = c4 == 0 ? c.x : (c4 == 1 ? c.y : (c4 == 2 ? c.z : c.w));
      ok = ok && (e >= m.k || v != 0u);
    }
    return ok;
  };
  uint4 cv = make_uint4(1u, 1u, 1u, 1u);
  if (poller) cv = Mem<true>::ld16(words, chunk);
  const int L = min(max(a.seq_lens[bh / m.hkv], 0), m.cap);  // not produced in this launch
  SparseRegs r;
  sparse_prologue<D, GC>(m, a.q, a.S, a.zbar, bh, x, a.n_wg, r, sm.sp);
  if constexpr (STEP)
    step_rank1<D>(m, a.k_step, a.v_step, a.appended, const_cast<float*>(a.S),
                  const_cast<float*>(a.zbar), bh, r);
  sparse_linear<D, GC>(m, a.S, bh, r, sm.sp);
  if (poller && !ready(cv)) {
    // three polls in flight: each turn issues one and takes the oldest, so
    // a published word is seen about one memory round trip after it lands
    // (one poll at a time would add up to another round trip); unrolled by
    // three so that no register of a poll in flight is copied (a copy
    // would wait for it)
    uint4 p1 = Mem<true>::ld16(words, chunk);
    __builtin_amdgcn_s_sleep(2);
    uint4 p2 = Mem<true>::ld16(words, chunk);
    uint4 p3;
    bool ok = false;
    for (int n = 0; n < kSpinLimit; n += 3) {
      __builtin_amdgcn_s_sleep(2);
      p3 = Mem<true>::ld16(words, chunk);
      if (ready(p1)) { cv = p1; ok = true; break; }
      __builtin_amdgcn_s_sleep(2);
      p1 = Mem<true>::ld16(words, chunk);
      if (ready(p2)) { cv = p2; ok = true; break; }
      __builtin_amdgcn_s_sleep(2);
      p2 = Mem<true>::ld16(words, chunk);
      if (ready(p3)) { cv = p3; ok = true; break; }
    }
    if (!ok) {
      report_sync_error(a);
      cv = make_uint4(0u, 0u, 0u, 0u);  // entries of a wait that gave up: no block
    }
  }
  if (poller) {
    const uint32_t vals[4] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
    for (int w = 0; w < kSparseWaves; ++w) s_words[w] = (int)vals[((x * kSparseWaves + w) / CPB) & 3];
  }
  __syncthreads();
  const int step = sparse_step_entry<BLK>(x);
  const int v = step < m.k ? s_words[tid >> 6] : 1;  // 0 only after a wait that gave up
  const int blk_sel = __builtin_amdgcn_readfirstlane(v) - 2;
  sparse_body<D, BLK, true, GC>(m, a.s, a.kc, a.vc, blk_sel, L, bh, x, a.n_wg, r, sm.sp, a.part,
                                a.stride, a.table);
  if (poller) {  // the workgroup's entries, read by it only
#pragma unroll
    for (int i = 0; i < NE; ++i)
      if (e0 + i < m.k) store_agent(const_cast<int32_t*>(words) + e0 + i, 0);
  }
  int32_t* recs = sy + y.recs_done + (int64_t)bh * kSyncLine;
  if (!arrive_last(recs, a.n_wg, &s_flag)) return;
  const int nb = (L + BLK - 1) / BLK;
  const int all_sel = nb <= m.k;
  const float* rec = a.part + (int64_t)bh * a.n_wg * a.stride;
  if constexpr (G > 4) {  // two query heads per wavefront (merge_halves)
    const int g = 2 * (tid >> 6);
    if (g < G)
      merge_head<bf16_t, D, true, false, true>(m, a.eps, a.flags, a.gamma, all_sel, L, rec,
                                               a.n_wg, a.stride, a.out, bh, g);
  } else {
    for (int g = tid >> 6; g < G; g += 4)
      merge_head<bf16_t, D, true>(m, a.eps, a.flags, a.gamma, all_sel, L, rec, a.n_wg, a.stride,
                                  a.out, bh, g);
  }
  if (tid == 0) store_agent(recs, 0);  // last, as for the item counter
}

// The (sequence, KV head) the sparse items start with: the heads whose
// statistics land last come first, so that their items are resident, with
// their prologue done, when their selections are published. With more
// items than slots the score items of heads slots / n_si .. run in the
// second round of slots and land last; with every item resident the loads
// complete in about issue order and the second half of the heads lands
// last. Measured against the plain order: 128K 29.83 -> 29.6 us (24 of 32
// heads), 32K 24.14 -> 23.29 us (32 of 64), G = 5 unchanged.
static int sparse_rotation(const FusedArgs& a, int slots) {
  const int grid = a.m.bh * (a.n_si + a.n_wg);
  return grid > slots ? (slots / a.n_si) % a.m.bh : a.m.bh / 2;
}

template <int G, int BLK, int R>
static void decode_gbr(const FusedArgs& a0, hipStream_t st) {
  const int grid = a0.m.bh * (a0.n_si + a0.n_wg);
  const int cus = compute_units();  // one workgroup per wave of each SIMD
  const bool four = !a0.appended && grid > kDecodeWaves * cus && grid <= 4 * cus;
  FusedArgs a = a0;
  a.rot = sparse_rotation(a, (four ? 4 : kDecodeWaves) * cus);
  if (a.appended)
    hipLaunchKernelGGL((decode_kernel<G, BLK, R, true, kDecodeWaves>), dim3((unsigned)grid),
                       dim3(256), 0, st, a);
  else if (four)
    hipLaunchKernelGGL((decode_kernel<G, BLK, R, false, 4>), dim3((unsigned)grid), dim3(256), 0,
                       st, a);
  else
    hipLaunchKernelGGL((decode_kernel<G, BLK, R, false, kDecodeWaves>), dim3((unsigned)grid),
                       dim3(256), 0, st, a);
}

template <int G, int R>
static void decode_gr(const FusedArgs& a, hipStream_t st) {
  if (a.m.B == 32) decode_gbr<G, 32, R>(a, st);
  else if (a.m.B == 64) decode_gbr<G, 64, R>(a, st);
  else decode_gbr<G, 128, R>(a, st);
}

template <int G>
static void decode_g(const FusedArgs& a, hipStream_t st) {
  if (a.m.nb_cap <= 256 * 8) decode_gr<G, 8>(a, st);
  else decode_gr<G, 32>(a, st);
}

static hipError_t decode_fused(const Dims& m, const spla_config& cfg, const spla_cache& c,
                               const void* q, const float* gamma, void* out, int32_t* sel_out,
                               const DecodeWs& ws, char* base, hipStream_t st,
                               const void* k_step, const void* v_step) {
  FusedArgs a;
  a.m = m;
  a.stats = c.blk_stats;
  a.seq_lens = c.seq_lens;
  a.q = (const bf16_t*)q;
  a.kc = (const bf16_t*)c.k_cache;
  a.vc = (const bf16_t*)c.v_cache;
  a.S = c.lin_state;
  a.zbar = c.lin_norm;
  a.gamma = gamma;
  a.out = (bf16_t*)out;
  a.sel_out = sel_out;
  a.err_flags = c.err_flags;
  a.e_vals = (float*)(base + ws.e_vals);
  a.tile_part = (double*)(base + ws.tile_part);
  a.sel = (int32_t*)(base + ws.sel);
  a.meta = (int32_t*)(base + ws.meta);
  a.part = (float*)(base + ws.part);
  a.sync = (int32_t*)(base + ws.sync);
  a.y = sync_layout(m);
  a.s_score = cfg.softmax_scale > 0.f ? (double)cfg.softmax_scale : 1.0 / sqrt((double)m.d);
  a.s = cfg.softmax_scale > 0.f ? cfg.softmax_scale : (float)(1.0 / sqrt((double)m.d));
  a.eps = cfg.rms_eps;
  a.flags = cfg.flags;
  a.first_order = (cfg.flags & SPLA_FLAG_FIRST_ORDER) != 0;
  a.n_si = (int)ceil_div(m.n_tiles, kTilesPerItem);
  a.n_wg = ws.n_wg;
  a.stride = ws.part_stride;
  a.table = m.pages > 0 ? c.block_table : nullptr;
  a.k_step = (const bf16_t*)k_step;
  a.v_step = (const bf16_t*)v_step;
  a.appended = k_step ? (const int32_t*)(base + ws.appended) : nullptr;
  switch (m.group) {
    case 1: decode_g<1>(a, st); break;
    case 2: decode_g<2>(a, st); break;
    case 3: decode_g<3>(a, st); break;
    case 4: decode_g<4>(a, st); break;
    case 5: decode_g<5>(a, st); break;
    case 6: decode_g<6>(a, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_decode_fused(const Dims& m, const spla_config& cfg, const spla_cache& c,
                               const void* q, const float* gamma, void* out, int32_t* sel_out,
                               const DecodeWs& ws, char* base, hipStream_t st) {
  return decode_fused(m, cfg, c, q, gamma, out, sel_out, ws, base, st, nullptr, nullptr);
}

hipError_t launch_decode_fused_step(const Dims& m, const spla_config& cfg, const spla_cache& c,
                                    const void* k_new, const void* v_new, const void* q,
                                    const float* gamma, void* out, int32_t* sel_out,
                                    const DecodeWs& ws, char* base, hipStream_t st) {
  if (!step_fusable(m) || !use_fused_decode(m)) return hipErrorInvalidValue;
  return decode_fused(m, cfg, c, q, gamma, out, sel_out, ws, base, st, k_new, v_new);
}

}  // namespace spla
