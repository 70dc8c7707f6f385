// Memory layout of the caller-owned cache buffers and of the decode / append
// workspaces. Shared by the host launch code and the kernels; plain C++ with
// no HIP types so that the host-only validation build can use it too.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "spla.h"

#if defined(__HIPCC__)
#define SPLA_HD __host__ __device__ inline
#else
#define SPLA_HD inline
#endif

namespace spla {

constexpr int kTileBlocks = 64;   // blocks per statistics tile (one wavefront)
constexpr int kSubTokens = 32;    // tokens per sparse-pass sub-tile
constexpr int kAppendChunkTarget = 512;   // append state-partial workgroups to aim for
constexpr int kMaxWindows = 16384;  // strided selection windows per sequence at capacity
constexpr int kSliceBlocks = 1024;  // blocks per slice of the two-stage selection

SPLA_HD int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
SPLA_HD int64_t align_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Shape numbers derived from a validated config.
struct Dims {
  int batch, hq, hkv, group, d, B, k, n_sink, n_local, cap;
  int nb_cap;    // blocks per sequence at capacity
  int us, ul;    // scoring units: unit u holds tokens u us .. u us + ul - 1 (the
                 // blocks, us = ul = B, or the strided selection windows)
  int nu_cap;    // units per sequence at capacity
  int n_tiles;   // statistics tiles (64 units) per (sequence, kv head)
  int pages;     // pages of a paged K/V pool (0: contiguous per-sequence caches)
  int bh;        // batch * hkv
  int elem;      // bytes per q / K / V / out element
};

SPLA_HD Dims make_dims(const spla_config& c) {
  Dims m;
  m.batch = c.batch;
  m.hq = c.n_q_heads;
  m.hkv = c.n_kv_heads;
  m.group = c.n_q_heads / c.n_kv_heads;
  m.d = c.head_dim;
  m.B = c.block_size;
  m.k = c.top_k;
  m.n_sink = c.n_sink_blocks;
  m.n_local = c.n_local_blocks;
  m.cap = c.max_seq_len;
  m.nb_cap = c.max_seq_len / c.block_size;
  const bool win = c.sel_window != 0 || c.sel_stride != 0;
  m.us = win ? c.sel_stride : c.block_size;
  m.ul = win ? c.sel_window : c.block_size;
  m.nu_cap = c.max_seq_len / m.us;
  m.n_tiles = (int)ceil_div(m.nu_cap, kTileBlocks);
  m.pages = c.kv_pages;
  m.bh = c.batch * c.n_kv_heads;
  m.elem = c.dtype == SPLA_F32 ? 4 : 2;
  return m;
}

// ---- cache buffers (element offsets) ---------------------------------------
// fp32 caches: k_cache [bh][cap][d] (token-major), v_cache [bh][nb_cap][d][B]
// (transposed inside each block). bf16 caches: both [bh][cap / 32][32 d],
// each 32-token step stored as the 16-byte chunks (8 elements) that lane l
// of the matrix-core pass loads, chunk q of a step at q * 8 elements:
//   keys    chunk (mt * d/32 + ks) * 64 + l holds token 8 (i / 4) + 4 mt +
//           i % 4, coordinates 32 ks + 8 g .. +7   (l = 16 g + i)
//   values  chunk t * 64 + l holds coordinate 16 t + i, tokens 8 g .. 8 g + 7
// so that each load instruction of a wavefront reads 1 KiB in one piece.
// Every block occupies B * d consecutive elements, its "slot": slot
// bh * nb_cap + i for block i of a contiguous cache, p * Hkv + h for a block
// on page p of a paged pool. Offsets of row tb (0 <= tb < B) of a slot:
SPLA_HD int64_t k_off_slot(const Dims& m, int64_t slot, int tb, int j) {
  if (m.elem == 4) return (slot * m.B + tb) * m.d + j;
  const int tt = tb & 31;
  const int mt = (tt >> 2) & 1, i = 4 * (tt >> 3) + (tt & 3);
  const int q = (mt * (m.d >> 5) + (j >> 5)) * 64 + ((j >> 3) & 3) * 16 + i;
  return (slot * m.B + (tb & ~31)) * m.d + q * 8 + (j & 7);
}
SPLA_HD int64_t v_off_slot(const Dims& m, int64_t slot, int tb, int c) {
  if (m.elem == 4) return (slot * m.d + c) * m.B + tb;
  const int tt = tb & 31;
  const int q = (c >> 4) * 64 + (tt >> 3) * 16 + (c & 15);
  return (slot * m.B + (tb & ~31)) * m.d + q * 8 + (tt & 7);
}
// Contiguous caches: token t of (sequence, kv head) bh.
SPLA_HD int64_t k_off(const Dims& m, int64_t bh, int64_t t, int j) {
  return k_off_slot(m, bh * m.nb_cap + t / m.B, (int)(t % m.B), j);
}
SPLA_HD int64_t v_off(const Dims& m, int64_t bh, int64_t t, int c) {
  return v_off_slot(m, bh * m.nb_cap + t / m.B, (int)(t % m.B), c);
}
// Page of block i of bh in a paged pool, or -1 when its table entry is out
// of range.
SPLA_HD int block_page(const Dims& m, const int32_t* table, int64_t bh, int64_t i) {
  const int p = table[(bh / m.hkv) * m.nb_cap + i];
  return (p >= 0 && p < m.pages) ? p : -1;
}
// Whether the scoring units are strided selection windows rather than blocks.
SPLA_HD bool windowed(const Dims& m) { return m.us != m.B || m.ul != m.B; }

// The separate selection runs in two stages (slices, then a pick) past 4096
// blocks per sequence; a single workgroup per (sequence, KV head) otherwise.
SPLA_HD bool two_stage_select(const Dims& m) { return !windowed(m) && m.nb_cap > 4 * kSliceBlocks; }

// blk_stats [bh][n_tiles][2][d/4][64][4]; returns the offset of the float4
// holding coordinates 4*j4 .. 4*j4+3 of unit `blk`, part 0 (mean) or 1 (M2).
SPLA_HD int64_t stats_off4(const Dims& m, int64_t bh, int64_t blk, int part, int j4) {
  return ((((bh * m.n_tiles + blk / kTileBlocks) * 2 + part) * (m.d / 4) + j4) * kTileBlocks +
          blk % kTileBlocks) * 4;
}

// ---- decode workspace ------------------------------------------------------
constexpr int kPartHead = 48;     // per-record header: m[16], l[16], zw[16]
constexpr int kSparseWaves = 4;   // waves per sparse workgroup
constexpr int kSparsePre = 4;     // S_bar entries per thread a sparse workgroup holds

struct DecodeWs {
  int64_t e_vals;     // f32 [bh][G][n_tiles*64]   exp(ell - tile max), per unit
  int64_t tile_part;  // f64 [bh][G][n_tiles][2]   (max, sum) per 64-unit tile
  int64_t sel;        // i32 [bh][k]               selected blocks, ascending
  int64_t meta;       // i32 [bh][4]               (n_selected, all_selected, length, 0)
  int64_t part;       // f32 [bh][n_wg][part_stride]  sparse workgroup partials
  int64_t appended;   // i32 [batch]               tokens a step appended (fused step)
  int64_t cand_key;   // u32 [bh][n_sl][k]         two-stage selection: slice candidates' keys
  int64_t cand_id;    // i32 [bh][n_sl][k]         ... their block ids (ascending per slice)
  int64_t cand_n;     // i32 [bh][n_sl]            ... their count per slice
  int64_t sync;       // i32 [sync_layout(m).words]  counters of the single-launch decode,
                      //   of the scoring launch that selects and of the two-stage
                      //   selection; zero between calls
  int64_t total;
  int n_sl;           // slices of the two-stage selection
  int n_wg;           // sparse workgroups per (sequence, kv head)
  int part_stride;    // floats per record: header + acc[G][d] + accw[G][d]
};

// The MFMA sparse pass handles bf16 with G <= 8; everything else uses the
// VALU pass. Both write records in the same format.
SPLA_HD bool use_mfma_sparse(const Dims& m) { return m.elem == 2 && m.group <= 8; }

// The single-launch decode covers the matrix-core shapes with d = 128,
// G <= 6 (larger groups exceed its register budget), at most 8192 blocks
// per sequence (its selection runs in one 256-thread workgroup, at most 32
// blocks per thread) and at most 128 (sequence, KV head) units: with more,
// every phase of the separate launches already fills the GPU and the
// hand-offs between workgroups cost more than the overlap gains (64
// sequences x 8 KV heads at 16K-64K tokens: 229 us in one launch, 211 us on
// the separate launches).
constexpr int kFusedMaxBlocks = 256 * 32;
constexpr int kFusedMaxGroup = 6;
constexpr int kFusedMaxUnits = 128;
SPLA_HD bool use_fused_decode(const Dims& m) {
  return use_mfma_sparse(m) && m.d == 128 && m.group <= kFusedMaxGroup &&
         m.nb_cap <= kFusedMaxBlocks && !windowed(m) && m.bh <= kFusedMaxUnits;
}

// The decode workspace's synchronisation area (int32 words). Every counter
// that many workgroups update sits alone in its 128-byte line (counters that
// share a line serialise their atomics).
constexpr int kSyncLine = 32;  // int32 words per line
struct SyncLayout {
  int64_t err;         // error word (bad waits)
  int64_t items_done;  // [bh], line stride: score items finished
  int64_t recs_done;   // [bh], line stride: sparse records written
  int64_t sel_ready;   // [bh][k]: selected block + 2 (1: none), 0 until the selection
                       //   of that (sequence, KV head) is published
  int64_t words;
};
SPLA_HD SyncLayout sync_layout(const Dims& m) {
  SyncLayout y;
  const int64_t per = (int64_t)m.bh * kSyncLine;
  y.err = 0;
  y.items_done = kSyncLine;
  y.recs_done = y.items_done + per;
  y.sel_ready = y.recs_done + per;
  // (+4: a workgroup reads its entries as the 16-byte chunk holding them,
  // which may reach 3 words past the last row)
  y.words = y.sel_ready + align_up((int64_t)m.bh * m.k + 4, kSyncLine);
  return y;
}

SPLA_HD DecodeWs decode_ws_layout(const Dims& m) {
  DecodeWs w;
  const int64_t A = SPLA_WORKSPACE_ALIGN;
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    int64_t o = off;
    off = align_up(off + bytes, A);
    return o;
  };
  // MFMA pass: one 32-token step per wavefront; VALU pass: one 32-token
  // sub-tile of a selected block per workgroup
  w.n_wg = use_mfma_sparse(m) ? (int)ceil_div((int64_t)m.k * (m.B / 32), kSparseWaves)
                              : m.k * (m.B / kSubTokens);
  w.part_stride = kPartHead + 2 * m.group * m.d;
  w.e_vals = take((int64_t)m.bh * m.group * m.n_tiles * kTileBlocks * 4);
  w.tile_part = take((int64_t)m.bh * m.n_tiles * m.group * 2 * 8);
  w.sel = take((int64_t)m.bh * m.k * 4);
  w.meta = take((int64_t)m.bh * 4 * 4);
  w.part = take((int64_t)m.bh * w.n_wg * w.part_stride * 4);
  w.appended = take((int64_t)m.batch * 4);
  w.n_sl = (int)ceil_div(m.nb_cap, kSliceBlocks);
  w.cand_key = take((int64_t)m.bh * w.n_sl * m.k * 4);
  w.cand_id = take((int64_t)m.bh * w.n_sl * m.k * 4);
  w.cand_n = take((int64_t)m.bh * w.n_sl * 4);
  w.sync = take(sync_layout(m).words * 4);
  w.total = off;
  return w;
}

// spla_step folds the token's rank-one update of S_bar into the rows of
// S_bar the matrix-core sparse pass reads (for o_bar) when every sparse
// workgroup holds all its rows in registers.
SPLA_HD bool step_fusable(const Dims& m) {
  if (!use_mfma_sparse(m)) return false;
  const DecodeWs ws = decode_ws_layout(m);
  return ceil_div(m.d, ws.n_wg) * m.d <= kSparsePre * 256;
}

// ---- chunked prefill workspace ------------------------------------------------
constexpr int kPrefillChunk = 32;  // positions per chunk of the chunked prefill
constexpr int kPrefillStepsPerWave = 8;  // 32-token steps per wavefront of its sparse pass

// The chunked prefill covers the matrix-core shapes (bf16, G <= 8); the other
// shapes run position by position (the single-token append, then a decode).
SPLA_HD bool use_chunked_prefill(const Dims& m) { return use_mfma_sparse(m); }

struct PrefillWs {
  int T;            // positions per chunk
  int nu_touch;     // statistics units that T consecutive tokens can touch
  int n_wg;         // sparse workgroups per query (kPrefillStepsPerWave steps per wavefront)
  int part_stride;  // floats per record
  int64_t ustat;    // f32 [bh][nu_touch][T][2][d]  running (mean, M2) of the touched units
  int64_t e_vals;   // f32 [bh T][G][n_tiles*64]    per query, as the decode's
  int64_t tile_part;  // f64 [bh T][G][n_tiles][2]
  int64_t sel;      // i32 [bh T][k]
  int64_t meta;     // i32 [bh T][4]
  int64_t part;     // f32 [bh T][n_wg][part_stride]
  int64_t obar;     // f32 [bh][T G][d]  o_bar of every query (row = position G + head)
  int64_t zq;       // f32 [bh][T G]     <phi(q), z_bar> of every query
  int64_t total;
};

SPLA_HD PrefillWs prefill_ws_layout(const Dims& m, int n_tokens) {
  PrefillWs w;
  const int64_t A = SPLA_WORKSPACE_ALIGN;
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    int64_t o = off;
    off = align_up(off + bytes, A);
    return o;
  };
  w.T = n_tokens < 1 ? 1 : (n_tokens < kPrefillChunk ? n_tokens : kPrefillChunk);
  // units u with u us < L0 + T and u us + ul > L0
  w.nu_touch = (int)ceil_div(w.T + m.ul, m.us) + 1;
  const DecodeWs d = decode_ws_layout(m);
  w.n_wg = (int)ceil_div((int64_t)m.k * (m.B / 32), kSparseWaves * kPrefillStepsPerWave);
  w.part_stride = d.part_stride;
  const int64_t nq = (int64_t)m.bh * w.T;
  w.ustat = take((int64_t)m.bh * w.nu_touch * w.T * 2 * m.d * 4);
  w.e_vals = take(nq * m.group * m.n_tiles * kTileBlocks * 4);
  w.tile_part = take(nq * m.n_tiles * m.group * 2 * 8);
  w.sel = take(nq * m.k * 4);
  w.meta = take(nq * 4 * 4);
  w.part = take(nq * w.n_wg * w.part_stride * 4);
  w.obar = take(nq * m.group * m.d * 4);
  w.zq = take(nq * m.group * 4);
  w.total = off;
  return w;
}

// ---- append workspace ------------------------------------------------------
struct AppendWs {
  int64_t part_s;  // f32 [bh][n_chunks][d][d]
  int64_t part_z;  // f32 [bh][n_chunks][d]
  int64_t total;
  int n_chunks;
  int chunk_tokens;
};

SPLA_HD AppendWs append_ws_layout(const Dims& m, int max_new) {
  AppendWs w;
  int64_t want = ceil_div(kAppendChunkTarget, m.bh);
  int64_t most = ceil_div(max_new > 0 ? max_new : 1, kSubTokens);
  int64_t n = want < most ? want : most;
  if (n < 1) n = 1;
  w.chunk_tokens = (int)align_up(ceil_div(max_new > 0 ? max_new : 1, n), kSubTokens);
  w.n_chunks = (int)ceil_div(max_new > 0 ? max_new : 1, w.chunk_tokens);
  const int64_t A = SPLA_WORKSPACE_ALIGN;
  w.part_s = 0;
  int64_t off = align_up((int64_t)m.bh * w.n_chunks * m.d * m.d * 4, A);
  w.part_z = off;
  off = align_up(off + (int64_t)m.bh * w.n_chunks * m.d * 4, A);
  w.total = off;
  return w;
}

}  // namespace spla
