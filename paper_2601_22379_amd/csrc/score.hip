// Block scoring kernel (Sec. 3.1): one workgroup per (sequence, KV head,
// tile of 64 blocks) item; every item's loads are in flight from the start
// (after the sequence length, which skips the tiles past the end). Items are
// in tile-major order (the same tile of every (sequence, KV head), then the
// next): the heads' statistics streams run side by side, and with lengths
// that vary the items past a sequence's end gather at the end of the grid
// (high-batch decode 176.4 -> 170.4 us, 1M tokens 50.4 -> 48.1 us, against
// (sequence, KV head)-major order). The per-tile arithmetic is score_items
// (spla_score.h).
#include "spla_kernels.h"
#include "spla_score.h"
#include "spla_select.h"

namespace spla {

template <int G, typename T, int D, int NT>
__global__ __launch_bounds__(256) void score_kernel(
    Dims m, const float* __restrict__ stats, const int32_t* __restrict__ seq_lens,
    const T* __restrict__ q, double s, int first_order, float* __restrict__ e_vals,
    double* __restrict__ tile_part) {
  __shared__ ScoreSmem<G> sm;
  // item x: tiles NT (x / bh) .. of (sequence, KV head) x % bh
  const int t = ((int)blockIdx.x % m.bh) * m.n_tiles + ((int)blockIdx.x / m.bh) * NT;
  // a tile wholly past the sequence end is neither read nor scored: the
  // selection reads the tiles that hold units only
  const int L = min(max(seq_lens[t / m.n_tiles / m.hkv], 0), m.cap);
  if ((t % m.n_tiles) * kTileBlocks * m.us >= L) return;
  score_items<G, T, D, false, NT>(m, stats, seq_lens, q, s, first_order, t, e_vals, tile_part,
                                  sm);
}

// Scoring with the selection folded in (score_selects shapes): items as in
// score_kernel, every tile's scores published device-coherent; the last
// workgroup of a (sequence, KV head) to finish (a counter in the
// synchronisation area, zero between calls and reset by that workgroup)
// selects its blocks (256 threads, R blocks each), so no selection launch
// follows. Same arithmetic as score_kernel + select_kernel: same selection.
template <int G, typename T, int D, int R>
__global__ __launch_bounds__(256) void score_select_kernel(
    Dims m, const float* __restrict__ stats, const int32_t* __restrict__ seq_lens,
    const T* __restrict__ q, double s, int first_order, float* __restrict__ e_vals,
    double* __restrict__ tile_part, int32_t* __restrict__ sel, int32_t* __restrict__ sel_out,
    int32_t* __restrict__ meta, int32_t* __restrict__ ctr) {
  constexpr int SWN = 4 * R * G;  // tile weights: n_tiles <= 4 R
  __shared__ union {
    ScoreSmem<G> sc;
    SelectSmem<256, SWN> se;
  } sm;
  __shared__ int s_flag;
  const int bh = (int)blockIdx.x % m.bh, tile = (int)blockIdx.x / m.bh;
  const int t = bh * m.n_tiles + tile;
  const int L = min(max(seq_lens[bh / m.hkv], 0), m.cap);
  // a tile wholly past the sequence end is neither read nor scored, but
  // still counts itself in
  if (tile * kTileBlocks * m.us < L)
    score_items<G, T, D, true, 1>(m, stats, seq_lens, q, s, first_order, t, e_vals, tile_part,
                                  sm.sc);
  int32_t* c = ctr + (int64_t)bh * kSyncLine;
  if (!arrive_last(c, m.n_tiles, &s_flag)) return;
  select_blocks<256, R, SWN, true, 0, false, G, true>(
      m, bh, L, e_vals, tile_part, sm.se, sel + (int64_t)bh * m.k, meta + bh * 4,
      sel_out ? sel_out + (int64_t)bh * m.k : nullptr);
  if (threadIdx.x == 0) store_agent(c, 0);  // last: vmcnt counts stores
}

// The shapes whose scoring launch also selects: blocks as the units, one
// selection workgroup of 256 threads enough (at most 2048 blocks), and the
// group sizes and element types the fold is built for.
bool score_selects(const Dims& m) {
  const bool types = (m.elem == 4 && m.d == 64) || (m.elem == 2 && m.d == 128);
  const bool g = m.group == 1 || m.group == 2 || m.group == 4 || m.group == 8;
  return types && g && !windowed(m) && !two_stage_select(m) && m.nb_cap <= 2048;
}

template <int G, typename T, int D, int R>
static void score_select_t(const Dims& m, double s, int fo, const spla_cache& c, const void* q,
                           const DecodeWs& ws, char* base, int32_t* sel_out, hipStream_t st) {
  hipLaunchKernelGGL((score_select_kernel<G, T, D, R>), dim3((unsigned)(m.bh * m.n_tiles)),
                     dim3(256), 0, st, m, (const float*)c.blk_stats, (const int32_t*)c.seq_lens,
                     (const T*)q, s, fo, (float*)(base + ws.e_vals),
                     (double*)(base + ws.tile_part), (int32_t*)(base + ws.sel), sel_out,
                     (int32_t*)(base + ws.meta),
                     (int32_t*)(base + ws.sync) + sync_layout(m).items_done);
}

template <int G, typename T, int D>
static void score_select_g(const Dims& m, double s, int fo, const spla_cache& c, const void* q,
                           const DecodeWs& ws, char* base, int32_t* sel_out, hipStream_t st) {
  if (m.nb_cap <= 256) score_select_t<G, T, D, 1>(m, s, fo, c, q, ws, base, sel_out, st);
  else if (m.nb_cap <= 512) score_select_t<G, T, D, 2>(m, s, fo, c, q, ws, base, sel_out, st);
  else if (m.nb_cap <= 1024) score_select_t<G, T, D, 4>(m, s, fo, c, q, ws, base, sel_out, st);
  else score_select_t<G, T, D, 8>(m, s, fo, c, q, ws, base, sel_out, st);
}

template <typename T, int D>
static void score_select_td(const Dims& m, double s, int fo, const spla_cache& c, const void* q,
                            const DecodeWs& ws, char* base, int32_t* sel_out, hipStream_t st) {
  switch (m.group) {
    case 1: score_select_g<1, T, D>(m, s, fo, c, q, ws, base, sel_out, st); break;
    case 2: score_select_g<2, T, D>(m, s, fo, c, q, ws, base, sel_out, st); break;
    case 4: score_select_g<4, T, D>(m, s, fo, c, q, ws, base, sel_out, st); break;
    default: score_select_g<8, T, D>(m, s, fo, c, q, ws, base, sel_out, st); break;
  }
}

hipError_t launch_score_select(const Dims& m, const spla_config& cfg, const spla_cache& c,
                               const void* q, const DecodeWs& ws, char* base, int32_t* sel_out,
                               hipStream_t st) {
  if (!score_selects(m)) return hipErrorInvalidValue;
  const double s = cfg.softmax_scale > 0.f ? (double)cfg.softmax_scale : 1.0 / sqrt((double)m.d);
  const int fo = (int)((cfg.flags & SPLA_FLAG_FIRST_ORDER) != 0);
  if (m.elem == 4) score_select_td<float, 64>(m, s, fo, c, q, ws, base, sel_out, st);
  else score_select_td<bf16_t, 128>(m, s, fo, c, q, ws, base, sel_out, st);
  return hipGetLastError();
}

template <int G, typename T, int D>
static void score_gtd(const Dims& m, const spla_config& cfg, const spla_cache& c, const void* q,
                      const DecodeWs& ws, char* base, hipStream_t st) {
  const double s = cfg.softmax_scale > 0.f ? (double)cfg.softmax_scale : 1.0 / sqrt((double)m.d);
  // window statistics (four times the tiles of blocks at s = B / 4): two
  // tiles per item halve the items and their fixed costs
  const int fo = (int)((cfg.flags & SPLA_FLAG_FIRST_ORDER) != 0);
  if (windowed(m))
    hipLaunchKernelGGL((score_kernel<G, T, D, 2>), dim3((unsigned)(m.bh * ceil_div(m.n_tiles, 2))),
                       dim3(256), 0, st, m, (const float*)c.blk_stats, (const int32_t*)c.seq_lens,
                       (const T*)q, s, fo, (float*)(base + ws.e_vals),
                       (double*)(base + ws.tile_part));
  else
    hipLaunchKernelGGL((score_kernel<G, T, D, 1>), dim3((unsigned)(m.bh * m.n_tiles)), dim3(256),
                       0, st, m, (const float*)c.blk_stats, (const int32_t*)c.seq_lens,
                       (const T*)q, s, fo, (float*)(base + ws.e_vals),
                       (double*)(base + ws.tile_part));
}

template <typename T, int D>
static void score_td(const Dims& m, const spla_config& cfg, const spla_cache& c, const void* q,
                     const DecodeWs& ws, char* base, hipStream_t st) {
  switch (m.group) {
#define SPLA_G(g) case g: score_gtd<g, T, D>(m, cfg, c, q, ws, base, st); break;
    SPLA_G(1) SPLA_G(2) SPLA_G(3) SPLA_G(4) SPLA_G(5) SPLA_G(6) SPLA_G(7) SPLA_G(8)
    SPLA_G(9) SPLA_G(10) SPLA_G(11) SPLA_G(12) SPLA_G(13) SPLA_G(14) SPLA_G(15) SPLA_G(16)
#undef SPLA_G
    default: break;
  }
}

hipError_t launch_score(const Dims& m, const spla_config& cfg, const spla_cache& c,
                        const void* q, const DecodeWs& ws, char* base, hipStream_t st) {
  if (m.elem == 4) {
    if (m.d == 64) score_td<float, 64>(m, cfg, c, q, ws, base, st);
    else score_td<float, 128>(m, cfg, c, q, ws, base, st);
  } else {
    if (m.d == 64) score_td<bf16_t, 64>(m, cfg, c, q, ws, base, st);
    else score_td<bf16_t, 128>(m, cfg, c, q, ws, base, st);
  }
  return hipGetLastError();
}

}  // namespace spla
