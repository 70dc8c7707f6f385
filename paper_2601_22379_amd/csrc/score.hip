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
