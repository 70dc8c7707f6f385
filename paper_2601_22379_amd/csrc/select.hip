// Block selection kernels: one 1024-thread workgroup per (sequence, KV head)
// (select_blocks), or past 4096 blocks per sequence the two-stage selection
// (select_slice, then select_pick in the last slice of each head to finish);
// the device code is in spla_select.h.
#include "spla_kernels.h"
#include "spla_select.h"

namespace spla {

constexpr int kSelThreads = 1024;

template <int R, bool WIN, int NT = kSelThreads>
__global__ __launch_bounds__(NT) void select_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const float* __restrict__ e_vals,
    const double* __restrict__ tile_part, int32_t* __restrict__ sel_ws,
    int32_t* __restrict__ sel_out, int32_t* __restrict__ meta) {
  __shared__ SelectSmem<NT, kMaxTiles * SPLA_MAX_GROUP> sm;
  __shared__ float wsc[WIN ? kMaxWindows : 1];  // window scores (strided selection)
  const int bh = blockIdx.x;
  select_blocks<NT, R, kMaxTiles * SPLA_MAX_GROUP, false, 0, WIN>(
      m, bh, seq_lens[bh / m.hkv], e_vals, tile_part, sm, sel_ws + (int64_t)bh * m.k,
      meta + bh * 4, sel_out ? sel_out + (int64_t)bh * m.k : nullptr, wsc);
}

// Two-stage selection in one launch, grid (n_sl, bh): every workgroup takes
// its slice's candidates (select_slice); the last slice of a (sequence, KV
// head) to finish (a counter in the synchronisation area, zero between
// calls and reset by that workgroup) picks from all of them (select_pick).
// No workgroup waits for another.
template <int TJ, int GM, int R2>
__global__ __launch_bounds__(kSliceThreads) void select_two_stage_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const float* __restrict__ e_vals,
    const double* __restrict__ tile_part, uint32_t* __restrict__ cand_key,
    int32_t* __restrict__ cand_id, int32_t* __restrict__ cand_n, int32_t* __restrict__ sel_ws,
    int32_t* __restrict__ sel_out, int32_t* __restrict__ meta, int32_t* __restrict__ ctr) {
  __shared__ float sw[kSliceTiles * SPLA_MAX_GROUP];
  __shared__ __align__(16) uint32_t hist[4096];
  __shared__ uint32_t scan[kSliceThreads / 64];
  __shared__ int32_t out[SPLA_MAX_TOP_K];
  __shared__ int s_flag;
  const int sl = blockIdx.x, bh = blockIdx.y, n_sl = gridDim.x;
  const int64_t row = (int64_t)bh * n_sl;
  select_slice<TJ, GM>(m, bh, sl, seq_lens, e_vals, tile_part, cand_key + (row + sl) * m.k,
                       cand_id + (row + sl) * m.k, cand_n + row + sl, sw, hist, scan);
  int32_t* c = ctr + (int64_t)bh * kSyncLine;
  if (!arrive_last(c, n_sl, &s_flag)) return;
  select_pick<R2, kSliceThreads>(m, bh, n_sl, seq_lens, cand_key + row * m.k,
                                 cand_id + row * m.k, cand_n + row, sel_ws + (int64_t)bh * m.k,
                                 meta + bh * 4, sel_out ? sel_out + (int64_t)bh * m.k : nullptr,
                                 hist, scan, out);
  if (threadIdx.x == 0) store_agent(c, 0);
}

template <int TJ, int GM>
static void two_stage_t(const Dims& m, const spla_cache& c, const DecodeWs& ws, char* base,
                        int32_t* sel_out, hipStream_t st) {
  // candidate slots per thread of the pick
  const int64_t r2 = ceil_div((int64_t)ws.n_sl * m.k, kSliceThreads);
  auto kern = r2 <= 4 ? select_two_stage_kernel<TJ, GM, 4>
                      : (r2 <= 16 ? select_two_stage_kernel<TJ, GM, 16>
                                  : select_two_stage_kernel<TJ, GM, 32>);
  hipLaunchKernelGGL(kern, dim3((unsigned)ws.n_sl, (unsigned)m.bh), dim3(kSliceThreads), 0, st,
                     m, c.seq_lens, (const float*)(base + ws.e_vals),
                     (const double*)(base + ws.tile_part), (uint32_t*)(base + ws.cand_key),
                     (int32_t*)(base + ws.cand_id), (int32_t*)(base + ws.cand_n),
                     (int32_t*)(base + ws.sel), sel_out, (int32_t*)(base + ws.meta),
                     (int32_t*)(base + ws.sync) + sync_layout(m).items_done);
}

template <int TJ>
static void two_stage_tj(const Dims& m, const spla_cache& c, const DecodeWs& ws, char* base,
                         int32_t* sel_out, hipStream_t st) {
  if (m.group <= 4) two_stage_t<TJ, 4>(m, c, ws, base, sel_out, st);
  else if (m.group <= 8) two_stage_t<TJ, 8>(m, c, ws, base, sel_out, st);
  else two_stage_t<TJ, SPLA_MAX_GROUP>(m, c, ws, base, sel_out, st);
}

static void launch_select_two_stage(const Dims& m, const spla_cache& c, const DecodeWs& ws,
                                    char* base, int32_t* sel_out, hipStream_t st) {
  const int tj = (int)ceil_div(m.n_tiles, 64);  // tile partials per lane for Z
  if (tj <= 2) two_stage_tj<2>(m, c, ws, base, sel_out, st);
  else if (tj <= 4) two_stage_tj<4>(m, c, ws, base, sel_out, st);
  else two_stage_tj<8>(m, c, ws, base, sel_out, st);
}

hipError_t launch_select(const Dims& m, const spla_cache& c, const DecodeWs& ws, char* base,
                         int32_t* sel_out, hipStream_t st) {
  if (two_stage_select(m)) {
    launch_select_two_stage(m, c, ws, base, sel_out, st);
    return hipGetLastError();
  }
  const float* ev = (const float*)(base + ws.e_vals);
  const double* tp = (const double*)(base + ws.tile_part);
  int32_t* sel = (int32_t*)(base + ws.sel);
  int32_t* meta = (int32_t*)(base + ws.meta);
  // blocks per thread of 1024: at most 4096 blocks here without windows
  // (two stages past that); with windows at most kMaxWindows windows, so at
  // most 16384 blocks
  const int per = (int)ceil_div(m.nb_cap, kSelThreads);
  auto launch = [&](auto kern, int nt) {
    hipLaunchKernelGGL(kern, dim3(m.bh), dim3(nt), 0, st, m, c.seq_lens, ev, tp, sel, sel_out,
                       meta);
  };
  if (windowed(m)) {
    if (per <= 1) launch(select_kernel<1, true>, kSelThreads);
    else if (per <= 2) launch(select_kernel<2, true>, kSelThreads);
    else if (per <= 4) launch(select_kernel<4, true>, kSelThreads);
    else if (per <= 8) launch(select_kernel<8, true>, kSelThreads);
    else launch(select_kernel<16, true>, kSelThreads);
  } else if (m.nb_cap <= 1024) {
    // at most one block per thread of 1024: 256 threads (four wavefronts,
    // so cheaper barriers) with up to four blocks each (many short
    // sequences: 64 x 8 heads at 512 blocks, high-batch decode
    // 170.1 -> 164.9 us)
    if (m.nb_cap <= 256) launch(select_kernel<1, false, 256>, 256);
    else if (m.nb_cap <= 512) launch(select_kernel<2, false, 256>, 256);
    else launch(select_kernel<4, false, 256>, 256);
  } else {
    if (per <= 2) launch(select_kernel<2, false>, kSelThreads);
    else launch(select_kernel<4, false>, kSelThreads);
  }
  return hipGetLastError();
}

}  // namespace spla
