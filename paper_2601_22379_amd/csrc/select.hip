// Block selection kernels: one 1024-thread workgroup per (sequence, KV head)
// (select_blocks), or past 4096 blocks per sequence the two-stage selection
// (select_slice, select_pick); the device code is in spla_select.h.
#include "spla_kernels.h"
#include "spla_select.h"

namespace spla {

constexpr int kSelThreads = 1024;

template <int R, bool WIN>
__global__ __launch_bounds__(kSelThreads) void select_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const float* __restrict__ e_vals,
    const double* __restrict__ tile_part, int32_t* __restrict__ sel_ws,
    int32_t* __restrict__ sel_out, int32_t* __restrict__ meta) {
  __shared__ SelectSmem<kSelThreads, kMaxTiles * SPLA_MAX_GROUP> sm;
  __shared__ float wsc[WIN ? kMaxWindows : 1];  // window scores (strided selection)
  const int bh = blockIdx.x;
  select_blocks<kSelThreads, R, kMaxTiles * SPLA_MAX_GROUP, false, 0, WIN>(
      m, bh, seq_lens[bh / m.hkv], e_vals, tile_part, sm, sel_ws + (int64_t)bh * m.k,
      meta + bh * 4, sel_out ? sel_out + (int64_t)bh * m.k : nullptr, wsc);
}

// Two-stage selection (select_slice, select_pick): grid (n_sl, bh), then bh.
template <int TJ, int GM>
__global__ __launch_bounds__(kSliceThreads) void select_slice_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const float* __restrict__ e_vals,
    const double* __restrict__ tile_part, uint32_t* __restrict__ cand_key,
    int32_t* __restrict__ cand_id, int32_t* __restrict__ cand_n) {
  __shared__ float sw[kSliceTiles * SPLA_MAX_GROUP];
  __shared__ __align__(16) uint32_t hist[4096];
  __shared__ uint32_t scan[kSliceThreads / 64];
  const int sl = blockIdx.x, bh = blockIdx.y, n_sl = gridDim.x;
  const int64_t row = (int64_t)bh * n_sl + sl;
  select_slice<TJ, GM>(m, bh, sl, seq_lens, e_vals, tile_part, cand_key + row * m.k,
                       cand_id + row * m.k, cand_n + row, sw, hist, scan);
}

template <int R2>
__global__ __launch_bounds__(kPickThreads) void select_pick_kernel(
    Dims m, int n_sl, const int32_t* __restrict__ seq_lens, const uint32_t* __restrict__ cand_key,
    const int32_t* __restrict__ cand_id, const int32_t* __restrict__ cand_n,
    int32_t* __restrict__ sel_ws, int32_t* __restrict__ sel_out, int32_t* __restrict__ meta) {
  __shared__ __align__(16) uint32_t hist[4096];
  __shared__ uint32_t scan[kPickThreads / 64];
  __shared__ int32_t out[SPLA_MAX_TOP_K];
  const int bh = blockIdx.x;
  const int64_t row = (int64_t)bh * n_sl;
  select_pick<R2>(m, bh, n_sl, seq_lens, cand_key + row * m.k, cand_id + row * m.k,
                  cand_n + row, sel_ws + (int64_t)bh * m.k, meta + bh * 4,
                  sel_out ? sel_out + (int64_t)bh * m.k : nullptr, hist, scan, out);
}

template <int TJ>
static void slice_t(const Dims& m, const spla_cache& c, const DecodeWs& ws, char* base,
                    hipStream_t st) {
  auto kern = m.group <= 4 ? select_slice_kernel<TJ, 4>
                           : (m.group <= 8 ? select_slice_kernel<TJ, 8>
                                           : select_slice_kernel<TJ, SPLA_MAX_GROUP>);
  hipLaunchKernelGGL(kern, dim3((unsigned)ws.n_sl, (unsigned)m.bh), dim3(kSliceThreads), 0, st,
                     m, c.seq_lens, (const float*)(base + ws.e_vals),
                     (const double*)(base + ws.tile_part), (uint32_t*)(base + ws.cand_key),
                     (int32_t*)(base + ws.cand_id), (int32_t*)(base + ws.cand_n));
}

static void launch_select_two_stage(const Dims& m, const spla_cache& c, const DecodeWs& ws,
                                    char* base, int32_t* sel_out, hipStream_t st) {
  const int tj = (int)ceil_div(m.n_tiles, 64);  // tile partials per lane for Z
  if (tj <= 2) slice_t<2>(m, c, ws, base, st);
  else if (tj <= 4) slice_t<4>(m, c, ws, base, st);
  else slice_t<8>(m, c, ws, base, st);
  const int64_t r2 = ceil_div((int64_t)ws.n_sl * m.k, kPickThreads);
  auto kern = r2 <= 1 ? select_pick_kernel<1>
                      : (r2 <= 2 ? select_pick_kernel<2>
                                 : (r2 <= 4 ? select_pick_kernel<4> : select_pick_kernel<8>));
  hipLaunchKernelGGL(kern, dim3((unsigned)m.bh), dim3(kPickThreads), 0, st, m, ws.n_sl,
                     c.seq_lens, (const uint32_t*)(base + ws.cand_key),
                     (const int32_t*)(base + ws.cand_id), (const int32_t*)(base + ws.cand_n),
                     (int32_t*)(base + ws.sel), sel_out, (int32_t*)(base + ws.meta));
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
  // blocks per thread: at most 4096 blocks here without windows (two stages
  // past that); with windows at most kMaxWindows windows, so at most 16384
  // blocks
  const int per = (int)ceil_div(m.nb_cap, kSelThreads);
  auto launch = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(m.bh), dim3(kSelThreads), 0, st, m, c.seq_lens, ev, tp, sel,
                       sel_out, meta);
  };
  if (windowed(m)) {
    if (per <= 1) launch(select_kernel<1, true>);
    else if (per <= 2) launch(select_kernel<2, true>);
    else if (per <= 4) launch(select_kernel<4, true>);
    else if (per <= 8) launch(select_kernel<8, true>);
    else launch(select_kernel<16, true>);
  } else {
    if (per <= 1) launch(select_kernel<1, false>);
    else if (per <= 2) launch(select_kernel<2, false>);
    else launch(select_kernel<4, false>);
  }
  return hipGetLastError();
}

}  // namespace spla
