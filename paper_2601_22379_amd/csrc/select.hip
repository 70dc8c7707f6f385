// Block selection kernel: one 1024-thread workgroup per (sequence, KV head);
// the selection itself is select_blocks (spla_select.h).
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

hipError_t launch_select(const Dims& m, const spla_cache& c, const DecodeWs& ws, char* base,
                         int32_t* sel_out, hipStream_t st) {
  const float* ev = (const float*)(base + ws.e_vals);
  const double* tp = (const double*)(base + ws.tile_part);
  int32_t* sel = (int32_t*)(base + ws.sel);
  int32_t* meta = (int32_t*)(base + ws.meta);
  const int per = (int)ceil_div(m.nb_cap, kSelThreads);
#define SPLA_R(r)                                                                            \
  if (windowed(m))                                                                           \
    hipLaunchKernelGGL((select_kernel<r, true>), dim3(m.bh), dim3(kSelThreads), 0, st, m,    \
                       c.seq_lens, ev, tp, sel, sel_out, meta);                              \
  else                                                                                       \
    hipLaunchKernelGGL((select_kernel<r, false>), dim3(m.bh), dim3(kSelThreads), 0, st, m,   \
                       c.seq_lens, ev, tp, sel, sel_out, meta)
  if (per <= 1) SPLA_R(1);
  else if (per <= 2) SPLA_R(2);
  else if (per <= 4) SPLA_R(4);
  else if (per <= 8) SPLA_R(8);
  else if (per <= 16) SPLA_R(16);
  else SPLA_R(32);
#undef SPLA_R
  return hipGetLastError();
}

}  // namespace spla
