// Device entry points of the C ABI: argument checks, then the kernel
// launches of each call on the caller's stream.
#include <hip/hip_runtime.h>

#include <mutex>

#include "spla_kernels.h"

using spla::Dims;

namespace spla {

int compute_units() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v < 1)
      v = 256;
    cached[dev] = v;
  }
  return cached[dev];
}

}  // namespace spla

namespace {

int32_t check_cache(const spla_config* cfg, const spla_cache* c) {
  if (!c) return SPLA_ERR_INVALID_ARG;
  if (!c->k_cache || !c->v_cache || !c->blk_stats || !c->lin_state || !c->lin_norm || !c->seq_lens)
    return SPLA_ERR_INVALID_ARG;
  if ((cfg->kv_pages > 0) != (c->block_table != nullptr)) return SPLA_ERR_INVALID_ARG;
  return SPLA_OK;
}

int32_t check_ws(const void* ws, size_t have, size_t need) {
  if (need == 0) return SPLA_OK;
  if (!ws || have < need) return SPLA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % SPLA_WORKSPACE_ALIGN != 0) return SPLA_ERR_WORKSPACE;
  return SPLA_OK;
}

struct PhaseMark {
  const spla_events* ev;
  hipStream_t st;
  int p;
  PhaseMark(const spla_events* e, hipStream_t s, int phase) : ev(e), st(s), p(phase) {
    if (ev && ev->start[p]) hipEventRecord((hipEvent_t)ev->start[p], st);
  }
  ~PhaseMark() {
    if (ev && ev->stop[p]) hipEventRecord((hipEvent_t)ev->stop[p], st);
  }
};

#define SPLA_TRY(expr)                               \
  do {                                               \
    hipError_t e_ = (expr);                          \
    if (e_ != hipSuccess) return SPLA_ERR_HIP;       \
  } while (0)

// k_step, v_step (or NULL): a step's token whose rank-one update of S_bar the
// decode's sparse pass applies (step_fusable shapes, rows and statistics
// already appended, ws.appended written by the finish kernel).
int32_t run_decode(const spla_config* cfg, const spla_cache* cache, const void* q,
                   const float* w, void* out, int32_t* sel_idx, void* ws, size_t ws_bytes,
                   const spla_events* ev, hipStream_t st, const void* k_step = nullptr,
                   const void* v_step = nullptr) {
  const Dims m = spla::make_dims(*cfg);
  const spla::DecodeWs L = spla::decode_ws_layout(m);
  char* base = static_cast<char*>(ws);
  if (spla::use_fused_decode(m) && !(cfg->flags & SPLA_FLAG_SEPARATE_KERNELS)) {
    PhaseMark pm(ev, st, SPLA_PHASE_DECODE);
    if (k_step)
      SPLA_TRY(spla::launch_decode_fused_step(m, *cfg, *cache, k_step, v_step, q, w, out, sel_idx,
                                              L, base, st));
    else
      SPLA_TRY(spla::launch_decode_fused(m, *cfg, *cache, q, w, out, sel_idx, L, base, st));
    return SPLA_OK;
  }
  // the selection runs in its own launch, or in the scoring launch's last
  // workgroup of each head, or in the sparse launch (the select phase empty)
  const bool in_sparse = spla::sparse_selects(m, k_step != nullptr);
  const bool in_score = !in_sparse && spla::score_selects(m);
  {
    PhaseMark pm(ev, st, SPLA_PHASE_SCORE);
    if (in_score)
      SPLA_TRY(spla::launch_score_select(m, *cfg, *cache, q, L, base, sel_idx, st));
    else
      SPLA_TRY(spla::launch_score(m, *cfg, *cache, q, L, base, st));
  }
  {
    PhaseMark pm(ev, st, SPLA_PHASE_SELECT);  // empty when folded into another launch
    if (!in_sparse && !in_score) SPLA_TRY(spla::launch_select(m, *cache, L, base, sel_idx, st));
  }
  {
    PhaseMark pm(ev, st, SPLA_PHASE_SPARSE);
    SPLA_TRY(spla::launch_sparse(m, *cfg, *cache, q, w, out, sel_idx, L, base, st, k_step,
                                 v_step));
  }
  {
    PhaseMark pm(ev, st, SPLA_PHASE_MERGE);
    SPLA_TRY(spla::launch_merge(m, *cfg, w, out, L, base, st));
  }
  return SPLA_OK;
}

int32_t check_decode_args(const spla_config* cfg, const spla_cache* cache, const void* q,
                          const float* w, void* out, void* ws, size_t ws_bytes) {
  int32_t s = spla_validate(cfg);
  if (s != SPLA_OK) return s;
  if ((s = check_cache(cfg, cache)) != SPLA_OK) return s;
  if (!q || !w || !out) return SPLA_ERR_INVALID_ARG;
  if (out == q) return SPLA_ERR_INVALID_ARG;
  size_t need = 0;
  spla_workspace_bytes(cfg, &need);
  return check_ws(ws, ws_bytes, need);
}

}  // namespace

extern "C" int32_t spla_reset(const spla_config* cfg, const spla_cache* cache, void* stream) {
  int32_t s = spla_validate(cfg);
  if (s != SPLA_OK) return s;
  if ((s = check_cache(cfg, cache)) != SPLA_OK) return s;
  size_t b[SPLA_CACHE_NUM_BUFFERS];
  spla_cache_bytes(cfg, b);
  hipStream_t st = static_cast<hipStream_t>(stream);
  SPLA_TRY(spla::launch_fill_zero(cache->blk_stats, b[2], st));
  SPLA_TRY(spla::launch_fill_zero(cache->lin_state, b[3], st));
  SPLA_TRY(spla::launch_fill_zero(cache->lin_norm, b[4], st));
  SPLA_TRY(spla::launch_fill_zero(cache->seq_lens, b[5], st));
  return SPLA_OK;
}

extern "C" int32_t spla_workspace_init(const spla_config* cfg, void* ws, size_t ws_bytes,
                                       void* stream) {
  int32_t s = spla_validate(cfg);
  if (s != SPLA_OK) return s;
  size_t need = 0;
  spla_workspace_bytes(cfg, &need);
  if ((s = check_ws(ws, ws_bytes, need)) != SPLA_OK) return s;
  SPLA_TRY(spla::launch_fill_zero(ws, need, static_cast<hipStream_t>(stream)));
  return SPLA_OK;
}

extern "C" int32_t spla_append(const spla_config* cfg, const spla_cache* cache, const void* k_new,
                               const void* v_new, int32_t max_new, const int32_t* n_new,
                               void* workspace, size_t workspace_bytes, void* stream) {
  int32_t s = spla_validate(cfg);
  if (s != SPLA_OK) return s;
  if ((s = check_cache(cfg, cache)) != SPLA_OK) return s;
  if (max_new < 0) return SPLA_ERR_INVALID_ARG;
  if (max_new > cfg->max_seq_len) return SPLA_ERR_CAPACITY;
  if (max_new == 0) return SPLA_OK;
  if (!k_new || !v_new) return SPLA_ERR_INVALID_ARG;
  size_t need = 0;
  spla_append_workspace_bytes(cfg, max_new, &need);
  if ((s = check_ws(workspace, workspace_bytes, need)) != SPLA_OK) return s;
  const Dims m = spla::make_dims(*cfg);
  const spla::AppendWs L = spla::append_ws_layout(m, max_new);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (spla::append_fusable(m)) {  // the lengths advance in its last launch
    SPLA_TRY(spla::launch_append_fused(m, *cache, k_new, v_new, max_new, n_new, L,
                                       static_cast<char*>(workspace), st));
  } else {
    SPLA_TRY(spla::launch_append_blocks(m, *cache, k_new, v_new, max_new, n_new, st));
    SPLA_TRY(spla::launch_append_state(m, *cache, k_new, v_new, max_new, n_new, L,
                                       static_cast<char*>(workspace), st));
    SPLA_TRY(spla::launch_append_finish(m, *cache, max_new, n_new, st));
  }
  return SPLA_OK;
}

extern "C" int32_t spla_decode_ex(const spla_config* cfg, const spla_cache* cache, const void* q,
                                  const float* w, void* out, int32_t* sel_idx, void* ws,
                                  size_t ws_bytes, const spla_events* ev, void* stream) {
  int32_t s = check_decode_args(cfg, cache, q, w, out, ws, ws_bytes);
  if (s != SPLA_OK) return s;
  return run_decode(cfg, cache, q, w, out, sel_idx, ws, ws_bytes, ev,
                    static_cast<hipStream_t>(stream));
}

extern "C" int32_t spla_decode(const spla_config* cfg, const spla_cache* cache, const void* q,
                               const float* w, void* out, int32_t* sel_idx, void* ws,
                               size_t ws_bytes, void* stream) {
  return spla_decode_ex(cfg, cache, q, w, out, sel_idx, ws, ws_bytes, nullptr, stream);
}

extern "C" int32_t spla_step_ex(const spla_config* cfg, const spla_cache* cache, const void* k_new,
                                const void* v_new, const void* q, const float* w, void* out,
                                int32_t* sel_idx, void* ws, size_t ws_bytes,
                                const spla_events* ev, void* stream) {
  int32_t s = check_decode_args(cfg, cache, q, w, out, ws, ws_bytes);
  if (s != SPLA_OK) return s;
  if (!k_new || !v_new) return SPLA_ERR_INVALID_ARG;
  const Dims m = spla::make_dims(*cfg);
  hipStream_t st = static_cast<hipStream_t>(stream);
  // the append's last workgroup of each sequence advances its length (the
  // counters: the workspace's item lines, zero between calls)
  const spla::DecodeWs L = spla::decode_ws_layout(m);
  char* base = static_cast<char*>(ws);
  int32_t* fin = reinterpret_cast<int32_t*>(base + L.sync) + spla::sync_layout(m).items_done;
  if (spla::step_fusable(m)) {
    // the token's rows and statistics first; its rank-one update of S_bar is
    // applied by the decode's sparse pass to the rows it reads anyway
    {
      PhaseMark pm(ev, st, SPLA_PHASE_APPEND);
      SPLA_TRY(spla::launch_append_one(m, *cache, k_new, v_new, st, false, fin,
                                       reinterpret_cast<int32_t*>(base + L.appended)));
    }
    return run_decode(cfg, cache, q, w, out, sel_idx, ws, ws_bytes, ev, st, k_new, v_new);
  }
  {
    PhaseMark pm(ev, st, SPLA_PHASE_APPEND);
    SPLA_TRY(spla::launch_append_one(m, *cache, k_new, v_new, st, true, fin));
  }
  return run_decode(cfg, cache, q, w, out, sel_idx, ws, ws_bytes, ev, st);
}

extern "C" int32_t spla_step(const spla_config* cfg, const spla_cache* cache, const void* k_new,
                             const void* v_new, const void* q, const float* w, void* out,
                             int32_t* sel_idx, void* ws, size_t ws_bytes, void* stream) {
  return spla_step_ex(cfg, cache, k_new, v_new, q, w, out, sel_idx, ws, ws_bytes, nullptr, stream);
}

extern "C" int32_t spla_prefill_ex(const spla_config* cfg, const spla_cache* cache,
                                   int32_t n_tokens, const void* k_new, const void* v_new,
                                   const void* q, const float* w, void* out, int32_t* sel_idx,
                                   void* ws, size_t ws_bytes, const spla_events* ev,
                                   void* stream) {
  int32_t s = spla_validate(cfg);
  if (s != SPLA_OK) return s;
  if ((s = check_cache(cfg, cache)) != SPLA_OK) return s;
  if (!q || !w || !out || out == q) return SPLA_ERR_INVALID_ARG;
  if (n_tokens < 0) return SPLA_ERR_INVALID_ARG;
  if (n_tokens > cfg->max_seq_len) return SPLA_ERR_CAPACITY;
  if (n_tokens == 0) return SPLA_OK;
  if (!k_new || !v_new) return SPLA_ERR_INVALID_ARG;
  size_t need = 0;
  spla_prefill_workspace_bytes(cfg, n_tokens, &need);
  if ((s = check_ws(ws, ws_bytes, need)) != SPLA_OK) return s;
  const Dims m = spla::make_dims(*cfg);
  hipStream_t st = static_cast<hipStream_t>(stream);
  // per position: the rows of token t, the queries at t, their outputs
  const size_t kv_step = (size_t)m.bh * m.d * m.elem;
  const size_t q_step = (size_t)m.batch * m.hq * m.d * m.elem;
  const size_t sel_step = (size_t)m.bh * m.k;
  const char* kb = static_cast<const char*>(k_new);
  const char* vb = static_cast<const char*>(v_new);
  const char* qb = static_cast<const char*>(q);
  char* ob = static_cast<char*>(out);
  if (spla::use_chunked_prefill(m)) {
    const spla::PrefillWs L = spla::prefill_ws_layout(m, n_tokens);
    for (int32_t c0 = 0; c0 < n_tokens; c0 += L.T) {
      const int T = n_tokens - c0 < L.T ? n_tokens - c0 : L.T;
      SPLA_TRY(spla::launch_prefill_chunk(m, *cfg, *cache, T, kb + c0 * kv_step,
                                          vb + c0 * kv_step, qb + c0 * q_step, w,
                                          ob + c0 * q_step,
                                          sel_idx ? sel_idx + c0 * sel_step : nullptr, L,
                                          static_cast<char*>(ws), ev, st));
    }
    return SPLA_OK;
  }
  // the decode workspace: its item lines count the append's workgroups; it
  // comes unprepared, so its synchronisation area is cleared first
  char* sync = static_cast<char*>(ws) + spla::decode_ws_layout(m).sync;
  SPLA_TRY(spla::launch_fill_zero(sync, (size_t)spla::sync_layout(m).words * 4, st));
  int32_t* fin = reinterpret_cast<int32_t*>(sync) + spla::sync_layout(m).items_done;
  for (int32_t t = 0; t < n_tokens; ++t) {
    SPLA_TRY(spla::launch_append_one(m, *cache, kb + t * kv_step, vb + t * kv_step, st, true,
                                     fin));
    if ((s = run_decode(cfg, cache, qb + t * q_step, w, ob + t * q_step,
                        sel_idx ? sel_idx + t * sel_step : nullptr, ws, ws_bytes, nullptr, st)) !=
        SPLA_OK)
      return s;
  }
  return SPLA_OK;
}

extern "C" int32_t spla_prefill(const spla_config* cfg, const spla_cache* cache, int32_t n_tokens,
                                const void* k_new, const void* v_new, const void* q,
                                const float* w, void* out, int32_t* sel_idx, void* ws,
                                size_t ws_bytes, void* stream) {
  return spla_prefill_ex(cfg, cache, n_tokens, k_new, v_new, q, w, out, sel_idx, ws, ws_bytes,
                         nullptr, stream);
}

// ---- decode without a caller workspace (callers that cannot allocate) ------
// The decode workspace of spla_decode_noalloc: one copy of this array per
// device, held by every GPU the library runs on until the process ends. In
// host code `scratch` only names the array; its device address is taken once
// per device with hipGetSymbolAddress and only that address is handed to
// kernels.
static __device__ __align__(256) unsigned char scratch[SPLA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's scratch; the first call on a device
// takes it (with that device current) and zero-fills the array on `st`.
int32_t device_scratch(hipStream_t st, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SPLA_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SPLA_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SPLA_ERR_HIP;
    if (spla::launch_fill_zero(p, SPLA_NOALLOC_SCRATCH_BYTES, st) != hipSuccess)
      return SPLA_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return SPLA_OK;
}

}  // namespace

extern "C" int32_t spla_decode_noalloc(const spla_config* cfg, const spla_cache* cache,
                                       const void* q, const float* w, void* out,
                                       int32_t* sel_idx, void* stream) {
  int32_t s = spla_validate(cfg);
  if (s != SPLA_OK) return s;
  if ((s = check_cache(cfg, cache)) != SPLA_OK) return s;
  if (!q || !w || !out || out == q) return SPLA_ERR_INVALID_ARG;
  size_t need = 0;
  spla_workspace_bytes(cfg, &need);
  if (need > (size_t)SPLA_NOALLOC_SCRATCH_BYTES) return SPLA_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* base = nullptr;
  if ((s = device_scratch(st, &base)) != SPLA_OK) return s;
  const Dims m = spla::make_dims(*cfg);
  const spla::DecodeWs L = spla::decode_ws_layout(m);
  // the counters (single launch, selection folded into the scoring launch,
  // two-stage selection) must start at zero; the previous call may have
  // left other data there (another layout), so the synchronisation area is
  // cleared with a fill kernel on every call
  SPLA_TRY(spla::launch_fill_zero(static_cast<char*>(base) + L.sync, (size_t)(L.total - L.sync),
                                  st));
  return run_decode(cfg, cache, q, w, out, sel_idx, base, need, nullptr, st);
}
