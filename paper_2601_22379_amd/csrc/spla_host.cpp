// Host-only part of the C ABI: argument validation, buffer sizing, status
// text. Builds with any C++17 compiler and never touches a device, so it can
// be checked on machines without a GPU (and under the host sanitizers).
#include <math.h>
#include <string.h>

#include "spla_layout.h"

using spla::Dims;

extern "C" const char* spla_status_string(int32_t s) {
  switch (s) {
    case SPLA_OK: return "ok";
    case SPLA_ERR_INVALID_ARG: return "invalid argument";
    case SPLA_ERR_UNSUPPORTED: return "unsupported shape";
    case SPLA_ERR_CAPACITY: return "capacity or library limit exceeded";
    case SPLA_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case SPLA_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

extern "C" const char* spla_phase_name(int32_t p) {
  switch (p) {
    case SPLA_PHASE_APPEND: return "append";
    case SPLA_PHASE_SCORE: return "score";
    case SPLA_PHASE_SELECT: return "select";
    case SPLA_PHASE_SPARSE: return "sparse";
    case SPLA_PHASE_MERGE: return "merge";
    case SPLA_PHASE_DECODE: return "decode";
    case SPLA_PHASE_LINEAR: return "linear";
    default: return nullptr;
  }
}

extern "C" int32_t spla_validate(const spla_config* c) {
  if (!c) return SPLA_ERR_INVALID_ARG;
  if (c->batch < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1) return SPLA_ERR_INVALID_ARG;
  if (c->n_q_heads % c->n_kv_heads != 0) return SPLA_ERR_INVALID_ARG;
  if (c->n_q_heads / c->n_kv_heads > SPLA_MAX_GROUP) return SPLA_ERR_UNSUPPORTED;
  if (c->head_dim < 1) return SPLA_ERR_INVALID_ARG;
  if (c->head_dim != 64 && c->head_dim != 128) return SPLA_ERR_UNSUPPORTED;
  if (c->block_size < 1) return SPLA_ERR_INVALID_ARG;
  if (c->block_size != 32 && c->block_size != 64 && c->block_size != 128) return SPLA_ERR_UNSUPPORTED;
  if (c->n_sink_blocks < 0 || c->n_local_blocks < 0) return SPLA_ERR_INVALID_ARG;
  if (c->top_k < 1) return SPLA_ERR_INVALID_ARG;
  if ((int64_t)c->n_sink_blocks + c->n_local_blocks > c->top_k) return SPLA_ERR_INVALID_ARG;
  if (c->top_k > SPLA_MAX_TOP_K) return SPLA_ERR_CAPACITY;
  if (c->max_seq_len < c->block_size || c->max_seq_len % c->block_size != 0) return SPLA_ERR_INVALID_ARG;
  if (c->max_seq_len / c->block_size > SPLA_MAX_BLOCKS) return SPLA_ERR_CAPACITY;
  if (c->dtype != SPLA_F32 && c->dtype != SPLA_BF16) return SPLA_ERR_INVALID_ARG;
  if (!isfinite(c->softmax_scale)) return SPLA_ERR_INVALID_ARG;
  if (!isfinite(c->rms_eps) || c->rms_eps < 0.0f) return SPLA_ERR_INVALID_ARG;
  const uint32_t known = SPLA_FLAG_NO_RLA | SPLA_FLAG_FIRST_ORDER | SPLA_FLAG_RLA_NORMALIZE |
                         SPLA_FLAG_SEPARATE_KERNELS;
  if (c->flags & ~known) return SPLA_ERR_INVALID_ARG;
  if (c->sel_window != 0 || c->sel_stride != 0) {  // strided selection windows
    if (c->sel_stride < 1 || c->sel_window < c->sel_stride) return SPLA_ERR_INVALID_ARG;
    if (c->block_size % c->sel_stride != 0 || c->sel_window % c->sel_stride != 0 ||
        c->sel_window > 4 * c->sel_stride)
      return SPLA_ERR_UNSUPPORTED;
    if (c->max_seq_len / c->sel_stride > spla::kMaxWindows) return SPLA_ERR_CAPACITY;
  }
  if (c->kv_pages < 0) return SPLA_ERR_INVALID_ARG;
  if (c->kv_pages > (1 << 24)) return SPLA_ERR_CAPACITY;
  // every derived byte count must fit comfortably in 63 bits
  const Dims m = spla::make_dims(*c);
  const double kv = (double)m.bh * m.cap * m.d * 4.0;
  if (kv > 4.0e18) return SPLA_ERR_CAPACITY;
  return SPLA_OK;
}

extern "C" int32_t spla_cache_bytes(const spla_config* c, size_t* out) {
  if (!out) return SPLA_ERR_INVALID_ARG;
  int32_t st = spla_validate(c);
  if (st != SPLA_OK) return st;
  const Dims m = spla::make_dims(*c);
  // K and V: one slot of B * d elements per block (contiguous) or per page
  // and KV head (paged pool)
  const size_t slots = m.pages > 0 ? (size_t)m.pages * m.hkv : (size_t)m.bh * m.nb_cap;
  out[0] = slots * m.B * m.d * m.elem;
  out[1] = slots * m.B * m.d * m.elem;
  out[2] = (size_t)m.bh * m.n_tiles * 2 * m.d * spla::kTileBlocks * 4;
  out[3] = (size_t)m.bh * m.d * m.d * 4;
  out[4] = (size_t)m.bh * m.d * 4;
  out[5] = (size_t)m.batch * 4;
  return SPLA_OK;
}

extern "C" int32_t spla_workspace_bytes(const spla_config* c, size_t* out) {
  if (!out) return SPLA_ERR_INVALID_ARG;
  int32_t st = spla_validate(c);
  if (st != SPLA_OK) return st;
  *out = (size_t)spla::decode_ws_layout(spla::make_dims(*c)).total;
  return SPLA_OK;
}

extern "C" int32_t spla_append_workspace_bytes(const spla_config* c, int32_t max_new, size_t* out) {
  if (!out) return SPLA_ERR_INVALID_ARG;
  int32_t st = spla_validate(c);
  if (st != SPLA_OK) return st;
  if (max_new < 0) return SPLA_ERR_INVALID_ARG;
  if (max_new > c->max_seq_len) return SPLA_ERR_CAPACITY;
  *out = (size_t)spla::append_ws_layout(spla::make_dims(*c), max_new).total;
  return SPLA_OK;
}

extern "C" int32_t spla_decode_phase_mask(const spla_config* c, uint32_t* out) {
  if (!out) return SPLA_ERR_INVALID_ARG;
  int32_t st = spla_validate(c);
  if (st != SPLA_OK) return st;
  if (spla::use_fused_decode(spla::make_dims(*c)) && !(c->flags & SPLA_FLAG_SEPARATE_KERNELS))
    *out = 1u << SPLA_PHASE_DECODE;
  else
    *out = (1u << SPLA_PHASE_SCORE) | (1u << SPLA_PHASE_SELECT) | (1u << SPLA_PHASE_SPARSE) |
           (1u << SPLA_PHASE_MERGE);
  return SPLA_OK;
}

extern "C" int32_t spla_prefill_workspace_bytes(const spla_config* c, int32_t n_tokens,
                                                size_t* out) {
  if (!out) return SPLA_ERR_INVALID_ARG;
  int32_t st = spla_validate(c);
  if (st != SPLA_OK) return st;
  if (n_tokens < 0) return SPLA_ERR_INVALID_ARG;
  if (n_tokens > c->max_seq_len) return SPLA_ERR_CAPACITY;
  const Dims m = spla::make_dims(*c);
  *out = (size_t)(spla::use_chunked_prefill(m) ? spla::prefill_ws_layout(m, n_tokens).total
                                               : spla::decode_ws_layout(m).total);
  return SPLA_OK;
}
