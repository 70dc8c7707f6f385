// Launchers of the SPLA kernels (host side). Each returns hipSuccess or the
// launch error; the C ABI maps that to a spla_status.
#pragma once

#include <hip/hip_runtime.h>

#include "spla_layout.h"

namespace spla {

// Compute units of the current device (queried once).
int compute_units();

// Records the start (stop = false) or stop event of phase p, if given.
inline void mark_phase(const spla_events* ev, int p, bool stop, hipStream_t st) {
  if (!ev) return;
  void* e = stop ? ev->stop[p] : ev->start[p];
  if (e) (void)hipEventRecord((hipEvent_t)e, st);
}

// append.hip
// position_major: the new rows are [max_new][batch][Hkv][d] instead of
// [batch][Hkv][max_new][d]
hipError_t launch_append_blocks(const Dims& m, const spla_cache& c, const void* k_new,
                                const void* v_new, int max_new, const int32_t* n_new,
                                hipStream_t st, bool position_major = false);
hipError_t launch_append_state(const Dims& m, const spla_cache& c, const void* k_new,
                               const void* v_new, int max_new, const int32_t* n_new,
                               const AppendWs& ws, char* wsbase, hipStream_t st);
// rows, block statistics and state partials of a bulk append in one pass over
// the new keys and values (append_fusable shapes: bf16, d = 128, blocks as
// the statistics units), then the state reduce, which also advances seq_lens;
// in place of launch_append_blocks + launch_append_state + launch_append_finish
bool append_fusable(const Dims& m);
hipError_t launch_append_fused(const Dims& m, const spla_cache& c, const void* k_new,
                               const void* v_new, int max_new, const int32_t* n_new,
                               const AppendWs& ws, char* wsbase, hipStream_t st);
// the single-token append of a step (statistics, K/V rows and, with rank1,
// the rank-one update of S_bar and z_bar) in one launch. With fin_ctr (the
// items_done lines of a decode workspace's synchronisation area) the last
// workgroup of each sequence advances seq_lens and writes the count the
// sequence received to appended (if not NULL); without it launch_append_finish
// must follow
hipError_t launch_append_one(const Dims& m, const spla_cache& c, const void* k_new,
                             const void* v_new, hipStream_t st, bool rank1 = true,
                             int32_t* fin_ctr = nullptr, int32_t* appended = nullptr);
hipError_t launch_append_finish(const Dims& m, const spla_cache& c, int max_new,
                                const int32_t* n_new, hipStream_t st,
                                int32_t* appended = nullptr);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st);

// score.hip: block scoring
// the scoring launch with the selection folded in (score_selects shapes; in
// place of launch_score + launch_select)
bool score_selects(const Dims& m);
hipError_t launch_score_select(const Dims& m, const spla_config& cfg, const spla_cache& c,
                               const void* q, const DecodeWs& ws, char* wsbase, int32_t* sel_out,
                               hipStream_t st);
hipError_t launch_score(const Dims& m, const spla_config& cfg, const spla_cache& c,
                        const void* q, const DecodeWs& ws, char* wsbase, hipStream_t st);

// select.hip
hipError_t launch_select(const Dims& m, const spla_cache& c, const DecodeWs& ws, char* wsbase,
                         int32_t* sel_out, hipStream_t st);

// sparse.hip: fused pass over the selected blocks (records), then the merge.
// When sparse_selects(m, step), the sparse pass makes the selection itself
// (and writes sel_out) and launch_select must not be called; step: the pass
// applies a step's rank-one update (k_step given to launch_sparse).
bool sparse_selects(const Dims& m, bool step);
// k_step, v_step (or NULL): the step's token, whose rank-one update of S_bar
// the matrix-core pass applies as the fused decode does (step_fusable shapes)
hipError_t launch_sparse(const Dims& m, const spla_config& cfg, const spla_cache& c,
                         const void* q, const float* rms_weight, void* out, int32_t* sel_out,
                         const DecodeWs& ws, char* wsbase, hipStream_t st,
                         const void* k_step = nullptr, const void* v_step = nullptr);
hipError_t launch_merge(const Dims& m, const spla_config& cfg, const float* rms_weight, void* out,
                        const DecodeWs& ws, char* wsbase, hipStream_t st);

// prefill.hip: one chunk of at most kPrefillChunk positions of the chunked
// causal prefill (use_chunked_prefill shapes); q, k_new, v_new, out and
// sel_out point at the chunk's first position
hipError_t launch_prefill_chunk(const Dims& m, const spla_config& cfg, const spla_cache& c,
                                int T, const void* k_new, const void* v_new, const void* q,
                                const float* rms_weight, void* out, int32_t* sel_out,
                                const PrefillWs& ws, char* wsbase, const spla_events* ev,
                                hipStream_t st);

// decode.hip: the single-launch decode (use_fused_decode shapes)
hipError_t launch_decode_fused(const Dims& m, const spla_config& cfg, const spla_cache& c,
                               const void* q, const float* rms_weight, void* out,
                               int32_t* sel_out, const DecodeWs& ws, char* wsbase,
                               hipStream_t st);
// The single-launch decode of a step whose token rows and statistics are
// already appended (launch_append_one without rank1, then launch_append_finish
// with ws.appended; step_fusable shapes): its sparse items add phi(k) v^T of
// the token to the rows of S_bar (and z_bar) they read, use them, and write
// them back, for each sequence that received the token.
hipError_t launch_decode_fused_step(const Dims& m, const spla_config& cfg, const spla_cache& c,
                                    const void* k_new, const void* v_new, const void* q,
                                    const float* rms_weight, void* out, int32_t* sel_out,
                                    const DecodeWs& ws, char* wsbase, hipStream_t st);

}  // namespace spla
