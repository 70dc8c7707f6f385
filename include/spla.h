/*
 * spla.h - C ABI of the SPLA decode-step library for AMD Instinct MI355X
 * (gfx950).
 *
 * SPLA ("Block Sparse Plus Linear Attention", arXiv 2601.22379) answers one
 * decode query per attention head by
 *   1. scoring every KV block with a second-order Taylor estimate of its
 *      attention mass built from the block's key mean and diagonal
 *      covariance (Sec. 3.1, Eqs. 8-10), summed over the GQA group after a
 *      per-head normalisation (Sec. 2.2, Eq. 6);
 *   2. selecting the top-k blocks per KV head, with a forced sink block and
 *      the most recent blocks (Sec. 2.1 Eq. 3; Sec. 4 "Sparsity
 *      Specifications");
 *   3. running exact softmax attention over the selected blocks (Eq. 5) and,
 *      from the same read of those blocks, their linear-attention term
 *      (Eq. 16);
 *   4. forming the residual linear attention by subtraction from the global
 *      linear-attention state (Eqs. 14-15) and adding its RMSNorm to the exact
 *      output (Sec. 3.3).
 * The append call maintains what step 1 and step 4 read: the per-block key
 * statistics and the global state S_bar = sum_t phi(k_t)^T v_t (Eq. 15),
 * with phi the softmax over the feature dimension (Sec. 3.2).
 *
 * Conventions shared by every call:
 *  - The library owns no memory. Every buffer is allocated by the caller;
 *    "device" pointers are HIP device memory of the current device, "host"
 *    pointers are ordinary host memory.
 *  - Every argument check happens on the host before anything is enqueued
 *    and returns a negative spla_status; nothing is enqueued on failure.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL is the null stream)
 *    and is asynchronous. Calls on one stream execute in order. Two calls
 *    that share a cache or a workspace must not run concurrently.
 *  - No C++ exception crosses this interface.
 *  - Conditions only the device can see (an append that would overflow the
 *    capacity) set bits in cache->err_flags (if non-NULL) and are otherwise
 *    handled as documented at the call.
 */
#ifndef SPLA_H_
#define SPLA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ status */
typedef enum spla_status {
  SPLA_OK = 0,
  SPLA_ERR_INVALID_ARG = -1, /* NULL pointer, inconsistent or out-of-range value */
  SPLA_ERR_UNSUPPORTED = -2, /* valid, but a shape the library does not implement */
  SPLA_ERR_CAPACITY = -3,    /* a size exceeds the cache capacity or a library limit */
  SPLA_ERR_WORKSPACE = -4,   /* workspace NULL, too small or misaligned */
  SPLA_ERR_HIP = -5          /* the HIP runtime reported an error at launch */
} spla_status;

typedef enum spla_dtype { SPLA_F32 = 0, SPLA_BF16 = 1 } spla_dtype;

/* cfg.flags: the ablations of Sec. 4 "Baselines" */
enum {
  SPLA_FLAG_NO_RLA = 1u,        /* SPA: output = exact sparse branch only */
  SPLA_FLAG_FIRST_ORDER = 2u,   /* block score with Eq. 11 (mean only) instead of Eq. 10 */
  SPLA_FLAG_RLA_NORMALIZE = 4u, /* divide the residual by <phi(q), z_bar - z_selected> */
  SPLA_FLAG_SEPARATE_KERNELS = 8u /* run the decode as separate score / select / sparse /
                                     merge launches instead of the single-launch kernel
                                     (same arithmetic, bit-identical results; for
                                     per-phase timing) */
};

/* err_flags bits written by the device */
enum {
  SPLA_DEVERR_CAPACITY = 1, /* an append was clipped at max_seq_len */
  SPLA_DEVERR_SYNC = 2,     /* a bounded wait of the single-launch decode gave up (for
                               instance because the workspace was never zeroed with
                               spla_workspace_init and a counter started non-zero): the
                               outputs and selection of that call are undefined, and
                               spla_workspace_init repairs the workspace. Only a wait
                               that gives up is detected; counters left non-zero by
                               other means are not checked at launch */
  SPLA_DEVERR_PAGE = 4      /* an append met a block_table entry outside [0, kv_pages):
                               its rows were not written */
};

/* Library limits. */
enum {
  SPLA_MAX_GROUP = 16,      /* query heads per KV head */
  SPLA_MAX_TOP_K = 256,     /* selected blocks per KV head */
  SPLA_MAX_BLOCKS = 32768,  /* blocks per sequence (max_seq_len / block_size) */
  SPLA_WORKSPACE_ALIGN = 256
};

/* ------------------------------------------------------------------ config */
typedef struct spla_config {
  int32_t batch;          /* sequences decoded together, >= 1 */
  int32_t n_q_heads;      /* Hq, a multiple of n_kv_heads */
  int32_t n_kv_heads;     /* Hkv; G = Hq / Hkv query heads share a KV head and one
                             block selection (Sec. 2.2); 1 <= G <= SPLA_MAX_GROUP */
  int32_t head_dim;       /* d: 64 or 128 */
  int32_t block_size;     /* B, the selection granularity (Sec. 2.1): 32, 64 or 128 */
  int32_t top_k;          /* k blocks selected per KV head, forced blocks included;
                             n_sink + n_local <= k <= SPLA_MAX_TOP_K */
  int32_t n_sink_blocks;  /* always-selected leading blocks (paper: 1) */
  int32_t n_local_blocks; /* always-selected most recent blocks (paper: 4) */
  int32_t max_seq_len;    /* per-sequence capacity in tokens, a multiple of B,
                             at most SPLA_MAX_BLOCKS * B */
  int32_t dtype;          /* spla_dtype of q, out and the K/V cache */
  float softmax_scale;    /* s; <= 0 selects 1/sqrt(head_dim). Scales the exact
                             logits and the query inside the block score */
  float rms_eps;          /* epsilon of the RMSNorm on the residual, >= 0 (1e-6). When
                             every token is selected there is no residual and the
                             output is the exact branch at any eps; with eps = 0, a
                             head whose residual is exactly zero while some token is
                             unselected has an undefined (0 / 0) output */
  uint32_t flags;         /* SPLA_FLAG_* */
  int32_t sel_window;     /* strided block selection (Sec. 3.1): the block score is
                             the largest group score of the windows of sel_window
                             tokens, one starting every sel_stride tokens, that
                             share a token with the block (the paper: 32 and 16).
                             Both 0: one window per block. Otherwise sel_stride
                             divides block_size, sel_window is 1 to 4 times
                             sel_stride, max_seq_len / sel_stride <= 16384, and
                             the decode runs as separate launches */
  int32_t sel_stride;
  int32_t kv_pages;       /* paged KV cache (PagedAttention-style, one page = one block
                             of B tokens, as in Sec. 2.1): 0 keeps k_cache / v_cache
                             per sequence as laid out below; > 0 makes them pools of
                             kv_pages pages addressed through spla_cache.block_table,
                             and the decode runs as separate launches */
} spla_config;

/* ------------------------------------------------------------------- cache
 * Caller-owned device buffers that persist across calls. Sizes in bytes are
 * given by spla_cache_bytes (index in brackets). Let nb_cap = max_seq_len / B
 * and n_tiles = ceil(nb_cap / 64) (see [2] for strided selection).
 *  [0] k_cache   dtype [batch][Hkv][max_seq_len * d]      keys
 *  [1] v_cache   dtype [batch][Hkv][max_seq_len * d]      values
 *                fp32: keys token-major ([t][c]), values transposed inside
 *                each block ([t / B][c][t % B]).
 *                bf16: both in 32-token steps of 32 d elements, each step
 *                stored in the order the matrix-core pass loads it, as
 *                16-byte chunks of 8 elements (chunk q at element q * 8 of
 *                step t / 32). With tt = t % 32, key (t, c) is element c % 8
 *                of chunk ((tt / 4) % 2 * (d / 32) + c / 32) * 64
 *                + (c / 8) % 4 * 16 + 4 * (tt / 8) + tt % 4, and value
 *                (t, c) is element tt % 8 of chunk (c / 16) * 64
 *                + (tt / 8) * 16 + c % 16.
 *  [2] blk_stats fp32  [batch][Hkv][n_tiles][2][d/4][64][4]
 *                part 0 the block key mean, part 1 the block's sum of
 *                squared deviations from it (M2; variance = M2 / n_i). Block
 *                i of a sequence is entry i % 64 of tile i / 64: for each
 *                group of four coordinates, 64 consecutive blocks are stored
 *                side by side. With strided selection the entries are the
 *                windows (window w: tokens w * sel_stride .. + sel_window - 1)
 *                and n_tiles = ceil(max_seq_len / sel_stride / 64)
 *  [3] lin_state fp32  [batch][Hkv][d][d]  S_bar[j][c] = sum_t phi(k_t)_j v_t,c (Eq. 15)
 *  [4] lin_norm  fp32  [batch][Hkv][d]     z_bar = sum_t phi(k_t)
 *  [5] seq_lens  int32 [batch]             tokens held by each sequence
 * err_flags: int32 [1] or NULL; SPLA_DEVERR_* bits are OR-ed in, never cleared
 * by the library.
 * Paged caches (kv_pages > 0): [0] and [1] are pools of kv_pages pages, page p
 * holding for every KV head h the B rows of one block in the layout above
 * (element offset (p * Hkv + h) * B * d of the pool); block_table is int32
 * [batch][max_seq_len / B], caller-owned, read-only to the library, entry
 * [b][i] naming the page of block i of sequence b. Every block a sequence
 * holds or will receive by an append must name a page in [0, kv_pages), and
 * no two live blocks may share one; an append skips rows whose entry is out
 * of range (SPLA_DEVERR_PAGE), and a decode reads page 0 for such an entry
 * (its output is then undefined). NULL when kv_pages is 0.
 * A zero-filled cache (spla_reset) is the empty cache.
 */
typedef struct spla_cache {
  void* k_cache;
  void* v_cache;
  float* blk_stats;
  float* lin_state;
  float* lin_norm;
  int32_t* seq_lens;
  int32_t* err_flags;
  const int32_t* block_table;
} spla_cache;

enum { SPLA_CACHE_NUM_BUFFERS = 6 };

/* Kernel phases that spla_decode_ex / spla_step_ex can bracket with events. */
enum {
  SPLA_PHASE_APPEND = 0, /* single-token append of spla_step */
  SPLA_PHASE_SCORE = 1,  /* block statistics stream -> per-head block mass */
  SPLA_PHASE_SELECT = 2, /* group score, top-k */
  SPLA_PHASE_SPARSE = 3, /* fused exact + selected-linear pass over the selected blocks,
                            with the rows of o_bar = phi(q) S_bar split over its workgroups */
  SPLA_PHASE_MERGE = 4,  /* merge of that pass, residual, RMSNorm, output */
  SPLA_PHASE_DECODE = 5, /* the single-launch decode kernel (all of phases 1-4) */
  SPLA_PHASE_LINEAR = 6, /* chunked prefill: the chunkwise linear-attention kernel
                            (o_bar of every query, S_bar and z_bar past the chunk) */
  SPLA_NUM_PHASES = 8
};

/* Optional timing hooks: each non-NULL start[p] / stop[p] (a hipEvent_t) is
 * recorded on the call's stream right before / after the launch(es) of phase
 * p. The phases a call records are given by spla_decode_phase_mask (plus
 * SPLA_PHASE_APPEND for spla_step_ex); the others record nothing. The chunked
 * prefill (spla_prefill_ex) records APPEND (the running unit statistics and
 * the rows and statistics of the chunk), LINEAR, SCORE, SELECT,
 * SPARSE and MERGE for every chunk, so with several chunks the events end up
 * bracketing the last one. */
typedef struct spla_events {
  void* start[SPLA_NUM_PHASES];
  void* stop[SPLA_NUM_PHASES];
} spla_events;

/* ---------------------------------------------------------- host-only calls */

/* Text of a status code (static storage). */
const char* spla_status_string(int32_t status);

/* Name of a phase id ("score", ...), or NULL for an unused id. */
const char* spla_phase_name(int32_t phase);

/* Checks cfg against the limits above. Host only; touches no device. */
int32_t spla_validate(const spla_config* cfg);

/* Bytes of each cache buffer, out_bytes[SPLA_CACHE_NUM_BUFFERS] (host array),
 * in the order listed at spla_cache. Host only. */
int32_t spla_cache_bytes(const spla_config* cfg, size_t* out_bytes);

/* Device workspace that spla_decode / spla_step need (host-only query). The
 * workspace holds scratch (block masses, the selection, per-workgroup
 * records) and, in its last words, the counters of the single-launch decode,
 * which must be zero when a call starts: zero the workspace once with
 * spla_workspace_init (or any zero fill) before its first use; every call
 * leaves the counters zero again. */
int32_t spla_workspace_bytes(const spla_config* cfg, size_t* out_bytes);

/* The phases whose events spla_decode_ex records for cfg, as bits
 * 1 << SPLA_PHASE_*: (1 << SPLA_PHASE_DECODE) when the decode runs as one
 * launch, otherwise the separate score, select, sparse and merge phases (the
 * select phase is folded into the sparse launch on grids of at most two
 * workgroups per compute unit; its two events are then recorded back to
 * back). Host only. */
int32_t spla_decode_phase_mask(const spla_config* cfg, uint32_t* out_mask);

/* Device workspace that spla_append needs for up to max_new tokens per
 * sequence (host-only query). */
int32_t spla_append_workspace_bytes(const spla_config* cfg, int32_t max_new, size_t* out_bytes);

/* Device workspace that spla_prefill needs for n_tokens positions per
 * sequence (host-only query): per-query scores, selections, records and
 * global terms of one chunk of at most 32 positions for the chunked shapes,
 * the decode workspace for the others. */
int32_t spla_prefill_workspace_bytes(const spla_config* cfg, int32_t n_tokens,
                                     size_t* out_bytes);

/* ---------------------------------------------------------- device calls */

/* Zero-fills a decode workspace of workspace_bytes bytes (at least
 * spla_workspace_bytes(cfg), 256-byte aligned) with a fill kernel on
 * `stream`. Needed once per workspace before its first decode. */
int32_t spla_workspace_init(const spla_config* cfg, void* workspace, size_t workspace_bytes,
                            void* stream);

/* Empties the cache: zero-fills blk_stats, lin_state, lin_norm and seq_lens
 * (K/V rows are left as they are; they are never read past seq_lens). */
int32_t spla_reset(const spla_config* cfg, const spla_cache* cache, void* stream);

/* Appends tokens to every (sequence, KV head) (Sec. 3.1 statistics; Eq. 15).
 *  k_new, v_new: device, dtype [batch][Hkv][max_new][d], token-major; only the
 *                first n_b rows of sequence b are read.
 *  n_new:        device int32 [batch] (n_b, 0 <= n_b <= max_new), or NULL for
 *                n_b = max_new for every sequence.
 *  workspace:    device, at least spla_append_workspace_bytes(cfg, max_new),
 *                256-byte aligned.
 * For each sequence b with length L_b = seq_lens[b], the tokens land at
 * positions L_b .. L_b + n_b - 1: key rows go to k_cache, value rows to
 * v_cache, the statistics of every touched block are updated (Chan's
 * parallel combination of mean and M2, computed in fp64), S_bar and z_bar
 * receive phi(k_t)^T v_t and phi(k_t) of every new token (partial sums over
 * token chunks, reduced in a fixed order: deterministic), and seq_lens[b]
 * becomes L_b + n_b. Tokens that would exceed max_seq_len are dropped and
 * SPLA_DEVERR_CAPACITY is set in err_flags. */
int32_t spla_append(const spla_config* cfg, const spla_cache* cache,
                    const void* k_new, const void* v_new, int32_t max_new,
                    const int32_t* n_new, void* workspace, size_t workspace_bytes,
                    void* stream);

/* One SPLA decode step for every sequence (Secs. 2.1-2.2, 3.1-3.3).
 *  q:          device, dtype [batch][Hq][d]; query head m reads KV head m / G.
 *  rms_weight: device fp32 [Hq][d], the RMSNorm weight gamma.
 *  out:        device, dtype [batch][Hq][d] (may not alias q).
 *  sel_idx:    device int32 [batch][Hkv][top_k] or NULL: the selected block
 *              ids of each KV head in ascending order, padded with -1 when a
 *              sequence has fewer than top_k blocks.
 *  workspace:  device, at least spla_workspace_bytes(cfg), 256-byte aligned,
 *              prepared once by spla_workspace_init.
 * Bf16 shapes with d = 128, G <= 6, at most 8192 blocks per sequence and no
 * strided selection run as one kernel launch (unless
 * SPLA_FLAG_SEPARATE_KERNELS); the others as separate score, select, sparse
 * and merge launches (spla_decode_phase_mask tells which).
 * For each sequence with L = seq_lens[b] tokens, nb = ceil(L / B) blocks:
 * if nb <= top_k every block is selected and the output is exact attention;
 * otherwise the sink and local blocks plus the top-scored remaining blocks
 * (ties to the lower block id) are selected, and
 *   out = o_sparse + gamma * r / sqrt(mean(r^2) + eps),  r = o_bar - o_tilde.
 * A sequence with L = 0 yields a zero output and no selection.
 * The cache is only read. */
int32_t spla_decode(const spla_config* cfg, const spla_cache* cache, const void* q,
                    const float* rms_weight, void* out, int32_t* sel_idx,
                    void* workspace, size_t workspace_bytes, void* stream);

/* spla_decode with optional timing events (events may be NULL). */
int32_t spla_decode_ex(const spla_config* cfg, const spla_cache* cache, const void* q,
                       const float* rms_weight, void* out, int32_t* sel_idx,
                       void* workspace, size_t workspace_bytes, const spla_events* events,
                       void* stream);

/* Appends one token per (sequence, KV head), then decodes (Sec. 2: the query
 * at position N attends to tokens 1..N, the new one included).
 *  k_new, v_new: device, dtype [batch][Hkv][d].
 * Equivalent to spla_append with max_new = 1 followed by spla_decode, with
 * the single-token update done in place (no append workspace). A sequence
 * already at capacity is not extended (SPLA_DEVERR_CAPACITY) and decodes
 * over its current tokens. */
int32_t spla_step(const spla_config* cfg, const spla_cache* cache, const void* k_new,
                  const void* v_new, const void* q, const float* rms_weight, void* out,
                  int32_t* sel_idx, void* workspace, size_t workspace_bytes, void* stream);

/* Causal prefill of n_tokens new tokens per sequence (Sec. 2: the decode
 * formulation carries over to prefill). Token t of every (sequence, KV head)
 * is appended at position L_b + t, and the queries at that position get
 * exactly what spla_step would give them there: they see the tokens up to and
 * including their own, with their own block selection, the statistics of
 * their partial blocks up to their position and S_bar over their prefix.
 *  k_new, v_new: device, dtype [n_tokens][batch][Hkv][d] (position-major).
 *  q:            device, dtype [n_tokens][batch][Hq][d].
 *  rms_weight:   device fp32 [Hq][d].
 *  out:          device, dtype [n_tokens][batch][Hq][d] (may not alias q).
 *  sel_idx:      device int32 [n_tokens][batch][Hkv][top_k] or NULL.
 *  workspace:    at least spla_prefill_workspace_bytes(cfg, n_tokens) bytes,
 *                256-byte aligned (no preparation needed).
 * bf16 shapes with G <= 8 run chunks of up to 32 positions through the
 * chunked kernels (Sec. 3.3 "Kernel Design": a chunkwise linear-attention
 * kernel for o_bar that also carries S_bar and z_bar past the chunk, and the
 * fused sparse kernel per query, after per-query scoring that reads each
 * statistics tile once per chunk and per-query top-k); other shapes (which
 * never decode in one launch) run the positions one at a time as spla_step
 * does, on the separate decode launches. n_tokens = 0 does nothing; tokens past max_seq_len
 * are dropped as in spla_step (SPLA_DEVERR_CAPACITY) and the queries at those
 * positions decode over the full cache. */
int32_t spla_prefill(const spla_config* cfg, const spla_cache* cache, int32_t n_tokens,
                     const void* k_new, const void* v_new, const void* q,
                     const float* rms_weight, void* out, int32_t* sel_idx, void* workspace,
                     size_t workspace_bytes, void* stream);

/* spla_prefill with optional timing events (events may be NULL; recorded by
 * the chunked shapes only). */
int32_t spla_prefill_ex(const spla_config* cfg, const spla_cache* cache, int32_t n_tokens,
                        const void* k_new, const void* v_new, const void* q,
                        const float* rms_weight, void* out, int32_t* sel_idx, void* workspace,
                        size_t workspace_bytes, const spla_events* events, void* stream);

/* spla_step with optional timing events (events may be NULL). */
int32_t spla_step_ex(const spla_config* cfg, const spla_cache* cache, const void* k_new,
                     const void* v_new, const void* q, const float* rms_weight, void* out,
                     int32_t* sel_idx, void* workspace, size_t workspace_bytes,
                     const spla_events* events, void* stream);

/* --------------------------------------------- decode without a workspace */

/* Bytes of the library-owned device scratch of spla_decode_noalloc. */
enum { SPLA_NOALLOC_SCRATCH_BYTES = 64 << 20 };

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * spla_decode with the library's own device scratch in place of a caller
 * workspace. Arguments, outputs and errors as spla_decode, without the
 * workspace; SPLA_ERR_WORKSPACE when spla_workspace_bytes(cfg) exceeds
 * SPLA_NOALLOC_SCRATCH_BYTES (the largest workload of 64 sequences x 8 KV
 * heads x 64K tokens at k = 16 needs about 40 MB).
 * The scratch is a static device array of SPLA_NOALLOC_SCRATCH_BYTES: every
 * GPU the library runs on holds one copy until the process ends. The first
 * call on a device takes its address (hipGetSymbolAddress, with that device
 * current) and zero-fills it on `stream`; later calls allocate nothing and
 * call no allocating routine. Every call clears the decode's counters (its
 * synchronisation area) in the scratch with a fill kernel before the decode
 * (the previous call may have used another shape). All calls on one device share the
 * scratch and it keeps the last call's contents: calls that overlap on one
 * GPU (other streams or threads) race, and their outputs are undefined. */
int32_t spla_decode_noalloc(const spla_config* cfg, const spla_cache* cache, const void* q,
                            const float* rms_weight, void* out, int32_t* sel_idx, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPLA_H_ */
