/* Host-only check of the C ABI: include/spla.h compiles as C, and the
 * validation / sizing calls return the documented codes. Built by
 * tests/test_abi_host.py with the host sanitizers and run on the CPU. */
#include <stdio.h>
#include <string.h>

#include "spla.h"

static spla_config base(void) {
  spla_config c;
  memset(&c, 0, sizeof c);
  c.batch = 4; c.n_q_heads = 32; c.n_kv_heads = 8; c.head_dim = 128; c.block_size = 64;
  c.top_k = 32; c.n_sink_blocks = 1; c.n_local_blocks = 4; c.max_seq_len = 131072;
  c.dtype = SPLA_BF16; c.softmax_scale = 0.0f; c.rms_eps = 1e-6f; c.flags = 0;
  return c;
}

int main(void) {
  int fails = 0;
#define EXPECT(expr, want)                                                        \
  do {                                                                            \
    int got_ = (int)(expr);                                                       \
    if (got_ != (want)) { printf("FAIL %s: got %d want %d\n", #expr, got_, want); ++fails; } \
  } while (0)
  spla_config c = base();
  EXPECT(spla_validate(&c), SPLA_OK);
  EXPECT(spla_validate(NULL), SPLA_ERR_INVALID_ARG);
  c = base(); c.n_q_heads = 30; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base(); c.n_q_heads = 8 * 17; EXPECT(spla_validate(&c), SPLA_ERR_UNSUPPORTED);
  c = base(); c.head_dim = 96; EXPECT(spla_validate(&c), SPLA_ERR_UNSUPPORTED);
  c = base(); c.block_size = 48; c.max_seq_len = 48 * 10; EXPECT(spla_validate(&c), SPLA_ERR_UNSUPPORTED);
  c = base(); c.top_k = 4; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base(); c.top_k = 5; EXPECT(spla_validate(&c), SPLA_OK);
  c = base(); c.top_k = 257; EXPECT(spla_validate(&c), SPLA_ERR_CAPACITY);
  c = base(); c.max_seq_len = 1000; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base(); c.max_seq_len = 64 * 32769; EXPECT(spla_validate(&c), SPLA_ERR_CAPACITY);
  c = base(); c.dtype = 7; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base(); c.rms_eps = -1.0f; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base(); c.flags = 16; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base(); c.flags = SPLA_FLAG_SEPARATE_KERNELS; EXPECT(spla_validate(&c), SPLA_OK);
  c = base(); c.n_sink_blocks = -1; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base(); c.batch = 0; EXPECT(spla_validate(&c), SPLA_ERR_INVALID_ARG);
  c = base();
  size_t b[SPLA_CACHE_NUM_BUFFERS];
  EXPECT(spla_cache_bytes(&c, b), SPLA_OK);
  EXPECT(b[0] == (size_t)4 * 8 * 131072 * 128 * 2, 1);
  EXPECT(b[1] == b[0], 1);
  EXPECT(b[2] == (size_t)4 * 8 * 32 * 2 * 128 * 64 * 4, 1);
  EXPECT(b[3] == (size_t)4 * 8 * 128 * 128 * 4, 1);
  EXPECT(b[4] == (size_t)4 * 8 * 128 * 4, 1);
  EXPECT(b[5] == (size_t)4 * 4, 1);
  EXPECT(spla_cache_bytes(&c, NULL), SPLA_ERR_INVALID_ARG);
  size_t ws = 0;
  EXPECT(spla_workspace_bytes(&c, &ws), SPLA_OK);
  EXPECT(ws > 0 && ws % SPLA_WORKSPACE_ALIGN == 0, 1);
  EXPECT(spla_append_workspace_bytes(&c, 16384, &ws), SPLA_OK);
  EXPECT(ws > 0 && ws % SPLA_WORKSPACE_ALIGN == 0, 1);
  EXPECT(spla_append_workspace_bytes(&c, -1, &ws), SPLA_ERR_INVALID_ARG);
  EXPECT(spla_append_workspace_bytes(&c, 131073, &ws), SPLA_ERR_CAPACITY);
  EXPECT(strcmp(spla_status_string(SPLA_ERR_WORKSPACE), "workspace missing, too small or misaligned") == 0, 1);
  EXPECT(spla_phase_name(SPLA_PHASE_SCORE) != NULL && strcmp(spla_phase_name(SPLA_PHASE_SCORE), "score") == 0, 1);
  EXPECT(spla_phase_name(99) == NULL, 1);
  printf("%s\n", fails ? "FAILED" : "ALL OK");
  return fails ? 1 : 0;
}
