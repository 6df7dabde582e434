/* A plain C99 caller of libchorus.so: checks that include/chorus.h is valid C
 * and that the host-side entry points behave as declared without a GPU (every
 * call below fails argument validation before anything is launched).  Built
 * and run by tests/test_abi.py. */
#include <stdio.h>
#include <string.h>

#include "chorus.h"

#define CHECK(cond)                                            \
  do {                                                         \
    if (!(cond)) {                                             \
      printf("FAILED line %d: %s\n", __LINE__, #cond);         \
      return 1;                                                \
    }                                                          \
  } while (0)

int main(void) {
  chorus_shape shape = {1, 100, 2, 128};
  chorus_tensor t = {(void*)0x10000, 100 * 2 * 128, 2 * 128, 128};
  chorus_block_mask mask = {1, 2, 2, 64, (const int32_t*)0x10000, (const int32_t*)0x10000};
  chorus_key_scale ks = {200, 1.5f};
  size_t ws;
  CHECK(chorus_version() > 0);
  CHECK(strcmp(chorus_status_string(CHORUS_OK), "CHORUS_OK") == 0);
  ws = chorus_build_block_mask_workspace_size(&shape);
  CHECK(ws > 0);
  /* top_p outside [0, 1] */
  CHECK(chorus_build_block_mask(CHORUS_BF16, &shape, &t, &t, 0.088, 1.5, 0.1, 64, NULL, (int32_t*)0x10000,
                                (int32_t*)0x10000, 2 * 2 * 2, NULL, (void*)0x10000, ws, NULL) ==
        CHORUS_ERR_INVALID_ARG);
  CHECK(strlen(chorus_last_error()) > 0);
  /* kv block of 96 */
  CHECK(chorus_build_block_mask(CHORUS_BF16, &shape, &t, &t, 0.088, 0.5, 0.1, 96, NULL, (int32_t*)0x10000,
                                (int32_t*)0x10000, 2 * 2 * 2, NULL, (void*)0x10000, ws, NULL) ==
        CHORUS_ERR_UNSUPPORTED);
  /* key scale past the sequence */
  ks.n_first = 101;
  CHECK(chorus_block_sparse_attn_fwd(CHORUS_BF16, &shape, &t, &t, &t, NULL, NULL, NULL, &mask, NULL, 0.088f, &ks,
                                     &t, NULL, NULL, 0, NULL) == CHORUS_ERR_INVALID_ARG);
  /* fp8 attention without scales */
  CHECK(chorus_block_sparse_attn_fwd_fp8(&shape, &t, &t, &t, NULL, NULL, NULL, &mask, NULL, 0.088f, NULL, &t, NULL,
                                         NULL, 0, NULL) == CHORUS_ERR_INVALID_ARG);
  /* visit map size of a kv-128 mask: 2 rows per head, ceil(1 / 32) word each */
  mask.block = 128;
  CHECK(chorus_visit_map_bytes(&mask) == 1 * 2 * 2 * 1 * 4);
  CHECK(chorus_visit_update(&mask, NULL, NULL) == CHORUS_ERR_INVALID_ARG);
  printf("ok\n");
  return 0;
}
