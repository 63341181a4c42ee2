/* Plain-C client of libkvec: the header compiles as C and the library's
 * host-only calls work without a GPU (sizing, argument validation, status
 * strings).  Built and run by tests/test_abi.py; exits non-zero on failure. */
#include <stdio.h>
#include <string.h>

#include "kvec.h"

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                    \
    }                                                              \
  } while (0)

int main(void) {
  kvec_config c;
  memset(&c, 0, sizeof(c));
  c.batch = 1;
  c.n_layers = 32;
  c.n_kv_heads = 8;
  c.n_q_heads = 32;
  c.head_dim = 128;
  c.seq_len = 32768;
  c.window = 32;
  c.window_ext = 64;
  c.budget = 1024;
  c.pool_kernel = 7;
  c.n_adjust_heads = 3;
  c.lambda = 1.0f;
  c.beta = 0.25f;
  c.dtype = KVEC_BF16;
  c.head_criterion = KVEC_HEADS_STD;

  size_t ws = 0, dws = 0;
  CHECK(kvec_workspace_size(&c, &ws) == KVEC_OK && ws > 0);
  CHECK(kvec_decode_workspace_size(&c, 1024, &dws) == KVEC_OK && dws > 0);
  CHECK(kvec_profile_points(&c) == 32 + 12);
  CHECK(kvec_profile_points_lse(&c) == 32 + 8);

  /* validation happens before any launch: bad configurations and null
   * pointers come back as statuses, with no device touched */
  kvec_config bad = c;
  bad.n_q_heads = 72; /* group 9 */
  CHECK(kvec_workspace_size(&bad, &ws) == KVEC_ERR_UNSUPPORTED);
  bad = c;
  bad.head_criterion = 5;
  CHECK(kvec_workspace_size(&bad, &ws) == KVEC_ERR_INVALID);
  const int64_t qs[3] = {32 * 64 * 128, 64 * 128, 128};
  const int64_t ks[3] = {8 * 32768 * 128, 32768 * 128, 128};
  void* fake = (void*)(size_t)(1 << 20);
  CHECK(kvec_score(&c, fake, qs, fake, ks, NULL, (float*)fake, (float*)fake, fake, (size_t)1 << 40,
                   NULL) == KVEC_ERR_INVALID);
  CHECK(kvec_select_cover(&c, 32, (const float*)fake, (const float*)fake, (const float*)fake,
                          (uint64_t*)fake, (int32_t*)fake, NULL, fake, (size_t)1 << 40,
                          NULL) == KVEC_ERR_INVALID);
  CHECK(kvec_coverage(&c, (const uint64_t*)fake, -1, (int64_t*)fake, NULL) == KVEC_ERR_INVALID);
  CHECK(strcmp(kvec_status_string(KVEC_OK), "ok") == 0);
  CHECK(strcmp(kvec_status_string(KVEC_ERR_WORKSPACE), "workspace too small") == 0);
  printf("abi_check: ok (workspace %zu bytes, decode workspace %zu bytes)\n", ws, dws);
  return 0;
}
