/* Plain C99 client of include/scale.h: host-only calls that need no GPU (validation, geometry,
 * status strings, null handles). Prints one line per check; exits non-zero on the first failure. */
#include <stdio.h>
#include <string.h>

#include "scale.h"

static int fail(const char* what) {
  printf("FAIL %s\n", what);
  return 1;
}

int main(void) {
  scale_config c;
  memset(&c, 0, sizeof c);
  c.num_q_heads = 32;
  c.num_kv_heads = 8;
  c.head_dim = 128;
  c.block_size = 128;
  c.sub_chunk = 512;
  c.top_k = 32;
  c.sink_tokens = 128;
  c.local_window = 4096;
  c.max_tokens = 131072;
  c.max_clusters = 32;

  /* cluster geometry of the 128K layer in clusters of 8 sub-chunks */
  int32_t cs[33];
  for (int j = 0; j <= 32; ++j) cs[j] = 8 * j;
  int32_t geo[32 * 6];
  if (scale_cluster_geometry(&c, 131072, cs, 32, geo) != SCALE_OK) return fail("geometry status");
  /* cluster 1: rows [4096, 8192), window from 4096 (block 32), sink block 0, candidates [1, 32) */
  const int32_t want[6] = {4096, 8192, 32, 1, 31, 31};
  for (int i = 0; i < 6; ++i)
    if (geo[6 + i] != want[i]) return fail("geometry of cluster 1");
  if (geo[0 * 6 + 4] != 0 || geo[31 * 6 + 4] != 991) return fail("candidate counts");   /* window from block 992 */
  printf("ok geometry\n");

  /* token-level selection counts candidates in tokens */
  c.select_tokens = 1;
  c.top_k = 4096;
  if (scale_cluster_geometry(&c, 131072, cs, 32, geo) != SCALE_OK) return fail("token geometry status");
  if (geo[6 + 4] != 31 * 128 || geo[6 + 5] != 3968) return fail("token geometry of cluster 1");
  printf("ok token geometry\n");

  /* validation happens before any HIP call */
  scale_handle h = (scale_handle)0;
  c.head_dim = 96;
  if (scale_init(&c, NULL, &h) != SCALE_ERR_UNSUPPORTED || h != NULL) return fail("unsupported head_dim");
  c.head_dim = 128;
  c.rep_kind = 1; /* bound keys with token selection */
  if (scale_init(&c, NULL, &h) != SCALE_ERR_UNSUPPORTED) return fail("bounds with tokens");
  c.rep_kind = 0;
  cs[5] = cs[4]; /* not strictly increasing */
  if (scale_cluster_geometry(&c, 131072, cs, 32, geo) != SCALE_ERR_INVALID_ARG) return fail("malformed clusters");
  printf("ok validation\n");

  /* every call rejects a null handle; freeing null is a no-op */
  int64_t calls = 0;
  if (scale_retrieval_calls(NULL, &calls) != SCALE_ERR_INVALID_ARG) return fail("null handle");
  scale_free(NULL);
  if (strcmp(scale_status_string(SCALE_OK), "ok") != 0) return fail("status string");
  if (scale_status_string((scale_status)42) == NULL) return fail("unknown status string");
  printf("ok handles\n");
  return 0;
}
