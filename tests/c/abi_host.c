/* Plain C99 client of include/scale.h: host-only calls that need no GPU (validation, geometry,
 * status strings, null handles), and compile-time checks that the configuration struct and the
 * four per-layer calls have the layout and signatures of the boundary the hot path is specified
 * with. Prints one line per check; exits non-zero on the first failure. */
#include <stddef.h>
#include <stdio.h>
#include <string.h>

#include "scale.h"

/* The boundary's signatures, spelled out independently of the header: assigning the library's
 * functions to these pointer types fails to compile (warnings are errors) if a signature drifts. */
typedef scale_status (*init_fn)(const scale_config*, void*, scale_handle*);
typedef scale_status (*rep_keys_fn)(scale_handle, const uint16_t*, const int32_t*, int32_t, float*);
typedef scale_status (*select_fn)(scale_handle, const uint16_t*, int32_t, const float*, const int32_t*, int32_t,
                                  int32_t*, int32_t*, float*);
typedef scale_status (*prefill_fn)(scale_handle, const uint16_t*, const uint16_t*, const uint16_t*, const int32_t*,
                                   int32_t, const int32_t*, int32_t, const int32_t*, const int32_t*, void*);
typedef void (*free_fn)(scale_handle);

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
  if (scale_cluster_geometry(&c, NULL, 131072, cs, 32, geo) != SCALE_OK) return fail("geometry status");
  /* cluster 1: rows [4096, 8192), window from 4096 (block 32), sink block 0, candidates [1, 32) */
  const int32_t want[6] = {4096, 8192, 32, 1, 31, 31};
  for (int i = 0; i < 6; ++i)
    if (geo[6 + i] != want[i]) return fail("geometry of cluster 1");
  if (geo[0 * 6 + 4] != 0 || geo[31 * 6 + 4] != 991) return fail("candidate counts");   /* window from block 992 */
  printf("ok geometry\n");

  /* token-level selection counts candidates in tokens */
  scale_variant v;
  memset(&v, 0, sizeof v);
  v.select_tokens = 1;
  c.top_k = 4096;
  if (scale_cluster_geometry(&c, &v, 131072, cs, 32, geo) != SCALE_OK) return fail("token geometry status");
  if (geo[6 + 4] != 31 * 128 || geo[6 + 5] != 3968) return fail("token geometry of cluster 1");
  printf("ok token geometry\n");

  /* validation happens before any HIP call */
  scale_handle h = (scale_handle)0;
  c.head_dim = 96;
  if (scale_init(&c, NULL, &h) != SCALE_ERR_UNSUPPORTED || h != NULL) return fail("unsupported head_dim");
  c.head_dim = 128;
  v.rep_kind = 1; /* bound keys with token selection */
  if (scale_init_variant(&c, &v, NULL, &h) != SCALE_ERR_UNSUPPORTED) return fail("bounds with tokens");
  v.rep_kind = 0;
  cs[5] = cs[4]; /* not strictly increasing */
  if (scale_cluster_geometry(&c, &v, 131072, cs, 32, geo) != SCALE_ERR_INVALID_ARG) return fail("malformed clusters");
  printf("ok validation\n");

  /* every call rejects a null handle; freeing null is a no-op */
  int64_t calls = 0;
  if (scale_retrieval_calls(NULL, &calls) != SCALE_ERR_INVALID_ARG) return fail("null handle");
  scale_free(NULL);
  if (strcmp(scale_status_string(SCALE_OK), "ok") != 0) return fail("status string");
  if (scale_status_string((scale_status)42) == NULL) return fail("unknown status string");
  printf("ok handles\n");

  /* the configuration holds exactly the boundary's thirteen 4-byte fields, in order */
  init_fn f_init = scale_init;
  rep_keys_fn f_rep = scale_rep_keys;
  select_fn f_sel = scale_select_cluster;
  prefill_fn f_pre = scale_sparse_prefill;
  free_fn f_free = scale_free;
  if (!f_init || !f_rep || !f_sel || !f_pre || !f_free) return fail("boundary functions");
  if (sizeof(scale_config) != 13 * 4 || offsetof(scale_config, num_q_heads) != 0 ||
      offsetof(scale_config, block_size) != 12 || offsetof(scale_config, top_k) != 20 ||
      offsetof(scale_config, max_clusters) != 36 || offsetof(scale_config, softmax_scale) != 40 ||
      offsetof(scale_config, score_scale) != 44 || offsetof(scale_config, out_dtype) != 48)
    return fail("configuration layout");
  printf("ok boundary layout\n");
  return 0;
}
