/*
 * scale.h -- C ABI of the MI355X (gfx950) cluster-level sparse-prefill library (libscale.so).
 *
 * The method is Similarity Chunk Rolling (SCR): during chunked prefill, the query sub-chunks of
 * an outer chunk are grouped into clusters of consecutive sub-chunks, the KV-selection function
 * runs once per cluster with the cluster's anchor fingerprint, and every member attends to the
 * shared selection plus attention sinks and a cluster-spanning local window (paper Sec. 5.1,
 * Eqs. 9 and 10, Algorithm 2). This library implements its per-layer hot path in block form:
 *
 *   scale_rep_keys        one representative key per KV block (mean of the block's keys)
 *   scale_select_cluster  anchor fingerprint, head soft-voting over candidate blocks, top-k,
 *                         once per cluster
 *   scale_sparse_prefill  block-sparse attention of every query row over sink blocks, the
 *                         cluster's selected blocks and the causal local window
 *
 * and, on a handle created by scale_init_variant with select_tokens = 1, its token-level form (the paper's own
 * granularity): scale_select_cluster_tokens scores every single candidate token with its own key,
 * top_k counts tokens, and scale_sparse_prefill attends over the selected tokens.
 *
 * Conventions shared by every call:
 *  - Plain C; no HIP or framework types. bf16 tensors are passed as uint16_t bit patterns.
 *  - Device pointers are caller-owned device allocations (any HIP allocation visible to the
 *    handle's device). The only host pointer is `cluster_start`. q, k_pages, v_pages, k_rep and
 *    out start at 16-byte-aligned addresses (every HIP allocation does; the kernels move 16 bytes
 *    per lane): a call given another address returns SCALE_ERR_INVALID_ARG.
 *  - Every call validates all arguments on the host BEFORE any device work and returns a status;
 *    on error nothing is launched and no output is touched. Calls enqueue on the stream given to
 *    scale_init and return without synchronising; a kernel fault surfaces at the caller's next
 *    synchronisation. No C++ exception crosses this boundary.
 *  - A handle is not thread-safe: use one handle per stream. Calls on one handle are ordered by
 *    its stream; the handle's scratch is reused by the next call only after the previous call's
 *    kernels, which the stream order guarantees.
 *
 * Layouts (row-major, innermost last; Hq query heads, Hkv KV heads, d = head_dim,
 * B = block_size, N = n_tokens, nb = N / B):
 *    q       bf16  [N][Hq][d]             token-major queries of the outer chunk
 *    k_pages bf16  [n_pages][Hkv][B][d]   paged key cache, one page = one block of B tokens
 *    v_pages bf16  [n_pages][Hkv][B][d]   paged value cache, same paging as k_pages
 *    block_table int32 [nb]               page holding logical block b; NULL = identity. The
 *                                         kernels index a cache row as (page * Hkv + g) * B in
 *                                         32 bits, so n_pages * Hkv * B < 2^31 (true of any K and
 *                                         V page pools that fit in one device's memory together)
 *    k_rep   fp32  [nb][Hkv][d]           representative keys ([nb][Hkv][2][d]: channel-wise
 *                                         minimum, then maximum, with rep_kind = SCALE_REP_BOUNDS)
 *    sel_idx int32 [n_clusters][top_k]    selected blocks per cluster, ascending, -1 padded
 *                                         ([n_clusters][Hkv][top_k] with kv_head_sets = 1)
 *    sel_cnt int32 [n_clusters]           number of valid entries of each sel_idx row
 *                                         ([n_clusters][Hkv] with kv_head_sets = 1)
 *    out     fp32 or bf16 [N][Hq][d]      attention output (config.out_dtype)
 * Query head h reads KV head floor(h * Hkv / Hq) (consecutive query heads share a KV head).
 *
 * Cluster geometry (cluster j covers sub-chunks [cluster_start[j], cluster_start[j+1]); L is the
 * sub-chunk size, S the sink tokens, W the base local window, k the top-k):
 *    s = cluster_start[j] * L,  e = min(cluster_start[j+1] * L, N),  anchor rows [s, min(s+L, e))
 *    lo_blk   = max(0, min(s, e - W)) / B         local window starts at token lo_blk * B
 *    sink_blk = ceil(S / B),  sink_eff = min(sink_blk, lo_blk)   sink blocks [0, sink_eff)
 *    candidates: blocks [sink_blk, lo_blk)  (n_cand = max(0, lo_blk - sink_blk))
 *    sel_cnt  = min(k, n_cand)
 *    keys of row p in [s, e): sink blocks U selected blocks U tokens [lo_blk * B, p]
 * The three key groups are disjoint and every key lies at or before its query (causal).
 * Token-level selection (select_tokens = 1): the candidates are the tokens
 * [sink_blk * B, lo_blk * B) (n_cand = B * max(0, lo_blk - sink_blk)), sel_cnt = min(k, n_cand),
 * the selected set is sel_cnt single tokens, and sinks and the local window keep their block form.
 */
#ifndef SCALE_H_
#define SCALE_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct scale_ctx* scale_handle;

/* In C++ the status enum has the fixed underlying type int (the size a C enum has), so any code a
 * C caller passes, known or not, is a valid value on the library's side. */
typedef enum
#ifdef __cplusplus
    : int
#endif
{
  SCALE_OK = 0,
  SCALE_ERR_INVALID_ARG = -1,   /* null pointer, inconsistent sizes, malformed cluster_start */
  SCALE_ERR_UNSUPPORTED = -2,   /* valid but outside what this library supports (head_dim, B, ...) */
  SCALE_ERR_OUT_OF_MEMORY = -3, /* scratch allocation failed in scale_init */
  SCALE_ERR_CAPACITY = -4,      /* n_tokens or n_clusters above the capacity given to scale_init */
  SCALE_ERR_HIP = -5            /* a HIP runtime call failed (no device, launch failure, ...) */
} scale_status;

typedef enum { SCALE_OUT_F32 = 0, SCALE_OUT_BF16 = 1 } scale_out_dtype;

/* How a KV block is summarised for block-level selection. */
typedef enum {
  SCALE_REP_MEAN = 0,   /* the mean key; logit sigma * v . mean                                    */
  SCALE_REP_BOUNDS = 1  /* channel-wise min / max of the block's keys (the page criticality of
                           Quest, cited in the paper's Sec. 2); logit sigma * sum_i max(v_i mn_i,
                           v_i mx_i), an upper bound of v . k over the block for sigma > 0          */
} scale_rep_kind;

typedef struct {
  int32_t num_q_heads;   /* Hq >= 1, a multiple of num_kv_heads                              */
  int32_t num_kv_heads;  /* Hkv >= 1                                                         */
  int32_t head_dim;      /* d: 64 or 128                                                     */
  int32_t block_size;    /* B: 64 or 128 tokens per KV block / page                          */
  int32_t sub_chunk;     /* L: query rows per sub-chunk, a positive multiple of B            */
  int32_t top_k;         /* k >= 0 blocks (tokens with select_tokens) selected per cluster;
                            sel_idx rows hold k entries                                      */
  int32_t sink_tokens;   /* S >= 0: attention-sink tokens, rounded up to whole blocks        */
  int32_t local_window;  /* W >= 0: base local window in tokens                              */
  int32_t max_tokens;    /* capacity: largest n_tokens any call will pass (sizes scratch)    */
  int32_t max_clusters;  /* capacity: largest n_clusters any call will pass                  */
  float softmax_scale;   /* attention logit scale; 0 means 1/sqrt(head_dim) (Eqs. 1, 10)     */
  float score_scale;     /* selection logit scale sigma; 0 means 1.0 (the literal v . k)     */
  int32_t out_dtype;     /* scale_out_dtype of the attention output                          */
} scale_config;

/* Variants of the selection step a handle can run instead of the default (all fields 0): the
 * block-level mean-key selection with one set per cluster. Passed to scale_init_variant only, so
 * scale_config keeps the fields of the default path. */
typedef struct {
  int32_t select_tokens; /* 0: block-level selection; 1: token-level selection (top_k counts
                            tokens; scale_init_variant also allocates the token calls' scratch)  */
  int32_t rep_kind;      /* scale_rep_kind of block-level selection (SCALE_REP_BOUNDS with
                            select_tokens = 1 is SCALE_ERR_UNSUPPORTED)                        */
  int32_t kv_head_sets;  /* 0: one selected set per cluster, voted by every query head (Sec.
                            5.1.3 head soft-voting); 1: one set per (cluster, KV head), voted by
                            that KV head's query heads only, and query head h attends over the
                            set of its KV head (sel_idx, sel_cnt and scores_out gain a KV-head
                            dimension)                                                         */
} scale_variant;

/* Create a handle bound to the current HIP device and to `hip_stream` (a hipStream_t; NULL is
 * the default stream). Validates `cfg` first (INVALID_ARG / UNSUPPORTED before any HIP call),
 * then allocates the scratch the calls need for cfg->max_tokens and cfg->max_clusters, once.
 * On success *out holds the handle; on failure *out is NULL. Paper: the per-layer inputs of
 * Algorithm 2 (Q, the KV cache, L, the budgets k, n_init and n_local). The handle runs the
 * default selection (block level, mean representative keys, one set per cluster). */
scale_status scale_init(const scale_config* cfg, void* hip_stream, scale_handle* out);

/* scale_init for a selection variant (see scale_variant); variant NULL is the default path, the
 * same as scale_init. */
scale_status scale_init_variant(const scale_config* cfg, const scale_variant* variant, void* hip_stream,
                                scale_handle* out);

/* Release the handle and its scratch (synchronises the handle's stream first). NULL is a no-op. */
void scale_free(scale_handle h);

/* Representative keys: k_rep[b][g][:] = mean over the B tokens of block b of K[t][g][:], for
 * every logical block b < n_tokens / B. Accumulation is exact for bf16 inputs of moderate
 * exponent range (fp64 sums), rounded once to fp32. The paper selects token by token; selecting
 * KV blocks scored by a representative key is this library's block-level form of the selection
 * function of Eq. 4 / Eq. 9.
 * Requires n_tokens % block_size == 0 and 0 < n_tokens <= max_tokens. */
scale_status scale_rep_keys(scale_handle h, const uint16_t* k_pages, const int32_t* block_table,
                            int32_t n_tokens, float* k_rep);

/* scale_rep_keys for the logical blocks [first_block, n_tokens / B) only, leaving the other rows of
 * k_rep as they are: the incremental form for the outer-chunk loop of Sec. 3.1, where each outer
 * chunk appends blocks to the cache. Requires 0 <= first_block <= n_tokens / B. */
scale_status scale_rep_keys_range(scale_handle h, const uint16_t* k_pages, const int32_t* block_table,
                                  int32_t first_block, int32_t n_tokens, float* k_rep);

/* Cluster-level selection (Eq. 9 with head soft-voting, Sec. 5.1.3), once per cluster:
 *   v[h]     = mean of q[p][h] over the anchor rows                      (Eq. 6 on the anchor)
 *   x[h][b]  = score_scale * v[h] . k_rep[b][g(h)]      for candidate blocks b
 *   score[b] = sum over h of softmax over candidates of x[h][.]   evaluated at b
 *   sel      = top sel_cnt candidates by (score descending, block index ascending), emitted in
 *              ascending block order into sel_idx[j][0..sel_cnt), the rest of the row is -1.
 * cluster_start: HOST int32[n_clusters + 1], strictly increasing, cluster_start[0] >= 0,
 *   cluster_start[n_clusters] = ceil(n_tokens / sub_chunk). cluster_start[0] > 0 is incremental
 *   prefill (the outer-chunk loop of Sec. 3.1): only the sub-chunks from cluster_start[0] on are
 *   processed, against a cache of all n_tokens keys; earlier output rows are not written.
 * sel_cnt (device) receives min(k, n_cand) per cluster (also host-computable from the geometry).
 * scores_out (optional, may be NULL): device fp32 [n_clusters][n_tokens / B]; candidate entries
 *   receive their score, every other entry -1.
 * Arithmetic: the fingerprint is an fp64 sum of the bf16 rows; logits, the per-head softmax
 *   normalisers and the score sum over heads are fp64; each score is rounded once to fp32, and the
 *   top-k orders those fp32 scores (two candidates whose fp64 scores round to one fp32 value tie,
 *   and the lower index wins).
 * On a handle whose variant has rep_kind = SCALE_REP_BOUNDS, k_rep holds the channel-wise bounds
 * and x[h][b] = score_scale * sum_i max(v[h][i] mn[b][g(h)][i], v[h][i] mx[b][g(h)][i]). With
 * kv_head_sets = 1, score and top-k are taken per (cluster j, KV head g) over the query heads of g
 * only, into row j * Hkv + g of sel_idx, sel_cnt and scores_out.
 * Each call adds n_clusters to the handle's retrieval-call counter. On a select_tokens handle
 * this call returns SCALE_ERR_UNSUPPORTED (use scale_select_cluster_tokens). */
scale_status scale_select_cluster(scale_handle h, const uint16_t* q, int32_t n_tokens,
                                  const float* k_rep, const int32_t* cluster_start,
                                  int32_t n_clusters, int32_t* sel_idx, int32_t* sel_cnt,
                                  float* scores_out);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving loops or
 * harnesses that forbid hipMalloc): scale_select_cluster on the default path (block level, mean
 * representative keys, one set per cluster) with no handle. The call allocates nothing: its
 * scratch is one 64 MiB device array of the library, which every device it runs on holds for the
 * life of the process, and the cluster geometry is computed on the device from cluster_start
 * passed by value. Arguments, validation, results and errors as for scale_init (cfg) and
 * scale_select_cluster, with `hip_stream` the stream to enqueue on (NULL: the default stream).
 * A call whose scratch would exceed the array (about n_clusters * Hq * (n_tokens / B) * 8 bytes
 * for the per-candidate weights, plus fingerprints and statistics; the 128K Llama-3-8B layer in
 * clusters of 8 needs about 10 MiB) returns SCALE_ERR_CAPACITY before any device work. Calls on
 * one device share the array: calls that overlap in time on one device race, so serialise them
 * (one stream, or events). No retrieval-call counter is kept (there is no handle). */
scale_status scale_select_cluster_static(const scale_config* cfg, void* hip_stream, const uint16_t* q,
                                         int32_t n_tokens, const float* k_rep, const int32_t* cluster_start,
                                         int32_t n_clusters, int32_t* sel_idx, int32_t* sel_cnt,
                                         float* scores_out);

/* Token-level cluster selection (Eq. 9 with head soft-voting, Sec. 5.1.3, at the granularity of
 * single tokens); handles created with select_tokens = 1 only (else SCALE_ERR_UNSUPPORTED):
 *   v[h]     = mean of q[p][h] over the anchor rows
 *   x[h][t]  = score_scale * v[h] . K[t][g(h)]    for candidate tokens t (their own keys, read
 *              from k_pages through block_table)
 *   score[t] = sum over h of softmax over candidates of x[h][.]   evaluated at t
 *   sel      = top sel_cnt candidates by (score descending, token position ascending), emitted
 *              in ascending order into sel_idx[j][0..sel_cnt), the rest of the row -1.
 * The logits are computed on the matrix cores from a two-piece bf16 split of the fp32
 * fingerprint (relative representation error <= 2^-18) with fp32 accumulation.
 * cluster_start and sel_cnt as for scale_select_cluster.
 * scores_out (optional, may be NULL): device fp32 [n_clusters][n_tokens]; candidate entries
 *   receive their score, every other entry -1.
 * kv_head_sets = 1 works as for scale_select_cluster (rows j * Hkv + g).
 * Each call adds n_clusters to the handle's retrieval-call counter. */
scale_status scale_select_cluster_tokens(scale_handle h, const uint16_t* q, int32_t n_tokens,
                                         const uint16_t* k_pages, const int32_t* block_table,
                                         const int32_t* cluster_start, int32_t n_clusters,
                                         int32_t* sel_idx, int32_t* sel_cnt, float* scores_out);

/* The anchor fingerprints of the most recent selection call on this handle (scale_select_cluster
 * or scale_select_cluster_tokens), each the fp32 rounding of the exact mean of its anchor rows:
 * device fp32 [n_clusters][Hq][d], copied on the handle's stream (no synchronisation). n_clusters
 * may not exceed that call's cluster count (INVALID_ARG, also when no selection call was made). */
scale_status scale_fingerprints(scale_handle h, float* fingerprints, int32_t n_clusters);

/* Block-sparse prefill attention (Eq. 10): for every row p of every cluster and every query
 * head h, out[p][h] = softmax over Kset(p) of (q[p][h] . k_t * softmax_scale) weighted sum of
 * v_t, with Kset(p) = sink blocks U sel_idx[j][0..sel_cnt[j]) U tokens [lo_blk * B, p].
 * sel_idx / sel_cnt are device arrays as written by scale_select_cluster (any ascending or
 * unordered set of distinct candidate blocks is accepted; entries are not re-validated on the
 * device beyond clamping sel_cnt to [0, top_k]). cluster_start is the same host array as for
 * the selection. bf16 output is the round-to-nearest-even of the fp32 result.
 * On a select_tokens handle, sel_idx rows hold token positions (as scale_select_cluster_tokens
 * writes them; each is clamped to [0, n_tokens)) and Kset(p) = sink blocks U those tokens U tokens
 * [lo_blk * B, p]; the selected keys and values are first gathered into handle scratch.
 * With kv_head_sets = 1, query head h of cluster j uses selection row j * Hkv + g(h). */
scale_status scale_sparse_prefill(scale_handle h, const uint16_t* q, const uint16_t* k_pages,
                                  const uint16_t* v_pages, const int32_t* block_table,
                                  int32_t n_tokens, const int32_t* cluster_start,
                                  int32_t n_clusters, const int32_t* sel_idx,
                                  const int32_t* sel_cnt, void* out);

/* Anchor-based clustering of the sub-chunks of an outer chunk (Sec. 5.1.1-5.1.2, Algorithm 1,
 * Eq. 8), producing the cluster_start the calls above take, for the sub-chunks [first_subchunk, M),
 * M = ceil(n_tokens / L) (first_subchunk > 0: the outer chunks of an incremental prefill that are
 * still to run). For every sub-chunk i (rows [i L, min((i + 1) L, n_tokens))) the fingerprint v_i is the mean
 * of its query rows over all heads concatenated (Eq. 6, in R^(Hq d)). One left-to-right pass then
 * forms the clusters: a cluster opens at anchor a and admits the next sub-chunk j while
 * cos(v_a, v_j) >= theta and the cluster holds |C| sub-chunks with |C| * L < l_max; the first j
 * failing either test opens the next cluster. With outer_subchunks > 0, a cluster also closes at
 * every multiple of outer_subchunks (clusters never span two outer chunks). Everything is fp64;
 * a zero fingerprint has an undefined (NaN) cosine and never joins or admits.
 *   q             device bf16 [n_tokens][Hq][d], 0 < n_tokens <= max_tokens
 *   theta         similarity threshold (any value but NaN; > 1 gives single sub-chunks)
 *   l_max         cluster cap in tokens, >= 1 (the paper's default is 8 L)
 *   first_subchunk 0 <= first_subchunk < M
 *   cluster_start HOST int32 with room for M - first_subchunk + 1 entries: receives first_subchunk, ..., M
 *   n_clusters    HOST: receives the number of clusters
 *   cos_band      optional HOST double [M - first_subchunk][span]: cos(v_i, v_{i+o}) at
 *                 [i - first_subchunk][o - 1], NaN past the last sub-chunk;
 *                 span = min(ceil(l_max / L), outer_subchunks if > 0, M - first_subchunk) - 1
 * span above 64 returns SCALE_ERR_UNSUPPORTED. Synchronous: waits for the handle's stream. The
 * result does not count as a selection call. */
scale_status scale_cluster_subchunks(scale_handle h, const uint16_t* q, int32_t n_tokens,
                                     int32_t first_subchunk, double theta, int32_t l_max,
                                     int32_t outer_subchunks, int32_t* cluster_start,
                                     int32_t* n_clusters, double* cos_band);

/* Static text for a status code. Never NULL. */
const char* scale_status_string(scale_status s);

/* Cumulative number of selection calls (clusters) issued on this handle (Sec. 5.1.2). */
scale_status scale_retrieval_calls(scale_handle h, int64_t* calls);

/* Stages of the path, for scale_stage_times. */
typedef enum {
  SCALE_STAGE_REP_KEYS = 0,     /* representative-key reduction                          */
  SCALE_STAGE_FINGERPRINT = 1,  /* anchor fingerprints (two kernels)                     */
  SCALE_STAGE_LOGITS = 2,       /* per-head block logits                                 */
  SCALE_STAGE_VOTE_TOPK = 3,    /* soft-voting scores and top-k                          */
  SCALE_STAGE_ATTENTION = 4,    /* block-sparse attention                                */
  SCALE_STAGE_CLUSTER = 5,      /* sub-chunk similarity of scale_cluster_subchunks        */
  SCALE_STAGE_GATHER = 6,       /* gather of the selected tokens' keys and values          */
  SCALE_NUM_STAGES = 7
} scale_stage;

/* Device-time instrumentation (off by default). While enabled, every stage's kernels of every
 * call are bracketed by a pair of HIP events on the handle's stream (event objects are created
 * on first use and recycled). */
scale_status scale_enable_timing(scale_handle h, int enable);

/* The same instrumentation for a subset of the stages: bit s of stage_mask (s a scale_stage)
 * brackets stage s with a pair of events; 0 turns timing off. scale_enable_timing(h, e) is
 * stage_mask = all stages for e != 0, none otherwise. Every event pair sits in the stream
 * between two launches, so timing only the stages one needs keeps the others' launches back to
 * back. SCALE_ERR_INVALID_ARG for bits at or above SCALE_NUM_STAGES. */
scale_status scale_enable_stage_timing(scale_handle h, uint32_t stage_mask);

/* Synchronises the handle's stream, then writes the accumulated device milliseconds and the
 * number of timed launches of each stage (arrays of SCALE_NUM_STAGES) since the last reset.
 * Either output may be NULL. reset != 0 zeroes the accumulators afterwards. */
scale_status scale_stage_times(scale_handle h, double* ms, int64_t* launches, int reset);

/* Host-only geometry of each cluster, exactly as the calls above use it (no HIP call; usable
 * without a device). For cluster j, writes geo[j*6 + 0..5] =
 *   { s, e, lo_blk, sink_eff, n_cand, sel_cnt }  (n_cand and sel_cnt in tokens when variant has
 *   select_tokens = 1; variant may be NULL).
 * Same validation of cfg, variant and cluster_start as the calls above. */
scale_status scale_cluster_geometry(const scale_config* cfg, const scale_variant* variant, int32_t n_tokens,
                                    const int32_t* cluster_start, int32_t n_clusters,
                                    int32_t* geo);

#ifdef __cplusplus
}
#endif

#endif /* SCALE_H_ */
