// Internal declarations shared by the host runtime and the gfx950 kernels of libscale.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scale.h"

namespace scale {

// Geometry of one cluster as the kernels read it (see include/scale.h for the definitions).
struct ClusterGeo {
  int32_t s;         // first query row
  int32_t e;         // one past the last query row
  int32_t anchor_end;
  int32_t lo_blk;    // local window starts at token lo_blk * B
  int32_t sink_eff;  // sink blocks [0, sink_eff)
  int32_t n_cand;    // candidate blocks [sink_blk, sink_blk + n_cand)
  int32_t sel_cnt;   // min(top_k, n_cand)
  int32_t item0;     // first attention work item of the cluster (host geometry; 0 where unused)
};
static_assert(sizeof(ClusterGeo) == 32, "ClusterGeo is uploaded as raw bytes");

// One attention work item: a tile of query positions of one cluster for one KV head group.
struct WorkItem {
  int32_t cluster;
  int32_t kv_head;
  int32_t p0;        // first query position of the tile
  int32_t n_rows;    // positions in the tile (<= the tile size)
};
static_assert(sizeof(WorkItem) == 16, "WorkItem is uploaded as raw bytes");

// ---- host validation and geometry (scale_api.cpp) ----

// The configuration rules of scale_init_variant (no HIP call).
scale_status validate_config(const scale_config* c, const scale_variant* v);
// Validates n_tokens and cluster_start against the configuration (the rules of every per-layer
// call, capacity included) and, when geo is not null, writes each cluster's geometry.
scale_status plan_geometry(const scale_config& c, const scale_variant& v, int32_t n_tokens,
                           const int32_t* cluster_start, int32_t n_clusters, ClusterGeo* geo);

// ---- launchers (each defined next to its kernel) ----

// k_rep[b][g][:] = mean over block b of K (fp64 accumulation, one rounding to fp32), or with
// `bounds` k_rep[b][g][0 / 1][:] = its channel-wise minimum / maximum, for the logical blocks b in
// [first_block, n_blocks).
hipError_t launch_rep_keys(const uint16_t* k_pages, const int32_t* block_table, int first_block, int n_blocks,
                           int num_kv_heads, int block_size, int head_dim, bool bounds, float* k_rep,
                           hipStream_t stream);

// Anchor fingerprints: mean of each cluster's anchor rows (fp64 sums), rounded once to fp32 into
// `fingerprints` and, when fingerprints64 is not null, stored unrounded there too.
hipError_t launch_fingerprints(const uint16_t* q, const ClusterGeo* geo, int n_clusters,
                               int num_q_heads, int head_dim, float* fingerprints, double* fingerprints64,
                               hipStream_t stream);

// Candidate chunks of the selection kernels for `max_cand` candidates: the statistics and factor
// scratch hold n_clusters * Hq * selection_chunks(max_cand) entries.
int selection_chunks(int max_cand);

// fp64 selection logits of candidate c of cluster j per query head, reduced per 64-candidate chunk
// k to the softmax partials stats[j][h][k] = (m, sum of exp(x - m)) and the weights
// weights[j][h][c] = exp(x - m) (row stride `cand_stride`); `bounds` scores the channel-wise key
// bounds.
hipError_t launch_block_logits(const double* fingerprints, const float* k_rep, const ClusterGeo* geo,
                               int n_clusters, int max_cand, int64_t cand_stride, int sink_blk,
                               int num_q_heads, int num_kv_heads, int head_dim, bool bounds, double score_scale,
                               double* weights, double2* stats, hipStream_t stream);

// Soft-voting scores (fp64, rounded once to fp32) and deterministic top-k per cluster, or per
// (cluster, KV head) with `per_kv` (output rows j * Hkv + g, each voted by the query heads of g).
// `factors` is scratch of the size of the statistics.
hipError_t launch_vote_topk(const double* weights, const double2* stats, double* factors, const ClusterGeo* geo,
                            int n_clusters, int max_cand, int64_t cand_stride, int sink_blk, int num_q_heads,
                            int num_kv_heads, bool per_kv, int top_k, int n_blocks, float* spill, int32_t* sel_idx,
                            int32_t* sel_cnt, float* scores_out, hipStream_t stream);

// Sub-chunk similarity for the anchor-based clustering of sub-chunks [first, M), M =
// ceil(n_tokens / sub_chunk), indexed from first: fp64 fingerprints [M - first][Hq * d], their
// inverse norms, and band[i][o - 1] = cos(v_i, v_{i+o}) for o = 1 .. span (NaN past the last).
hipError_t launch_subchunk_similarity(const uint16_t* q, int n_tokens, int first_subchunk, int sub_chunk,
                                      int num_q_heads, int head_dim, int span, double* fingerprints,
                                      double* inv_norm, double* band, hipStream_t stream);
constexpr int kMaxClusterSpan = 64;   // largest band width (cluster cap - 1) the library supports

// ---- token-level selection ----
// Layout plan of the token scoring kernels for one call: fingerprint rows are (cluster, head of the
// group) with the group padded to gp = a power of two; r_pad rows per KV head in groups of 128;
// candidates in chunks of chunk_tokens (= tiles_per_chunk 64-token tiles), n_chunks of them.
constexpr int kTokenTile = 64;        // rows per gathered tile of selected tokens
constexpr int kTokenChunkTiles = 16;  // candidate tiles per statistics chunk (1024 tokens)
inline int token_chunks(int max_tokens) {
  return (max_tokens + kTokenTile * kTokenChunkTiles - 1) / (kTokenTile * kTokenChunkTiles);
}
struct TokenPlan {
  int gp, r_pad, n_rowgroups, tiles_per_chunk, n_chunks, chunk_tokens;
};
int token_group_pad(int group);
int token_row_pad(int n_clusters, int group);
TokenPlan plan_token_selection(int n_clusters, int group, int num_kv_heads, int max_cand);

// Per-KV-head partial soft-voting scores of every candidate token: partial[j][g][c] = sum over the
// query heads h of g of softmax_c(x[j][h][.]) at c, x = sigma * v[j][h] . K[first_token + c][g].
// Scratch: F [Hkv][r_pad][2][d] bf16, stats [Hkv][r_pad][n_chunks], lse2 [Hkv][r_pad].
hipError_t launch_token_selection(const float* fingerprints, const uint16_t* k_pages, const int32_t* block_table,
                                  const ClusterGeo* geo, int n_clusters, int max_cand, int first_token,
                                  int num_q_heads, int num_kv_heads, int head_dim, int block_size,
                                  float score_scale, int64_t cand_stride, uint16_t* F, float2* stats, float* lse2,
                                  float* partial, hipStream_t stream);

// Score = sum of the partials over KV heads (into spill [cluster][cand_stride]), or with `per_kv`
// each KV head's own partial row, then the deterministic top-k of vote_topk; entries are token
// positions first_token + c. scores_out (optional) rows have n_tokens entries.
hipError_t launch_vote_topk_tokens(const float* partial, const ClusterGeo* geo, int n_clusters, int64_t cand_stride,
                                   int max_cand, int first_token, int num_kv_heads, bool per_kv, int top_k,
                                   int n_tokens, float* spill, int32_t* sel_idx, int32_t* sel_cnt, float* scores_out,
                                   hipStream_t stream);

// Selected keys and values of every cluster copied to gk / gv [cluster][Hkv][kpad][d] in selection
// order, kpad = top_k rounded up to kTokenTile; the rows of the last partial tile past sel_cnt are
// zero.
hipError_t launch_gather_selected(const uint16_t* k_pages, const uint16_t* v_pages, const int32_t* block_table,
                                  const int32_t* sel_idx, const int32_t* sel_cnt, bool per_kv, int n_clusters,
                                  int top_k, int kpad, int n_tokens, int num_kv_heads, int head_dim, int block_size,
                                  uint16_t* gk, uint16_t* gv, hipStream_t stream);

// Block-sparse attention over the work list. With gk != null (token-level selection) the selected
// keys are the gathered rows gk / gv [cluster][Hkv][kpad][d], sel_cnt of them, instead of the
// blocks sel_idx names. With `per_kv` the selection row of (cluster j, KV head g) is j * Hkv + g.
// `queue` holds kAttentionQueues + 1 counters, zero before the launch and zero again after it (the
// launch's persistent work-groups take their items from them).
hipError_t launch_sparse_attention(const uint16_t* q, const uint16_t* k_pages, const uint16_t* v_pages,
                                   const int32_t* block_table, const ClusterGeo* geo,
                                   const WorkItem* items, int n_items, const int32_t* sel_idx,
                                   const int32_t* sel_cnt, bool per_kv, int top_k, int num_q_heads,
                                   int num_kv_heads, int head_dim, int block_size, int n_blocks,
                                   float qk_scale_log2, int out_bf16, void* out, const uint16_t* gk,
                                   const uint16_t* gv, int kpad, uint32_t* queue, hipStream_t stream);
constexpr int kAttentionQueues = 8;

// The attention work list of the clusters [0, n_clusters) written to `items` from their device
// geometry: cluster j's items start at geo[j].item0; inside a cluster, position tiles from the last
// to the first, each once per (head group, KV head), KV head fastest.
hipError_t launch_build_work_items(const ClusterGeo* geo, int n_clusters, int tile_positions, int head_groups,
                                   int num_kv_heads, WorkItem* items, hipStream_t stream);

// Query positions per attention work item for a group of `group` query heads per KV head and a
// head dim (a multiple of kTilePositions), and the number of head groups one KV head's query heads
// are split into. WorkItem.kv_head carries the KV head in its low 16 bits and the head group above.
int attention_tile_positions(int group, int head_dim);
int attention_head_groups(int group, int head_dim);
constexpr int kTilePositions = 32;

}  // namespace scale
