// Host runtime of libscale: argument validation, cluster geometry, scratch, the attention work
// list, and the launches behind the C ABI declared in include/scale.h.
//
// Every entry point validates on the host before touching the device. Per-call metadata (the
// cluster geometry and the attention work list) is written into a ring of pinned host slots and
// copied to device scratch asynchronously on the handle's stream; a slot is reused only after
// the event recorded behind its copy has completed.
#include "scale.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include "common.h"

namespace {

using scale::ClusterGeo;
using scale::WorkItem;

constexpr int kRingSlots = 4;

struct Slot {
  void* host = nullptr;      // pinned
  hipEvent_t done = nullptr; // recorded after the copy that reads `host`
  bool pending = false;
};

struct TimedLaunch {
  int stage;
  hipEvent_t start, stop;
};

}  // namespace

struct scale_ctx {
  scale_config cfg{};
  scale_variant var{};
  hipStream_t stream = nullptr;
  int device = 0;
  int64_t retrieval_calls = 0;
  int max_blocks = 0;        // max_tokens / B (rounded up)
  int max_items = 0;
  int last_clusters = 0;     // clusters of the most recent selection call (its fingerprints)
  // device scratch
  ClusterGeo* d_geo = nullptr;
  WorkItem* d_items = nullptr;
  uint32_t* d_attn_queue = nullptr;   // attention work-queue counters (zero between launches)
  float* d_fingerprints = nullptr;
  // block-level selection: fp64 fingerprints, per-chunk weights and softmax partials, chunk factors
  double* d_fp64 = nullptr;
  double* d_weights = nullptr;
  double2* d_stats = nullptr;
  double* d_factors = nullptr;
  float* d_spill = nullptr;
  // sub-chunk clustering: fp64 fingerprints, inverse norms, cosine band (device) and the band's
  // pinned host copy
  int max_subchunks = 0;
  double* d_sub_fp = nullptr;
  double* d_inv_norm = nullptr;
  double* d_band = nullptr;
  double* h_band = nullptr;
  // token-level selection (select_tokens): fingerprint pieces, chunk statistics, log-normalisers,
  // per-KV-head partial scores, the score rows of the top-k, and the gathered keys / values
  int kpad = 0;              // top_k rounded up to a whole gathered tile
  int64_t tok_stride = 0;    // row stride of the partial scores and score rows: max_tokens rounded up to
                             // a whole token tile, so every row starts 256-byte aligned
  uint16_t* d_tok_F = nullptr;
  float2* d_tok_stats = nullptr;
  float* d_tok_lse = nullptr;
  float* d_tok_partial = nullptr;
  float* d_tok_score = nullptr;
  uint16_t* d_gk = nullptr;
  uint16_t* d_gv = nullptr;
  // cluster geometry: the copy the device holds in d_geo (geo_dev_clusters entries; -1 when none) and
  // a host scratch of max_clusters entries; items_valid when d_items holds the work list of d_geo
  std::vector<ClusterGeo> geo_dev, geo_tmp;
  int geo_dev_clusters = -1;
  bool items_valid = false;
  // pinned staging ring
  size_t slot_bytes = 0;
  Slot slots[kRingSlots];
  int next_slot = 0;
  // stage timing: bit s set = stage s bracketed by events
  uint32_t timing_mask = 0;
  std::vector<TimedLaunch> timed;       // recorded, not yet read
  std::vector<hipEvent_t> spare_events; // recycled
  double stage_ms[SCALE_NUM_STAGES] = {};
  int64_t stage_launches[SCALE_NUM_STAGES] = {};
  hipEvent_t open_start = nullptr;
};

namespace {

}  // namespace

namespace scale {

scale_status validate_config(const scale_config* c, const scale_variant* v) {
  if (!c || !v) return SCALE_ERR_INVALID_ARG;
  if (c->num_q_heads < 1 || c->num_kv_heads < 1 || c->num_q_heads % c->num_kv_heads) return SCALE_ERR_INVALID_ARG;
  if (c->head_dim < 1 || c->block_size < 1 || c->sub_chunk < 1) return SCALE_ERR_INVALID_ARG;
  if (c->top_k < 0 || c->sink_tokens < 0 || c->local_window < 0) return SCALE_ERR_INVALID_ARG;
  if (c->max_tokens < 1 || c->max_clusters < 1) return SCALE_ERR_INVALID_ARG;
  if (!std::isfinite(c->softmax_scale) || c->softmax_scale < 0.f) return SCALE_ERR_INVALID_ARG;
  if (!std::isfinite(c->score_scale)) return SCALE_ERR_INVALID_ARG;
  if (c->out_dtype != SCALE_OUT_F32 && c->out_dtype != SCALE_OUT_BF16) return SCALE_ERR_INVALID_ARG;
  if (v->select_tokens != 0 && v->select_tokens != 1) return SCALE_ERR_INVALID_ARG;
  if (v->rep_kind != SCALE_REP_MEAN && v->rep_kind != SCALE_REP_BOUNDS) return SCALE_ERR_INVALID_ARG;
  if (v->kv_head_sets != 0 && v->kv_head_sets != 1) return SCALE_ERR_INVALID_ARG;
  if (v->select_tokens && v->rep_kind == SCALE_REP_BOUNDS) return SCALE_ERR_UNSUPPORTED;   // tokens use their keys
  if (c->head_dim != 64 && c->head_dim != 128) return SCALE_ERR_UNSUPPORTED;
  if (c->block_size != 64 && c->block_size != 128) return SCALE_ERR_UNSUPPORTED;
  if (c->sub_chunk % c->block_size) return SCALE_ERR_UNSUPPORTED;
  if (c->num_q_heads / c->num_kv_heads > 8) return SCALE_ERR_UNSUPPORTED;
  // sizes that keep every int32 index of the kernels in range
  if ((int64_t)c->max_tokens * c->num_q_heads * c->head_dim >= ((int64_t)1 << 40)) return SCALE_ERR_UNSUPPORTED;
  {
    // attention work items of the largest call (one per tile of positions, per head group and KV head)
    const int group = c->num_q_heads / c->num_kv_heads;
    const int64_t tiles = ((int64_t)c->max_tokens + kTilePositions - 1) / kTilePositions + c->max_clusters;
    if (tiles * c->num_kv_heads * attention_head_groups(group, c->head_dim) >= INT32_MAX) return SCALE_ERR_UNSUPPORTED;
  }
  if (v->select_tokens) {
    // gathered rows and token-scoring rows are int32 indices in the kernels
    const int64_t kpad = ((int64_t)c->top_k + scale::kTokenTile - 1) / scale::kTokenTile * scale::kTokenTile;
    if ((int64_t)c->max_clusters * c->num_kv_heads * kpad >= ((int64_t)1 << 31)) return SCALE_ERR_UNSUPPORTED;
    if ((int64_t)c->max_clusters * 8 * c->num_kv_heads >= ((int64_t)1 << 24)) return SCALE_ERR_UNSUPPORTED;
  }
  return SCALE_OK;
}

// Validates n_tokens and cluster_start against the config; fills the geometry when geo != null.
scale_status plan_geometry(const scale_config& c, const scale_variant& v, int32_t n_tokens,
                           const int32_t* cluster_start, int32_t n_clusters, ClusterGeo* geo) {
  if (!cluster_start || n_clusters < 1 || n_tokens < 1) return SCALE_ERR_INVALID_ARG;
  if (n_tokens % c.block_size) return SCALE_ERR_UNSUPPORTED;
  if (n_tokens > c.max_tokens || n_clusters > c.max_clusters) return SCALE_ERR_CAPACITY;
  const int64_t M = ((int64_t)n_tokens + c.sub_chunk - 1) / c.sub_chunk;
  if (cluster_start[0] < 0 || cluster_start[n_clusters] != M) return SCALE_ERR_INVALID_ARG;
  for (int j = 0; j < n_clusters; ++j)
    if (cluster_start[j + 1] <= cluster_start[j]) return SCALE_ERR_INVALID_ARG;
  if (!geo) return SCALE_OK;
  const int B = c.block_size;
  const int sink_blk = (c.sink_tokens + B - 1) / B;
  const int group = c.num_q_heads / c.num_kv_heads;
  const int tp = attention_tile_positions(group, c.head_dim);
  const int64_t items_per_tile = (int64_t)attention_head_groups(group, c.head_dim) * c.num_kv_heads;
  int64_t item0 = 0;
  for (int j = 0; j < n_clusters; ++j) {
    ClusterGeo& g = geo[j];
    g.s = (int32_t)((int64_t)cluster_start[j] * c.sub_chunk);
    g.e = (int32_t)std::min<int64_t>((int64_t)cluster_start[j + 1] * c.sub_chunk, n_tokens);
    g.anchor_end = std::min(g.s + c.sub_chunk, g.e);
    const int lo = std::max(0, std::min(g.s, g.e - c.local_window));
    g.lo_blk = lo / B;
    g.sink_eff = std::min(sink_blk, g.lo_blk);
    g.n_cand = std::max(0, g.lo_blk - sink_blk) * (v.select_tokens ? B : 1);
    g.sel_cnt = std::min(c.top_k, g.n_cand);
    // capped: a cluster set whose work list exceeds the handle's capacity is refused before use
    g.item0 = (int32_t)std::min<int64_t>(item0, INT32_MAX);
    item0 += (int64_t)((g.e - g.s + tp - 1) / tp) * items_per_tile;
  }
  return SCALE_OK;
}

}  // namespace scale

namespace {

using scale::plan_geometry;
using scale::validate_config;

int64_t max_work_items(const scale_config& c) {
  const int64_t tiles = ((int64_t)c.max_tokens + scale::kTilePositions - 1) / scale::kTilePositions + c.max_clusters;
  return tiles * c.num_kv_heads * scale::attention_head_groups(c.num_q_heads / c.num_kv_heads, c.head_dim);
}

hipEvent_t take_event(scale_ctx* h) {
  if (!h->spare_events.empty()) {
    hipEvent_t e = h->spare_events.back();
    h->spare_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Opens / closes the timing bracket of one stage (no-ops unless timing is enabled).
void stage_begin(scale_ctx* h, int stage) {
  if (!(h->timing_mask >> stage & 1u)) return;
  h->open_start = take_event(h);
  if (h->open_start) (void)hipEventRecord(h->open_start, h->stream);
}
void stage_end(scale_ctx* h, int stage) {
  if (!(h->timing_mask >> stage & 1u) || !h->open_start) return;
  hipEvent_t stop = take_event(h);
  if (stop && hipEventRecord(stop, h->stream) == hipSuccess) {
    h->timed.push_back({stage, h->open_start, stop});
  } else {
    h->spare_events.push_back(h->open_start);
    if (stop) h->spare_events.push_back(stop);
  }
  h->open_start = nullptr;
}

void release(scale_ctx* h) {
  if (!h) return;
  for (auto& t : h->timed) {
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  for (auto e : h->spare_events) (void)hipEventDestroy(e);
  for (auto& s : h->slots) {
    if (s.done) (void)hipEventDestroy(s.done);
    if (s.host) (void)hipHostFree(s.host);
  }
  (void)hipFree(h->d_geo);
  (void)hipFree(h->d_items);
  (void)hipFree(h->d_attn_queue);
  (void)hipFree(h->d_fingerprints);
  (void)hipFree(h->d_fp64);
  (void)hipFree(h->d_weights);
  (void)hipFree(h->d_stats);
  (void)hipFree(h->d_factors);
  (void)hipFree(h->d_spill);
  (void)hipFree(h->d_sub_fp);
  (void)hipFree(h->d_inv_norm);
  (void)hipFree(h->d_band);
  if (h->h_band) (void)hipHostFree(h->h_band);
  (void)hipFree(h->d_tok_F);
  (void)hipFree(h->d_tok_stats);
  (void)hipFree(h->d_tok_lse);
  (void)hipFree(h->d_tok_partial);
  (void)hipFree(h->d_tok_score);
  (void)hipFree(h->d_gk);
  (void)hipFree(h->d_gv);
  delete h;
}

// Next pinned staging slot, waiting (rarely) for the copy that last read it.
scale_status acquire_slot(scale_ctx* h, Slot** out) {
  Slot& s = h->slots[h->next_slot];
  h->next_slot = (h->next_slot + 1) % kRingSlots;
  if (s.pending) {
    if (hipEventSynchronize(s.done) != hipSuccess) return SCALE_ERR_HIP;
    s.pending = false;
  }
  *out = &s;
  return SCALE_OK;
}

// Copies the first `bytes` of the slot to `dst` and marks the slot busy until the copy is done.
scale_status upload(scale_ctx* h, Slot* s, void* dst, size_t bytes) {
  if (bytes == 0) return SCALE_OK;
  if (hipMemcpyAsync(dst, s->host, bytes, hipMemcpyHostToDevice, h->stream) != hipSuccess) return SCALE_ERR_HIP;
  if (hipEventRecord(s->done, h->stream) != hipSuccess) return SCALE_ERR_HIP;
  s->pending = true;
  return SCALE_OK;
}

scale_status check_launch(hipError_t e) { return e == hipSuccess ? SCALE_OK : SCALE_ERR_HIP; }

// The kernels move 16 bytes per lane through q, k_pages, v_pages, k_rep and out.
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Makes d_geo hold geo[0, n_clusters): uploaded through a staging slot unless the device already
// holds exactly these entries (the calls of one layer, and the layers of a prefill chunk, share
// their clusters). Every call on the handle is ordered on its stream, so the host record of what
// was last enqueued is what the device holds when the next launch runs.
scale_status sync_geometry(scale_ctx* h, const ClusterGeo* geo, int n_clusters) {
  const size_t bytes = sizeof(ClusterGeo) * (size_t)n_clusters;
  if (n_clusters == h->geo_dev_clusters && std::memcmp(geo, h->geo_dev.data(), bytes) == 0) return SCALE_OK;
  Slot* slot = nullptr;
  scale_status st = acquire_slot(h, &slot);
  if (st != SCALE_OK) return st;
  std::memcpy(slot->host, geo, bytes);
  h->geo_dev_clusters = -1;
  h->items_valid = false;
  if ((st = upload(h, slot, h->d_geo, bytes)) != SCALE_OK) return st;
  std::memcpy(h->geo_dev.data(), geo, bytes);
  h->geo_dev_clusters = n_clusters;
  return SCALE_OK;
}

}  // namespace

extern "C" {

const char* scale_status_string(scale_status s) {
  switch (s) {
    case SCALE_OK: return "ok";
    case SCALE_ERR_INVALID_ARG: return "invalid argument";
    case SCALE_ERR_UNSUPPORTED: return "unsupported configuration";
    case SCALE_ERR_OUT_OF_MEMORY: return "out of device or pinned memory";
    case SCALE_ERR_CAPACITY: return "size above the capacity given to scale_init";
    case SCALE_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

scale_status scale_cluster_geometry(const scale_config* cfg, const scale_variant* variant, int32_t n_tokens,
                                    const int32_t* cluster_start, int32_t n_clusters, int32_t* geo_out) {
  const scale_variant var = variant ? *variant : scale_variant{};
  scale_status st = validate_config(cfg, &var);
  if (st != SCALE_OK) return st;
  if (!geo_out) return SCALE_ERR_INVALID_ARG;
  st = plan_geometry(*cfg, var, n_tokens, cluster_start, n_clusters, nullptr);
  if (st != SCALE_OK) return st;
  std::vector<ClusterGeo> geo(n_clusters);
  plan_geometry(*cfg, var, n_tokens, cluster_start, n_clusters, geo.data());
  for (int j = 0; j < n_clusters; ++j) {
    const ClusterGeo& g = geo[j];
    int32_t* o = geo_out + 6 * j;
    o[0] = g.s; o[1] = g.e; o[2] = g.lo_blk; o[3] = g.sink_eff; o[4] = g.n_cand; o[5] = g.sel_cnt;
  }
  return SCALE_OK;
}

scale_status scale_init(const scale_config* cfg, void* hip_stream, scale_handle* out) {
  return scale_init_variant(cfg, nullptr, hip_stream, out);
}

scale_status scale_init_variant(const scale_config* cfg, const scale_variant* variant, void* hip_stream,
                                scale_handle* out) {
  if (!out) return SCALE_ERR_INVALID_ARG;
  *out = nullptr;
  const scale_variant var = variant ? *variant : scale_variant{};
  scale_status st = validate_config(cfg, &var);
  if (st != SCALE_OK) return st;

  scale_ctx* h = new (std::nothrow) scale_ctx();
  if (!h) return SCALE_ERR_OUT_OF_MEMORY;
  h->cfg = *cfg;
  h->var = var;
  h->stream = reinterpret_cast<hipStream_t>(hip_stream);
  if (hipGetDevice(&h->device) != hipSuccess) { release(h); return SCALE_ERR_HIP; }
  const scale_config& c = h->cfg;
  const scale_variant& v = h->var;
  h->max_blocks = (c.max_tokens + c.block_size - 1) / c.block_size;
  h->max_subchunks = (c.max_tokens + c.sub_chunk - 1) / c.sub_chunk;
  h->max_items = (int)max_work_items(c);
  const int64_t row_elems = (int64_t)c.num_q_heads * c.head_dim;
  const int64_t mc = c.max_clusters;

  auto dev = [&](void** p, size_t bytes) -> bool {
    if (bytes == 0) return true;
    return hipMalloc(p, bytes) == hipSuccess;
  };
  const int64_t chunk_entries = mc * c.num_q_heads * scale::selection_chunks(h->max_blocks);
  const bool blocks = !v.select_tokens;
  bool ok = dev((void**)&h->d_geo, sizeof(ClusterGeo) * mc) &&
            dev((void**)&h->d_items, sizeof(WorkItem) * (size_t)h->max_items) &&
            dev((void**)&h->d_attn_queue, sizeof(uint32_t) * (scale::kAttentionQueues + 1)) &&
            hipMemset(h->d_attn_queue, 0, sizeof(uint32_t) * (scale::kAttentionQueues + 1)) == hipSuccess &&
            dev((void**)&h->d_fingerprints, sizeof(float) * mc * row_elems) &&
            dev((void**)&h->d_fp64, blocks ? sizeof(double) * mc * row_elems : 0) &&
            dev((void**)&h->d_weights, blocks ? sizeof(double) * mc * c.num_q_heads * (int64_t)h->max_blocks : 0) &&
            dev((void**)&h->d_stats, blocks ? sizeof(double2) * chunk_entries : 0) &&
            dev((void**)&h->d_factors, blocks ? sizeof(double) * chunk_entries : 0) &&
            dev((void**)&h->d_spill, blocks && h->max_blocks > 8192
                                         ? sizeof(float) * mc * (v.kv_head_sets ? c.num_kv_heads : 1) * h->max_blocks
                                         : 0) &&
            dev((void**)&h->d_sub_fp, sizeof(double) * (size_t)h->max_subchunks * row_elems) &&
            dev((void**)&h->d_inv_norm, sizeof(double) * (size_t)h->max_subchunks) &&
            dev((void**)&h->d_band, sizeof(double) * (size_t)h->max_subchunks * scale::kMaxClusterSpan) &&
            hipHostMalloc((void**)&h->h_band, sizeof(double) * (size_t)h->max_subchunks * scale::kMaxClusterSpan,
                          hipHostMallocDefault) == hipSuccess;
  if (ok && v.select_tokens) {
    const int group = c.num_q_heads / c.num_kv_heads;
    const int64_t rows = (int64_t)c.num_kv_heads * scale::token_row_pad(c.max_clusters, group);
    h->kpad = (c.top_k + scale::kTokenTile - 1) / scale::kTokenTile * scale::kTokenTile;
    h->tok_stride = ((int64_t)c.max_tokens + scale::kTokenTile - 1) / scale::kTokenTile * scale::kTokenTile;
    const int64_t gathered = mc * c.num_kv_heads * h->kpad * c.head_dim;
    ok = dev((void**)&h->d_tok_F, sizeof(uint16_t) * rows * 2 * c.head_dim) &&
         dev((void**)&h->d_tok_stats, sizeof(float2) * rows * scale::token_chunks(c.max_tokens)) &&
         dev((void**)&h->d_tok_lse, sizeof(float) * rows) &&
         dev((void**)&h->d_tok_partial, sizeof(float) * mc * c.num_kv_heads * h->tok_stride) &&
         dev((void**)&h->d_tok_score, sizeof(float) * mc * h->tok_stride) &&
         dev((void**)&h->d_gk, sizeof(uint16_t) * gathered) && dev((void**)&h->d_gv, sizeof(uint16_t) * gathered);
  }
  if (!ok) {
    (void)hipGetLastError();
    release(h);
    return SCALE_ERR_OUT_OF_MEMORY;
  }
  h->slot_bytes = std::max(sizeof(ClusterGeo) * (size_t)mc, (size_t)256);
  h->geo_dev.resize(mc);
  h->geo_tmp.resize(mc);
  for (auto& s : h->slots) {
    if (hipHostMalloc(&s.host, h->slot_bytes, hipHostMallocDefault) != hipSuccess ||
        hipEventCreateWithFlags(&s.done, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      release(h);
      return SCALE_ERR_OUT_OF_MEMORY;
    }
  }
  *out = h;
  return SCALE_OK;
}

void scale_free(scale_handle h) {
  if (!h) return;
  (void)hipStreamSynchronize(h->stream);
  release(h);
}

scale_status scale_retrieval_calls(scale_handle h, int64_t* calls) {
  if (!h || !calls) return SCALE_ERR_INVALID_ARG;
  *calls = h->retrieval_calls;
  return SCALE_OK;
}

scale_status scale_fingerprints(scale_handle h, float* fingerprints, int32_t n_clusters) {
  if (!h || !fingerprints || n_clusters < 1 || n_clusters > h->last_clusters) return SCALE_ERR_INVALID_ARG;
  const size_t bytes = sizeof(float) * (size_t)n_clusters * h->cfg.num_q_heads * h->cfg.head_dim;
  return hipMemcpyAsync(fingerprints, h->d_fingerprints, bytes, hipMemcpyDeviceToDevice, h->stream) == hipSuccess
             ? SCALE_OK
             : SCALE_ERR_HIP;
}

scale_status scale_rep_keys(scale_handle h, const uint16_t* k_pages, const int32_t* block_table, int32_t n_tokens,
                            float* k_rep) {
  if (!h || !k_pages || !k_rep || n_tokens < 1 || !aligned16(k_pages)) return SCALE_ERR_INVALID_ARG;
  const scale_config& c = h->cfg;
  if (n_tokens % c.block_size) return SCALE_ERR_UNSUPPORTED;
  if (n_tokens > c.max_tokens) return SCALE_ERR_CAPACITY;
  stage_begin(h, SCALE_STAGE_REP_KEYS);
  const hipError_t e = scale::launch_rep_keys(k_pages, block_table, 0, n_tokens / c.block_size, c.num_kv_heads,
                                              c.block_size, c.head_dim, h->var.rep_kind == SCALE_REP_BOUNDS, k_rep,
                                              h->stream);
  stage_end(h, SCALE_STAGE_REP_KEYS);
  return check_launch(e);
}

scale_status scale_rep_keys_range(scale_handle h, const uint16_t* k_pages, const int32_t* block_table,
                                  int32_t first_block, int32_t n_tokens, float* k_rep) {
  if (!h || !k_pages || !k_rep || n_tokens < 1 || first_block < 0 || !aligned16(k_pages)) return SCALE_ERR_INVALID_ARG;
  const scale_config& c = h->cfg;
  if (n_tokens % c.block_size) return SCALE_ERR_UNSUPPORTED;
  if (n_tokens > c.max_tokens) return SCALE_ERR_CAPACITY;
  if (first_block > n_tokens / c.block_size) return SCALE_ERR_INVALID_ARG;
  stage_begin(h, SCALE_STAGE_REP_KEYS);
  const hipError_t e = scale::launch_rep_keys(k_pages, block_table, first_block, n_tokens / c.block_size,
                                              c.num_kv_heads, c.block_size, c.head_dim, h->var.rep_kind == SCALE_REP_BOUNDS,
                                              k_rep, h->stream);
  stage_end(h, SCALE_STAGE_REP_KEYS);
  return check_launch(e);
}

scale_status scale_select_cluster(scale_handle h, const uint16_t* q, int32_t n_tokens, const float* k_rep,
                                  const int32_t* cluster_start, int32_t n_clusters, int32_t* sel_idx,
                                  int32_t* sel_cnt, float* scores_out) {
  if (!h || !q || !k_rep || !sel_idx || !sel_cnt || !aligned16(q) || !aligned16(k_rep)) return SCALE_ERR_INVALID_ARG;
  const scale_config& c = h->cfg;
  const scale_variant& v = h->var;
  if (v.select_tokens) return SCALE_ERR_UNSUPPORTED;
  scale_status st = plan_geometry(c, v, n_tokens, cluster_start, n_clusters, nullptr);
  if (st != SCALE_OK) return st;

  ClusterGeo* geo = h->geo_tmp.data();
  plan_geometry(c, v, n_tokens, cluster_start, n_clusters, geo);
  int max_cand = 0;
  for (int j = 0; j < n_clusters; ++j) max_cand = std::max(max_cand, geo[j].n_cand);
  if ((st = sync_geometry(h, geo, n_clusters)) != SCALE_OK) return st;

  const int n_blocks = n_tokens / c.block_size;
  const int sink_blk = (c.sink_tokens + c.block_size - 1) / c.block_size;
  const double sigma = c.score_scale == 0.f ? 1.0 : (double)c.score_scale;
  stage_begin(h, SCALE_STAGE_FINGERPRINT);
  st = check_launch(scale::launch_fingerprints(q, h->d_geo, n_clusters, c.num_q_heads, c.head_dim, h->d_fingerprints,
                                               h->d_fp64, h->stream));
  stage_end(h, SCALE_STAGE_FINGERPRINT);
  if (st != SCALE_OK) return st;
  h->last_clusters = n_clusters;
  stage_begin(h, SCALE_STAGE_LOGITS);
  st = check_launch(scale::launch_block_logits(h->d_fp64, k_rep, h->d_geo, n_clusters, max_cand, h->max_blocks,
                                               sink_blk, c.num_q_heads, c.num_kv_heads, c.head_dim,
                                               v.rep_kind == SCALE_REP_BOUNDS, sigma, h->d_weights, h->d_stats,
                                               h->stream));
  stage_end(h, SCALE_STAGE_LOGITS);
  if (st != SCALE_OK) return st;
  stage_begin(h, SCALE_STAGE_VOTE_TOPK);
  st = check_launch(scale::launch_vote_topk(h->d_weights, h->d_stats, h->d_factors, h->d_geo, n_clusters, max_cand,
                                            h->max_blocks, sink_blk, c.num_q_heads, c.num_kv_heads,
                                            v.kv_head_sets != 0, c.top_k, n_blocks, h->d_spill, sel_idx, sel_cnt,
                                            scores_out, h->stream));
  stage_end(h, SCALE_STAGE_VOTE_TOPK);
  if (st != SCALE_OK) return st;
  h->retrieval_calls += n_clusters;
  return SCALE_OK;
}

scale_status scale_select_cluster_tokens(scale_handle h, const uint16_t* q, int32_t n_tokens, const uint16_t* k_pages,
                                         const int32_t* block_table, const int32_t* cluster_start, int32_t n_clusters,
                                         int32_t* sel_idx, int32_t* sel_cnt, float* scores_out) {
  if (!h || !q || !k_pages || !sel_idx || !sel_cnt || !aligned16(q) || !aligned16(k_pages)) return SCALE_ERR_INVALID_ARG;
  const scale_config& c = h->cfg;
  const scale_variant& v = h->var;
  if (!v.select_tokens) return SCALE_ERR_UNSUPPORTED;
  scale_status st = plan_geometry(c, v, n_tokens, cluster_start, n_clusters, nullptr);
  if (st != SCALE_OK) return st;

  ClusterGeo* geo = h->geo_tmp.data();
  plan_geometry(c, v, n_tokens, cluster_start, n_clusters, geo);
  int max_cand = 0;
  for (int j = 0; j < n_clusters; ++j) max_cand = std::max(max_cand, geo[j].n_cand);
  if ((st = sync_geometry(h, geo, n_clusters)) != SCALE_OK) return st;

  const int first_token = (c.sink_tokens + c.block_size - 1) / c.block_size * c.block_size;
  const float sigma = c.score_scale == 0.f ? 1.0f : c.score_scale;
  float* fps = h->d_fingerprints;
  stage_begin(h, SCALE_STAGE_FINGERPRINT);
  st = check_launch(scale::launch_fingerprints(q, h->d_geo, n_clusters, c.num_q_heads, c.head_dim, fps, nullptr,
                                               h->stream));
  stage_end(h, SCALE_STAGE_FINGERPRINT);
  if (st != SCALE_OK) return st;
  h->last_clusters = n_clusters;
  stage_begin(h, SCALE_STAGE_LOGITS);
  st = check_launch(scale::launch_token_selection(fps, k_pages, block_table, h->d_geo, n_clusters, max_cand,
                                                  first_token, c.num_q_heads, c.num_kv_heads, c.head_dim,
                                                  c.block_size, sigma, h->tok_stride, h->d_tok_F, h->d_tok_stats,
                                                  h->d_tok_lse, h->d_tok_partial, h->stream));
  stage_end(h, SCALE_STAGE_LOGITS);
  if (st != SCALE_OK) return st;
  stage_begin(h, SCALE_STAGE_VOTE_TOPK);
  st = check_launch(scale::launch_vote_topk_tokens(h->d_tok_partial, h->d_geo, n_clusters, h->tok_stride, max_cand,
                                                   first_token, c.num_kv_heads, v.kv_head_sets != 0, c.top_k,
                                                   n_tokens, h->d_tok_score, sel_idx, sel_cnt, scores_out,
                                                   h->stream));
  stage_end(h, SCALE_STAGE_VOTE_TOPK);
  if (st != SCALE_OK) return st;
  h->retrieval_calls += n_clusters;
  return SCALE_OK;
}

// Width of the cosine band: the largest number of sub-chunks a cluster may hold, minus one.
static int32_t cluster_span(int32_t l_max, int32_t sub_chunk, int32_t outer_subchunks, int32_t m) {
  int64_t cap = ((int64_t)l_max + sub_chunk - 1) / sub_chunk;
  if (outer_subchunks > 0) cap = std::min<int64_t>(cap, outer_subchunks);
  cap = std::min<int64_t>(cap, m);
  return (int32_t)(cap - 1);
}

scale_status scale_cluster_subchunks(scale_handle h, const uint16_t* q, int32_t n_tokens, int32_t first_subchunk,
                                     double theta, int32_t l_max, int32_t outer_subchunks, int32_t* cluster_start,
                                     int32_t* n_clusters, double* cos_band) {
  if (!h || !q || !cluster_start || !n_clusters || !aligned16(q)) return SCALE_ERR_INVALID_ARG;
  if (n_tokens < 1 || std::isnan(theta) || l_max < 1 || outer_subchunks < 0) return SCALE_ERR_INVALID_ARG;
  const scale_config& c = h->cfg;
  if (n_tokens > c.max_tokens) return SCALE_ERR_CAPACITY;
  const int32_t L = c.sub_chunk;
  const int32_t M = (n_tokens + L - 1) / L;
  if (first_subchunk < 0 || first_subchunk >= M) return SCALE_ERR_INVALID_ARG;
  const int32_t m = M - first_subchunk;     // sub-chunks clustered; band rows are indexed from first
  const int32_t span = cluster_span(l_max, L, outer_subchunks, m);
  if (span > scale::kMaxClusterSpan) return SCALE_ERR_UNSUPPORTED;

  stage_begin(h, SCALE_STAGE_CLUSTER);
  scale_status st = check_launch(scale::launch_subchunk_similarity(q, n_tokens, first_subchunk, L, c.num_q_heads,
                                                                   c.head_dim, span, h->d_sub_fp, h->d_inv_norm,
                                                                   h->d_band, h->stream));
  if (st == SCALE_OK && span > 0 &&
      hipMemcpyAsync(h->h_band, h->d_band, sizeof(double) * (size_t)m * span, hipMemcpyDeviceToHost, h->stream) !=
          hipSuccess)
    st = SCALE_ERR_HIP;
  stage_end(h, SCALE_STAGE_CLUSTER);
  if (st != SCALE_OK) return st;
  if (hipStreamSynchronize(h->stream) != hipSuccess) return SCALE_ERR_HIP;

  // Algorithm 1: the open cluster starts at anchor a and admits j while cos(v_a, v_j) >= theta and
  // the cluster holds fewer than ceil(l_max / L) sub-chunks (|C| L < l_max, Eq. 8); it also closes
  // at an outer-chunk boundary. j - a - 1 < span always holds in the loop.
  const int64_t cap = ((int64_t)l_max + L - 1) / L;
  int32_t k = 0;
  int32_t a = first_subchunk;
  while (a < M) {
    cluster_start[k++] = a;
    const int32_t end = outer_subchunks > 0 ? std::min(M, (a / outer_subchunks + 1) * outer_subchunks) : M;
    int64_t size = 1;
    int32_t j = a + 1;
    while (j < end && size < cap && h->h_band[(int64_t)(a - first_subchunk) * span + (j - a - 1)] >= theta) {
      ++size;
      ++j;
    }
    a = j;
  }
  cluster_start[k] = M;
  *n_clusters = k;
  if (cos_band && span > 0) std::memcpy(cos_band, h->h_band, sizeof(double) * (size_t)m * span);
  return SCALE_OK;
}

scale_status scale_sparse_prefill(scale_handle h, const uint16_t* q, const uint16_t* k_pages, const uint16_t* v_pages,
                                  const int32_t* block_table, int32_t n_tokens, const int32_t* cluster_start,
                                  int32_t n_clusters, const int32_t* sel_idx, const int32_t* sel_cnt, void* out) {
  if (!h || !q || !k_pages || !v_pages || !sel_idx || !sel_cnt || !out) return SCALE_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(out)) return SCALE_ERR_INVALID_ARG;
  const scale_config& c = h->cfg;
  const scale_variant& v = h->var;
  scale_status st = plan_geometry(c, v, n_tokens, cluster_start, n_clusters, nullptr);
  if (st != SCALE_OK) return st;

  ClusterGeo* geo = h->geo_tmp.data();
  plan_geometry(c, v, n_tokens, cluster_start, n_clusters, geo);

  // Work list: clusters in order; inside a cluster, position tiles from the last (most keys) to
  // the first; each tile once per (head group, KV head), KV head fastest. Work-groups are handed to
  // the 8 XCDs round-robin, so a KV head stays on the same XCDs (and their L2) while the tiles of
  // one cluster, which share the sink, selected and local K/V blocks, run together. It is built on
  // the device from the geometry, and again only when the geometry changes.
  const int B = c.block_size;
  const int group = c.num_q_heads / c.num_kv_heads;
  const int TP = scale::attention_tile_positions(group, c.head_dim);
  const int HG = scale::attention_head_groups(group, c.head_dim);
  const ClusterGeo& last = geo[n_clusters - 1];
  const int64_t n_items = (int64_t)last.item0 + (int64_t)((last.e - last.s + TP - 1) / TP) * c.num_kv_heads * HG;
  if (n_items > h->max_items) return SCALE_ERR_CAPACITY;
  if ((st = sync_geometry(h, geo, n_clusters)) != SCALE_OK) return st;
  if (!h->items_valid) {
    if ((st = check_launch(scale::launch_build_work_items(h->d_geo, n_clusters, TP, HG, c.num_kv_heads, h->d_items,
                                                          h->stream))) != SCALE_OK)
      return st;
    h->items_valid = true;
  }

  const float scale = c.softmax_scale == 0.f ? 1.0f / std::sqrt((float)c.head_dim) : c.softmax_scale;
  const float qk_scale_log2 = scale * 1.4426950408889634f;
  const bool tokens = v.select_tokens && h->kpad > 0;
  if (tokens) {
    stage_begin(h, SCALE_STAGE_GATHER);
    st = check_launch(scale::launch_gather_selected(k_pages, v_pages, block_table, sel_idx, sel_cnt,
                                                    v.kv_head_sets != 0, n_clusters, c.top_k, h->kpad, n_tokens,
                                                    c.num_kv_heads, c.head_dim, B, h->d_gk, h->d_gv, h->stream));
    stage_end(h, SCALE_STAGE_GATHER);
    if (st != SCALE_OK) return st;
  }
  stage_begin(h, SCALE_STAGE_ATTENTION);
  const hipError_t e = scale::launch_sparse_attention(
      q, k_pages, v_pages, block_table, h->d_geo, h->d_items, (int)n_items, sel_idx, sel_cnt, v.kv_head_sets != 0,
      c.top_k, c.num_q_heads, c.num_kv_heads, c.head_dim, B, n_tokens / B, qk_scale_log2,
      c.out_dtype == SCALE_OUT_BF16, out, tokens ? h->d_gk : nullptr, tokens ? h->d_gv : nullptr, h->kpad,
      h->d_attn_queue, h->stream);
  stage_end(h, SCALE_STAGE_ATTENTION);
  return check_launch(e);
}

scale_status scale_enable_timing(scale_handle h, int enable) {
  return scale_enable_stage_timing(h, enable ? (1u << SCALE_NUM_STAGES) - 1u : 0u);
}

scale_status scale_enable_stage_timing(scale_handle h, uint32_t stage_mask) {
  if (!h || (stage_mask >> SCALE_NUM_STAGES) != 0) return SCALE_ERR_INVALID_ARG;
  h->timing_mask = stage_mask;
  return SCALE_OK;
}

scale_status scale_stage_times(scale_handle h, double* ms, int64_t* launches, int reset) {
  if (!h) return SCALE_ERR_INVALID_ARG;
  if (hipStreamSynchronize(h->stream) != hipSuccess) return SCALE_ERR_HIP;
  for (const TimedLaunch& t : h->timed) {
    float e = 0.f;
    if (hipEventElapsedTime(&e, t.start, t.stop) != hipSuccess) return SCALE_ERR_HIP;
    h->stage_ms[t.stage] += e;
    h->stage_launches[t.stage] += 1;
    h->spare_events.push_back(t.start);
    h->spare_events.push_back(t.stop);
  }
  h->timed.clear();
  for (int i = 0; i < SCALE_NUM_STAGES; ++i) {
    if (ms) ms[i] = h->stage_ms[i];
    if (launches) launches[i] = h->stage_launches[i];
    if (reset) {
      h->stage_ms[i] = 0.0;
      h->stage_launches[i] = 0;
    }
  }
  return SCALE_OK;
}

}  // extern "C"
