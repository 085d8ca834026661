// scale_select_cluster_static: the cluster-level selection of scale_select_cluster for callers that
// cannot allocate device memory. No handle: the scratch of the selection kernels (cluster geometry,
// fingerprints, per-chunk weights and softmax partials, chunk factors, top-k spill) lives in one
// file-scope device array of kStaticScratchBytes, and the cluster geometry is computed on the
// device from the cluster boundaries passed by value as kernel arguments, so the call needs no
// host staging buffer and no copy either. The kernels are the ones the handle path launches.
//
// Each device the library runs on holds its own copy of the array for the life of the process.
// Its device address is taken once per device with hipGetSymbolAddress, with that device current,
// and only that address is handed to kernels (the array's name in host code is not a device
// address). Calls on one device share the array: calls that overlap in time on one device race.
// No kernel of the selection needs zeroed scratch (every entry is written before it is read), so
// nothing is cleared between calls.
#include <algorithm>
#include <mutex>

#include "common.h"
#include "scale.h"

namespace scale {
namespace {

constexpr size_t kStaticScratchBytes = size_t(64) << 20;   // 64 MiB
constexpr int kMaxDevices = 64;
constexpr int kGeoArgClusters = 512;    // cluster boundaries per geometry launch (by value)
constexpr int kCandInLds = 8192;        // larger candidate counts spill the scores to scratch

__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

struct GeoArgs {
  int32_t first, count;                 // clusters [first, first + count) of this launch
  int32_t n_tokens, sub_chunk, block_size, sink_tokens, local_window, top_k;
  int32_t starts[kGeoArgClusters + 1];  // cluster_start[first .. first + count]
};

// The per-cluster geometry of include/scale.h (block-level selection), one thread per cluster.
__global__ __launch_bounds__(256) void geometry_kernel(GeoArgs a, ClusterGeo* __restrict__ geo) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= a.count) return;
  const int B = a.block_size;
  const int sink_blk = (a.sink_tokens + B - 1) / B;
  ClusterGeo g;
  g.s = (int32_t)((int64_t)a.starts[i] * a.sub_chunk);
  g.e = (int32_t)min((int64_t)a.starts[i + 1] * a.sub_chunk, (int64_t)a.n_tokens);
  g.anchor_end = min(g.s + a.sub_chunk, g.e);
  const int lo = max(0, min(g.s, g.e - a.local_window));
  g.lo_blk = lo / B;
  g.sink_eff = min(sink_blk, g.lo_blk);
  g.n_cand = max(0, g.lo_blk - sink_blk);
  g.sel_cnt = min(a.top_k, g.n_cand);
  g.item0 = 0;
  geo[a.first + i] = g;
}

std::mutex g_scratch_mutex;
unsigned char* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch, taken once per device with the device current.
scale_status device_scratch(unsigned char** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SCALE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SCALE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SCALE_ERR_HIP;
    g_scratch_ptr[dev] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return SCALE_OK;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace
}  // namespace scale

extern "C" scale_status scale_select_cluster_static(const scale_config* cfg, void* hip_stream, const uint16_t* q,
                                                    int32_t n_tokens, const float* k_rep,
                                                    const int32_t* cluster_start, int32_t n_clusters,
                                                    int32_t* sel_idx, int32_t* sel_cnt, float* scores_out) {
  using namespace scale;
  // Host validation (the rules of scale_init and scale_select_cluster), before any HIP call.
  if (!q || !k_rep || !sel_idx || !sel_cnt) return SCALE_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k_rep)) & 15u) return SCALE_ERR_INVALID_ARG;
  const scale_variant v{};
  scale_status st = validate_config(cfg, &v);
  if (st != SCALE_OK) return st;
  const scale_config& c = *cfg;
  if ((st = plan_geometry(c, v, n_tokens, cluster_start, n_clusters, nullptr)) != SCALE_OK) return st;
  const int B = c.block_size;
  const int sink_blk = (c.sink_tokens + B - 1) / B;
  int max_cand = 0;                     // the host needs only the largest candidate count
  for (int j = 0; j < n_clusters; ++j) {
    const int64_t s = (int64_t)cluster_start[j] * c.sub_chunk;
    const int64_t e = std::min<int64_t>((int64_t)cluster_start[j + 1] * c.sub_chunk, n_tokens);
    const int64_t lo = std::max<int64_t>(0, std::min<int64_t>(s, e - c.local_window));
    max_cand = std::max(max_cand, (int)std::max<int64_t>(0, lo / B - sink_blk));
  }

  // Scratch layout of this call (256-byte aligned pieces); above the array's size the call is
  // rejected.
  const int n_blocks = n_tokens / B;
  const int64_t row_elems = (int64_t)c.num_q_heads * c.head_dim;
  const int64_t chunk_entries = (int64_t)n_clusters * c.num_q_heads * selection_chunks(max_cand);
  const size_t off_geo = 0;
  const size_t off_fp32 = off_geo + align256(sizeof(ClusterGeo) * n_clusters);
  const size_t off_fp64 = off_fp32 + align256(sizeof(float) * n_clusters * row_elems);
  const size_t off_weights = off_fp64 + align256(sizeof(double) * n_clusters * row_elems);
  const size_t off_stats = off_weights + align256(sizeof(double) * n_clusters * c.num_q_heads * (size_t)n_blocks);
  const size_t off_factors = off_stats + align256(sizeof(double2) * chunk_entries);
  const size_t off_spill = off_factors + align256(sizeof(double) * chunk_entries);
  const size_t total = off_spill + (n_blocks > kCandInLds ? align256(sizeof(float) * n_clusters * (size_t)n_blocks) : 0);
  if (total > kStaticScratchBytes) return SCALE_ERR_CAPACITY;

  unsigned char* base = nullptr;
  st = device_scratch(&base);
  if (st != SCALE_OK) return st;
  hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
  ClusterGeo* geo = reinterpret_cast<ClusterGeo*>(base + off_geo);
  float* fp32 = reinterpret_cast<float*>(base + off_fp32);
  double* fp64 = reinterpret_cast<double*>(base + off_fp64);
  double* weights = reinterpret_cast<double*>(base + off_weights);
  double2* stats = reinterpret_cast<double2*>(base + off_stats);
  double* factors = reinterpret_cast<double*>(base + off_factors);
  float* spill = n_blocks > kCandInLds ? reinterpret_cast<float*>(base + off_spill) : nullptr;

  for (int first = 0; first < n_clusters; first += kGeoArgClusters) {
    GeoArgs a{};
    a.first = first;
    a.count = std::min(kGeoArgClusters, n_clusters - first);
    a.n_tokens = n_tokens;
    a.sub_chunk = c.sub_chunk;
    a.block_size = B;
    a.sink_tokens = c.sink_tokens;
    a.local_window = c.local_window;
    a.top_k = c.top_k;
    for (int i = 0; i <= a.count; ++i) a.starts[i] = cluster_start[first + i];
    geometry_kernel<<<(a.count + 255) / 256, 256, 0, stream>>>(a, geo);
    if (hipGetLastError() != hipSuccess) return SCALE_ERR_HIP;
  }
  const double sigma = c.score_scale == 0.f ? 1.0 : (double)c.score_scale;
  if (launch_fingerprints(q, geo, n_clusters, c.num_q_heads, c.head_dim, fp32, fp64, stream) != hipSuccess ||
      launch_block_logits(fp64, k_rep, geo, n_clusters, max_cand, n_blocks, sink_blk, c.num_q_heads, c.num_kv_heads,
                          c.head_dim, false, sigma, weights, stats, stream) != hipSuccess ||
      launch_vote_topk(weights, stats, factors, geo, n_clusters, max_cand, n_blocks, sink_blk, c.num_q_heads,
                       c.num_kv_heads, false, c.top_k, n_blocks, spill, sel_idx, sel_cnt, scores_out,
                       stream) != hipSuccess)
    return SCALE_ERR_HIP;
  return SCALE_OK;
}
