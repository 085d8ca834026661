// The attention work list, built on the device from the cluster geometry (the order the attention
// kernel's XCD-aware schedule relies on; see launch_build_work_items in common.h).
#include "common.h"

namespace scale {
namespace {

// grid: one work-group per cluster; the items of cluster j in the order of the work list.
__global__ __launch_bounds__(256) void build_work_items_kernel(const ClusterGeo* __restrict__ geo, int tile_positions,
                                                               int head_groups, int num_kv_heads,
                                                               WorkItem* __restrict__ items) {
  const int j = blockIdx.x;
  const ClusterGeo g = geo[j];
  const int n_tiles = (g.e - g.s + tile_positions - 1) / tile_positions;
  const int per_tile = head_groups * num_kv_heads;
  for (int i = threadIdx.x; i < n_tiles * per_tile; i += blockDim.x) {
    const int p0 = g.s + (n_tiles - 1 - i / per_tile) * tile_positions;
    const int rem = i % per_tile;
    items[g.item0 + i] = {j, (rem % num_kv_heads) | ((rem / num_kv_heads) << 16), p0, min(tile_positions, g.e - p0)};
  }
}

}  // namespace

hipError_t launch_build_work_items(const ClusterGeo* geo, int n_clusters, int tile_positions, int head_groups,
                                   int num_kv_heads, WorkItem* items, hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  build_work_items_kernel<<<n_clusters, 256, 0, stream>>>(geo, tile_positions, head_groups, num_kv_heads, items);
  return hipGetLastError();
}

}  // namespace scale
