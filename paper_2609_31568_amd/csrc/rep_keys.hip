// Representative key of every KV block: the mean of the block's keys, per KV head.
//
// One work-group reduces one (block, KV head) tile: B rows of d bf16 values, contiguous in the
// page (B * d * 2 bytes, 32 KiB at B = d = 128). Each thread streams 16-byte vectors of one
// column chunk down a strided set of rows and accumulates in fp64; the row groups are combined
// in LDS in a fixed order. Sums of bf16 values are exact in fp64 unless the values span more
// than ~2^38 in magnitude, so the result is the fp32 rounding of the exact mean. HBM-bound:
// B * d * 2 bytes read and d * 4 bytes written per tile.
#include "common.h"

namespace scale {
namespace {

constexpr int kThreads = 256;

template <int D, int B>
__global__ __launch_bounds__(kThreads) void rep_keys_kernel(const uint16_t* __restrict__ k_pages,
                                                            const int32_t* __restrict__ block_table,
                                                            int first_block, int num_kv_heads,
                                                            float* __restrict__ k_rep) {
  constexpr int kChunks = D / 8;                 // 16-byte chunks per row
  constexpr int kRowGroups = kThreads / kChunks; // rows handled in parallel
  constexpr int kRowsPerThread = B / kRowGroups; // all of a thread's loads are issued together
  static_assert(B % kRowGroups == 0, "whole rows per thread");
  const int b = first_block + (int)(blockIdx.x / num_kv_heads);
  const int g = blockIdx.x % num_kv_heads;
  const int page = block_table ? block_table[b] : b;
  const uint16_t* tile = k_pages + ((int64_t)page * num_kv_heads + g) * B * D;

  const int chunk = threadIdx.x % kChunks;
  const int rg = threadIdx.x / kChunks;
  double acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0;
  uint4 v[kRowsPerThread];
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u)
    v[u] = *reinterpret_cast<const uint4*>(tile + (int64_t)(rg + u * kRowGroups) * D + chunk * 8);
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u) {
    const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += (double)__uint_as_float(w[i] << 16);
      acc[2 * i + 1] += (double)__uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __shared__ double part[kRowGroups][D];
#pragma unroll
  for (int i = 0; i < 8; ++i) part[rg][chunk * 8 + i] = acc[i];
  __syncthreads();
  if (threadIdx.x < D) {
    double s = 0.0;
#pragma unroll 4
    for (int r = 0; r < kRowGroups; ++r) s += part[r][threadIdx.x];
    k_rep[((int64_t)b * num_kv_heads + g) * D + threadIdx.x] = (float)(s / (double)B);
  }
}

}  // namespace

hipError_t launch_rep_keys(const uint16_t* k_pages, const int32_t* block_table, int first_block, int n_blocks,
                           int num_kv_heads, int block_size, int head_dim, float* k_rep,
                           hipStream_t stream) {
  if (n_blocks <= first_block) return hipSuccess;
  const dim3 grid((unsigned)((int64_t)(n_blocks - first_block) * num_kv_heads));
  if (head_dim == 128 && block_size == 128)
    rep_keys_kernel<128, 128><<<grid, kThreads, 0, stream>>>(k_pages, block_table, first_block, num_kv_heads, k_rep);
  else if (head_dim == 128)
    rep_keys_kernel<128, 64><<<grid, kThreads, 0, stream>>>(k_pages, block_table, first_block, num_kv_heads, k_rep);
  else if (block_size == 128)
    rep_keys_kernel<64, 128><<<grid, kThreads, 0, stream>>>(k_pages, block_table, first_block, num_kv_heads, k_rep);
  else
    rep_keys_kernel<64, 64><<<grid, kThreads, 0, stream>>>(k_pages, block_table, first_block, num_kv_heads, k_rep);
  return hipGetLastError();
}

}  // namespace scale
