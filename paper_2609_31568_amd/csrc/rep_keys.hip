// Representative key of every KV block: the mean of the block's keys, per KV head; or, for the
// bound form of block scoring, the channel-wise minimum and maximum of the block's keys (the
// page criticality bounds of Quest, cited in paper Sec. 2), exact since every key is a bf16 value.
//
// One work-group reduces one (block, KV head) tile: B rows of d bf16 values, contiguous in the
// page (B * d * 2 bytes, 32 KiB at B = d = 128). Each thread streams 16-byte vectors of one
// column chunk down a strided set of rows and accumulates in fp64; the row groups are combined
// in LDS in a fixed order. Sums of bf16 values are exact in fp64 unless the values span more
// than ~2^38 in magnitude, so the result is the fp32 rounding of the exact mean. HBM-bound:
// B * d * 2 bytes read and d * 4 bytes written per tile.
#include <math.h>

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

// Bound form: k_rep[b][g][0][:] = channel-wise minimum, k_rep[b][g][1][:] = maximum; same tile
// walk, fp32 min / max (exact), row groups combined in LDS.
template <int D, int B>
__global__ __launch_bounds__(kThreads) void rep_bounds_kernel(const uint16_t* __restrict__ k_pages,
                                                              const int32_t* __restrict__ block_table,
                                                              int first_block, int num_kv_heads,
                                                              float* __restrict__ k_rep) {
  constexpr int kChunks = D / 8;
  constexpr int kRowGroups = kThreads / kChunks;
  constexpr int kRowsPerThread = B / kRowGroups;
  static_assert(B % kRowGroups == 0, "whole rows per thread");
  const int b = first_block + (int)(blockIdx.x / num_kv_heads);
  const int g = blockIdx.x % num_kv_heads;
  const int page = block_table ? block_table[b] : b;
  const uint16_t* tile = k_pages + ((int64_t)page * num_kv_heads + g) * B * D;

  const int chunk = threadIdx.x % kChunks;
  const int rg = threadIdx.x / kChunks;
  float lo[8], hi[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    lo[i] = INFINITY;
    hi[i] = -INFINITY;
  }
  uint4 v[kRowsPerThread];
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u)
    v[u] = *reinterpret_cast<const uint4*>(tile + (int64_t)(rg + u * kRowGroups) * D + chunk * 8);
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u) {
    const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a = __uint_as_float(w[i] << 16), c = __uint_as_float(w[i] & 0xFFFF0000u);
      lo[2 * i] = fminf(lo[2 * i], a);
      hi[2 * i] = fmaxf(hi[2 * i], a);
      lo[2 * i + 1] = fminf(lo[2 * i + 1], c);
      hi[2 * i + 1] = fmaxf(hi[2 * i + 1], c);
    }
  }
  __shared__ float part[2][kRowGroups][D];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    part[0][rg][chunk * 8 + i] = lo[i];
    part[1][rg][chunk * 8 + i] = hi[i];
  }
  __syncthreads();
  if (threadIdx.x < 2 * D) {
    const int which = threadIdx.x / D, col = threadIdx.x % D;
    float r = part[which][0][col];
    for (int k = 1; k < kRowGroups; ++k) r = which ? fmaxf(r, part[1][k][col]) : fminf(r, part[0][k][col]);
    k_rep[(((int64_t)b * num_kv_heads + g) * 2 + which) * D + col] = r;
  }
}

template <int D, int B>
void launch_db(bool bounds, dim3 grid, const uint16_t* k_pages, const int32_t* block_table, int first_block,
               int num_kv_heads, float* k_rep, hipStream_t stream) {
  if (bounds)
    rep_bounds_kernel<D, B><<<grid, kThreads, 0, stream>>>(k_pages, block_table, first_block, num_kv_heads, k_rep);
  else
    rep_keys_kernel<D, B><<<grid, kThreads, 0, stream>>>(k_pages, block_table, first_block, num_kv_heads, k_rep);
}

}  // namespace

hipError_t launch_rep_keys(const uint16_t* k_pages, const int32_t* block_table, int first_block, int n_blocks,
                           int num_kv_heads, int block_size, int head_dim, bool bounds, float* k_rep,
                           hipStream_t stream) {
  if (n_blocks <= first_block) return hipSuccess;
  const dim3 grid((unsigned)((int64_t)(n_blocks - first_block) * num_kv_heads));
  if (head_dim == 128 && block_size == 128)
    launch_db<128, 128>(bounds, grid, k_pages, block_table, first_block, num_kv_heads, k_rep, stream);
  else if (head_dim == 128)
    launch_db<128, 64>(bounds, grid, k_pages, block_table, first_block, num_kv_heads, k_rep, stream);
  else if (block_size == 128)
    launch_db<64, 128>(bounds, grid, k_pages, block_table, first_block, num_kv_heads, k_rep, stream);
  else
    launch_db<64, 64>(bounds, grid, k_pages, block_table, first_block, num_kv_heads, k_rep, stream);
  return hipGetLastError();
}

}  // namespace scale
