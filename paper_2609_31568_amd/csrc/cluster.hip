// Similarity of consecutive sub-chunks for the anchor-based clustering of an outer chunk (paper
// Sec. 5.1.1-5.1.2, Algorithm 1, Eq. 8).
//
//  subchunk_sums   (column slice, sub-chunk) -> fp64 mean of the sub-chunk's query rows, all heads
//                  concatenated (Eq. 6); sums of bf16 values are exact in fp64
//  inv_norms       sub-chunk -> 1 / ||v_i||_2 (fp64, fixed-order reduction)
//  cos_band        (sub-chunk i, offset) -> cos(v_i, v_{i+offset}) = (v_i . v_j) / (||v_i|| ||v_j||) for
//                  offsets 1 .. span, NaN past the last sub-chunk
//
// The linear clustering pass over the band runs on the host (it is O(M) and sequential). All of
// it is fp64, so the threshold decisions match an fp64 evaluation of the definition except within
// a few ulps of theta.
#include <math.h>

#include "common.h"

namespace scale {
namespace {

constexpr int kThreads = 256;
constexpr int kSumThreads = 512;
constexpr int kSumCols = 512;   // columns of the Hq*d row per work-group (64 lanes x 8)

// grid: (column slice, sub-chunk). Lane l of wave w owns 8 columns and sums rows w, w + 8, ...
__global__ __launch_bounds__(kSumThreads) void subchunk_sums(const uint16_t* __restrict__ q, int n_tokens,
                                                             int first_subchunk, int sub_chunk, int row_elems,
                                                             double* __restrict__ fp) {
  constexpr int kWaves = kSumThreads / 64;
  __shared__ double part[kWaves][kSumCols];
  const int i = blockIdx.y;                       // local index: sub-chunk first_subchunk + i
  const int r0 = (first_subchunk + i) * sub_chunk;
  const int n_rows = min(sub_chunk, n_tokens - r0);
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int col = blockIdx.x * kSumCols + lane * 8;
  double acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.0;
  if (col < row_elems) {   // row_elems is a multiple of 64
    const uint16_t* base = q + (int64_t)r0 * row_elems + col;
    for (int r = wave; r < n_rows; r += kWaves) {
      const uint4 v = *reinterpret_cast<const uint4*>(base + (int64_t)r * row_elems);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        acc[2 * k] += (double)__uint_as_float(w[k] << 16);
        acc[2 * k + 1] += (double)__uint_as_float(w[k] & 0xFFFF0000u);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) part[wave][lane * 8 + k] = acc[k];
  __syncthreads();
  const int c = blockIdx.x * kSumCols + threadIdx.x;
  if (threadIdx.x < kSumCols && c < row_elems) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += part[w][threadIdx.x];
    fp[(int64_t)i * row_elems + c] = s / (double)n_rows;
  }
}

// Fixed-order sum of one double per thread over the work-group (kThreads = 256).
__device__ inline double block_sum_f64(double v, double* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();
  if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// grid: sub-chunk.
__global__ __launch_bounds__(kThreads) void inv_norms(const double* __restrict__ fp, int row_elems,
                                                     double* __restrict__ inv) {
  __shared__ double red[4];
  const double* v = fp + (int64_t)blockIdx.x * row_elems;
  double s = 0.0;
  for (int c = threadIdx.x; c < row_elems; c += kThreads) s = fma(v[c], v[c], s);
  s = block_sum_f64(s, red);
  if (threadIdx.x == 0) inv[blockIdx.x] = 1.0 / sqrt(s);   // inf for a zero fingerprint
}

// grid: (offset - 1, sub-chunk). band[i][offset - 1] = cos(v_i, v_{i + offset}).
__global__ __launch_bounds__(kThreads) void cos_band(const double* __restrict__ fp, const double* __restrict__ inv,
                                                     int m, int row_elems, int span, double* __restrict__ band) {
  __shared__ double red[4];
  const int i = blockIdx.y;
  const int j = i + 1 + blockIdx.x;
  double* dst = band + (int64_t)i * span + blockIdx.x;
  if (j >= m) {
    if (threadIdx.x == 0) *dst = __builtin_nan("");
    return;                                              // uniform over the work-group
  }
  const double* a = fp + (int64_t)i * row_elems;
  const double* b = fp + (int64_t)j * row_elems;
  double s = 0.0;
  for (int c = threadIdx.x; c < row_elems; c += kThreads) s = fma(a[c], b[c], s);
  s = block_sum_f64(s, red);
  if (threadIdx.x == 0) *dst = s * inv[i] * inv[j];     // NaN when either fingerprint is zero
}

}  // namespace

hipError_t launch_subchunk_similarity(const uint16_t* q, int n_tokens, int first_subchunk, int sub_chunk,
                                      int num_q_heads, int head_dim, int span, double* fingerprints,
                                      double* inv_norm, double* band, hipStream_t stream) {
  const int m = (n_tokens + sub_chunk - 1) / sub_chunk - first_subchunk;
  if (m <= 0) return hipSuccess;
  const int row_elems = num_q_heads * head_dim;
  subchunk_sums<<<dim3((row_elems + kSumCols - 1) / kSumCols, m), kSumThreads, 0, stream>>>(
      q, n_tokens, first_subchunk, sub_chunk, row_elems, fingerprints);
  inv_norms<<<m, kThreads, 0, stream>>>(fingerprints, row_elems, inv_norm);
  if (span > 0)
    cos_band<<<dim3(span, m), kThreads, 0, stream>>>(fingerprints, inv_norm, m, row_elems, span, band);
  return hipGetLastError();
}

}  // namespace scale
