// Cluster-level block selection: anchor fingerprints, per-head logits, head soft-voting and a
// deterministic top-k, once per cluster (paper Sec. 5.1.3, Eq. 9 and the head soft-voting
// instantiation of the selection function).
//
//  fingerprint_partial  (cluster, row chunk) -> fp64 column sums of the anchor rows, all heads
//  fingerprint_final    cluster -> fp32 mean = fixed-order sum of the partials / anchor length
//  block_logits         (cluster, candidate chunk) -> x[h][c] = sigma * v[h] . k_rep[c][g(h)]
//  vote_topk            cluster -> per-head softmax over candidates, sum over heads, top-k by
//                       (score desc, block index asc), emitted ascending
//
// All of it is HBM/L2-bandwidth work (a few FLOP per byte); every reduction has a fixed order,
// so two runs give identical bits.
#include <float.h>

#include "common.h"

namespace scale {
namespace {

constexpr int kThreads = 256;
constexpr int kFpRowsPerChunk = 64;   // anchor rows per fingerprint_partial work-group

// grid: (row chunk, cluster); each thread owns 8 consecutive columns of the Hq*d row.
__global__ __launch_bounds__(kThreads) void fingerprint_partial(const uint16_t* __restrict__ q,
                                                                const ClusterGeo* __restrict__ geo,
                                                                int row_elems, int fp_chunks,
                                                                double* __restrict__ partial) {
  const int j = blockIdx.y;
  const int chunk = blockIdx.x;
  const ClusterGeo G = geo[j];
  const int r0 = G.s + chunk * kFpRowsPerChunk;
  const int r1 = min(G.anchor_end, r0 + kFpRowsPerChunk);
  double* dst = partial + ((int64_t)j * fp_chunks + chunk) * row_elems;
  for (int c0 = threadIdx.x * 8; c0 < row_elems; c0 += kThreads * 8) {
    double acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.0;
    for (int r = r0; r < r1; ++r) {
      const uint4 v = *reinterpret_cast<const uint4*>(q + (int64_t)r * row_elems + c0);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += (double)__uint_as_float(w[i] << 16);
        acc[2 * i + 1] += (double)__uint_as_float(w[i] & 0xFFFF0000u);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) dst[c0 + i] = acc[i];
  }
}

// grid: cluster; sums the partials of its chunks in chunk order.
__global__ __launch_bounds__(kThreads) void fingerprint_final(const double* __restrict__ partial,
                                                              const ClusterGeo* __restrict__ geo,
                                                              int row_elems, int fp_chunks,
                                                              float* __restrict__ fingerprints) {
  const int j = blockIdx.x;
  const ClusterGeo G = geo[j];
  const int n_rows = G.anchor_end - G.s;
  const int used = (n_rows + kFpRowsPerChunk - 1) / kFpRowsPerChunk;
  const double* src = partial + (int64_t)j * fp_chunks * row_elems;
  for (int c = threadIdx.x; c < row_elems; c += kThreads) {
    double s = 0.0;
    for (int k = 0; k < used; ++k) s += src[(int64_t)k * row_elems + c];
    fingerprints[(int64_t)j * row_elems + c] = (float)(s / (double)n_rows);
  }
}

// grid: (candidate chunk of 64, cluster). Thread t of the work-group owns candidate
// (chunk * 64 + t % 64) and the KV heads g = t / 64, t / 64 + 4, ...; it forms the dot products
// of k_rep[b][g] with the fingerprints of the query heads reading KV head g.
template <int D>
__global__ __launch_bounds__(kThreads) void block_logits_kernel(
    const float* __restrict__ fingerprints, const float* __restrict__ k_rep,
    const ClusterGeo* __restrict__ geo, int cand_stride, int sink_blk, int num_q_heads,
    int num_kv_heads, float score_scale, float* __restrict__ logits) {
  extern __shared__ float v_lds[];                  // [Hq][D] fingerprints of this cluster
  const int j = blockIdx.y;
  const ClusterGeo G = geo[j];
  const int c = blockIdx.x * 64 + threadIdx.x % 64;
  if (blockIdx.x * 64 >= G.n_cand) return;          // uniform over the work-group
  const int row_elems = num_q_heads * D;
  for (int i = threadIdx.x; i < row_elems; i += kThreads) v_lds[i] = fingerprints[(int64_t)j * row_elems + i];
  __syncthreads();
  if (c >= G.n_cand) return;
  const int group = num_q_heads / num_kv_heads;
  const int b = sink_blk + c;
  for (int g = threadIdx.x / 64; g < num_kv_heads; g += kThreads / 64) {
    const float4* kr = reinterpret_cast<const float4*>(k_rep + ((int64_t)b * num_kv_heads + g) * D);
    for (int h0 = 0; h0 < group; h0 += 4) {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      const int nh = min(4, group - h0);
      for (int i = 0; i < D / 4; ++i) {
        const float4 k4 = kr[i];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (u < nh) {
            const float* v = v_lds + (g * group + h0 + u) * D + 4 * i;
            acc[u] = fmaf(v[0], k4.x, acc[u]);
            acc[u] = fmaf(v[1], k4.y, acc[u]);
            acc[u] = fmaf(v[2], k4.z, acc[u]);
            acc[u] = fmaf(v[3], k4.w, acc[u]);
          }
        }
      }
      for (int u = 0; u < nh; ++u)
        logits[((int64_t)j * num_q_heads + g * group + h0 + u) * cand_stride + c] = score_scale * acc[u];
    }
  }
}

// ---- block-wide helpers with a fixed reduction order ----
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
// Block-wide reductions for kThreads = 256 (4 waves); `red` holds 4 floats / ints.
__device__ inline float block_max(float v, float* red) {
  v = wave_max(v);
  __syncthreads();
  if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
__device__ inline float block_sum(float v, float* red) {
  v = wave_sum(v);
  __syncthreads();
  if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}
// Exclusive prefix sum over threads in thread order; returns the total through *total.
__device__ inline int block_exclusive_scan(int v, int* red, int* total) {
  const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  __syncthreads();
  if (lane == 63) red[wave] = incl;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += red[w];
  *total = red[0] + red[1] + red[2] + red[3];
  return before + incl - v;
}

// grid: cluster. Scores live in LDS when n_cand fits, else in `spill` (global, per cluster).
constexpr int kMaxLdsCand = 8192;

__global__ __launch_bounds__(kThreads) void vote_topk_kernel(
    const float* __restrict__ logits, const ClusterGeo* __restrict__ geo, int cand_stride,
    int sink_blk, int num_q_heads, int top_k, int n_blocks, float* __restrict__ spill,
    int32_t* __restrict__ sel_idx, int32_t* __restrict__ sel_cnt, float* __restrict__ scores_out) {
  __shared__ float score_lds[kMaxLdsCand];
  __shared__ float red_f[4];
  __shared__ int red_i[4];
  __shared__ unsigned hist[256];
  const int j = blockIdx.x;
  const ClusterGeo G = geo[j];
  const int n = G.n_cand;
  const int cnt = G.sel_cnt;
  float* score = n <= kMaxLdsCand ? score_lds : spill + (int64_t)j * cand_stride;
  const float* x = logits + (int64_t)j * num_q_heads * cand_stride;

  // 1. soft-voting: per-head max and normaliser, then the sum over heads, head order fixed.
  for (int c = threadIdx.x; c < n; c += kThreads) score[c] = 0.f;
  for (int h = 0; h < num_q_heads; ++h) {
    const float* xh = x + (int64_t)h * cand_stride;
    float m = -FLT_MAX;
    for (int c = threadIdx.x; c < n; c += kThreads) m = fmaxf(m, xh[c]);
    m = block_max(m, red_f);
    float s = 0.f;
    for (int c = threadIdx.x; c < n; c += kThreads) s += expf(xh[c] - m);
    s = block_sum(s, red_f);
    const float inv = 1.0f / s;
    for (int c = threadIdx.x; c < n; c += kThreads) score[c] += expf(xh[c] - m) * inv;
  }
  __syncthreads();
  if (scores_out) {
    float* so = scores_out + (int64_t)j * n_blocks;
    for (int b = threadIdx.x; b < n_blocks; b += kThreads) {
      const int c = b - sink_blk;
      so[b] = (c >= 0 && c < n) ? score[c] : -1.0f;
    }
  }
  int32_t* out = sel_idx + (int64_t)j * top_k;
  if (threadIdx.x == 0) sel_cnt[j] = cnt;

  // 2. threshold: the cnt-th largest score (scores are >= 0, so their bit patterns order like
  //    their values). Radix select, 8 bits per pass, most significant first.
  unsigned prefix = 0, prefix_mask = 0;
  int want = cnt;             // rank (1-based) of the threshold among the still-matching values
  if (cnt > 0 && cnt < n) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = threadIdx.x; i < 256; i += kThreads) hist[i] = 0;
      __syncthreads();
      for (int c = threadIdx.x; c < n; c += kThreads) {
        const unsigned u = __float_as_uint(score[c]);
        if ((u & prefix_mask) == prefix) atomicAdd(&hist[(u >> shift) & 0xFF], 1u);
      }
      __syncthreads();
      // walk the digits from the top; every thread does the same 256-step walk
      int acc = 0, digit = 0;
      for (int dgt = 255; dgt >= 0; --dgt) {
        const int hcount = (int)hist[dgt];
        if (acc + hcount >= want) { digit = dgt; break; }
        acc += hcount;
      }
      want -= acc;
      prefix |= (unsigned)digit << shift;
      prefix_mask |= 0xFFu << shift;
      __syncthreads();
    }
  }
  const unsigned thr = prefix;   // bit pattern of the threshold value (valid when 0 < cnt < n)

  // 3. selected = (score > thr) or (score == thr and among the first `want` ties in index order).
  //    Thread t owns a contiguous index range, so prefix sums follow index order.
  const int per = (n + kThreads - 1) / kThreads;
  const int c0 = min(n, threadIdx.x * per), c1 = min(n, c0 + per);
  int n_tie = 0, n_sel_local = 0;
  if (cnt >= n) {
    n_sel_local = c1 - c0;
  } else if (cnt > 0) {
    for (int c = c0; c < c1; ++c) n_tie += (__float_as_uint(score[c]) == thr);
  }
  int tie_total = 0;
  const int tie_before = block_exclusive_scan(n_tie, red_i, &tie_total);
  if (cnt > 0 && cnt < n) {
    int ties_seen = tie_before;
    for (int c = c0; c < c1; ++c) {
      const unsigned u = __float_as_uint(score[c]);
      if (u > thr) ++n_sel_local;
      else if (u == thr && ties_seen++ < want) ++n_sel_local;
    }
  }
  int sel_total = 0;
  int pos = block_exclusive_scan(n_sel_local, red_i, &sel_total);
  if (cnt > 0) {
    int ties_seen = tie_before;
    for (int c = c0; c < c1; ++c) {
      bool take;
      if (cnt >= n) {
        take = true;
      } else {
        const unsigned u = __float_as_uint(score[c]);
        take = u > thr || (u == thr && ties_seen++ < want);
      }
      if (take) out[pos++] = sink_blk + c;
    }
  }
  for (int i = cnt + threadIdx.x; i < top_k; i += kThreads) out[i] = -1;
}

}  // namespace

hipError_t launch_fingerprints(const uint16_t* q, const ClusterGeo* geo, int n_clusters,
                               int num_q_heads, int head_dim, int sub_chunk, int fp_chunks,
                               double* partial, float* fingerprints, hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  (void)sub_chunk;
  const int row_elems = num_q_heads * head_dim;
  fingerprint_partial<<<dim3(fp_chunks, n_clusters), kThreads, 0, stream>>>(q, geo, row_elems, fp_chunks,
                                                                            partial);
  fingerprint_final<<<n_clusters, kThreads, 0, stream>>>(partial, geo, row_elems, fp_chunks, fingerprints);
  return hipGetLastError();
}

int fingerprint_chunks(int sub_chunk) { return (sub_chunk + kFpRowsPerChunk - 1) / kFpRowsPerChunk; }

hipError_t launch_block_logits(const float* fingerprints, const float* k_rep, const ClusterGeo* geo,
                               int n_clusters, int max_cand, int cand_stride, int sink_blk,
                               int num_q_heads, int num_kv_heads, int head_dim, float score_scale,
                               float* logits, hipStream_t stream) {
  if (n_clusters <= 0 || max_cand <= 0) return hipSuccess;
  const dim3 grid((max_cand + 63) / 64, n_clusters);
  const size_t lds = (size_t)num_q_heads * head_dim * sizeof(float);
  if (head_dim == 128)
    block_logits_kernel<128><<<grid, kThreads, lds, stream>>>(fingerprints, k_rep, geo, cand_stride, sink_blk,
                                                             num_q_heads, num_kv_heads, score_scale, logits);
  else
    block_logits_kernel<64><<<grid, kThreads, lds, stream>>>(fingerprints, k_rep, geo, cand_stride, sink_blk,
                                                            num_q_heads, num_kv_heads, score_scale, logits);
  return hipGetLastError();
}

hipError_t launch_vote_topk(const float* logits, const ClusterGeo* geo, int n_clusters, int cand_stride,
                            int sink_blk, int num_q_heads, int top_k, int n_blocks, float* spill,
                            int32_t* sel_idx, int32_t* sel_cnt, float* scores_out, hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  vote_topk_kernel<<<n_clusters, kThreads, 0, stream>>>(logits, geo, cand_stride, sink_blk, num_q_heads, top_k,
                                                        n_blocks, spill, sel_idx, sel_cnt, scores_out);
  return hipGetLastError();
}

}  // namespace scale
