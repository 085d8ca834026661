// Cluster-level block selection: anchor fingerprints, per-head logits, head soft-voting and a
// deterministic top-k, once per cluster (paper Sec. 5.1.3, Eq. 9 and the head soft-voting
// instantiation of the selection function).
//
//  fingerprint   (column slice, cluster) -> fp32 mean of the anchor rows (fp64 sums)
//  block_logits  (cluster, candidate chunks, KV head) -> x[h][c] = sigma * v[h] . k_rep[c][g(h)]
//                for the query heads h of KV head g (bound form: sigma * sum_i max(v_i mn_i,
//                v_i mx_i) over the block's channel-wise key bounds), plus each chunk's softmax
//                partials (max_c x[h][c], sum_c exp(x[h][c] - max)) per head
//  vote_topk     cluster (or (cluster, KV head) with one set per KV head) -> per-head softmax
//                normaliser from the chunk partials, score = sum over the voting heads of the
//                softmax weights, top-k by (score desc, index asc), ascending; token mode takes
//                the scores of the token scoring kernels (select_tokens.hip)
//  token_sum     (candidate slice, cluster) -> token scores: the per-KV-head partial scores summed
//                in KV-head order
//
// All of it is HBM/L2-bandwidth work (a few FLOP per byte); every reduction has a fixed order,
// so two runs give identical bits.
#include <float.h>

#include <algorithm>

#include "common.h"

namespace scale {
namespace {

constexpr int kThreads = 256;
constexpr int kFpThreads = 512;          // fingerprint: 8 waves
constexpr int kFpCols = 512;             // columns of the Hq*d row per fingerprint work-group
constexpr int kFpRowsInFlight = 4;       // 16-byte loads in flight per lane
constexpr int kCandChunk = 64;           // candidates per block_logits step
constexpr int kLogitsTargetGroups = 4096;

// grid: (column slice, cluster). Lane l of wave w owns the 8 columns [slice*512 + 8l, +8) and
// sums anchor rows w, w+8, w+16, ... in fp64 (exact for bf16 inputs of moderate range); the 8
// waves' sums are combined in LDS in wave order and divided once.
__global__ __launch_bounds__(kFpThreads) void fingerprint_kernel(const uint16_t* __restrict__ q,
                                                                 const ClusterGeo* __restrict__ geo,
                                                                 int row_elems, float* __restrict__ fingerprints) {
  constexpr int kWaves = kFpThreads / 64;
  __shared__ double part[kWaves][kFpCols];
  const int j = blockIdx.y;
  const ClusterGeo G = geo[j];
  const int n_rows = G.anchor_end - G.s;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int col = blockIdx.x * kFpCols + lane * 8;
  double acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0;
  if (col < row_elems) {   // row_elems is a multiple of 64, so a lane's 8 columns are all in range
    const uint16_t* base = q + (int64_t)G.s * row_elems + col;
    auto add = [&](const uint4& v) {
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += (double)__uint_as_float(w[i] << 16);
        acc[2 * i + 1] += (double)__uint_as_float(w[i] & 0xFFFF0000u);
      }
    };
    int r = wave;
    for (; r + (kFpRowsInFlight - 1) * kWaves < n_rows; r += kFpRowsInFlight * kWaves) {
      uint4 v[kFpRowsInFlight];
#pragma unroll
      for (int u = 0; u < kFpRowsInFlight; ++u)
        v[u] = *reinterpret_cast<const uint4*>(base + (int64_t)(r + u * kWaves) * row_elems);
#pragma unroll
      for (int u = 0; u < kFpRowsInFlight; ++u) add(v[u]);
    }
    for (; r < n_rows; r += kWaves) add(*reinterpret_cast<const uint4*>(base + (int64_t)r * row_elems));
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) part[wave][lane * 8 + i] = acc[i];
  __syncthreads();
  const int c = blockIdx.x * kFpCols + threadIdx.x;
  if (threadIdx.x < kFpCols && c < row_elems) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += part[w][threadIdx.x];
    fingerprints[(int64_t)j * row_elems + c] = (float)(s / (double)n_rows);
  }
}

// grid: linear over (cluster j, part p, KV head g) with g fastest: work-groups are handed to the
// 8 XCDs round-robin, so one XCD reads one KV head's slice of k_rep from its own L2. The work-group
// takes candidate chunks p, p + parts, ... of cluster j. In a chunk, wave w holds candidates
// [16w, 16w + 16) with four lanes per candidate; lane quarter q loads the float4s {4i + q} of the
// candidate's representative key (64 contiguous bytes per candidate per load), forms partial dot
// products with the fingerprints of the (at most 8) query heads of g held in LDS, and the four
// lanes add their partials.
template <int D, bool kBounds>
__global__ __launch_bounds__(kThreads) void block_logits_kernel(
    const float* __restrict__ fingerprints, const float* __restrict__ k_rep,
    const ClusterGeo* __restrict__ geo, int parts, int n_chunks, int cand_stride, int sink_blk,
    int num_q_heads, int num_kv_heads, float score_scale, float* __restrict__ logits,
    float2* __restrict__ head_stats) {
  constexpr int kVec = D / 16;                      // float4 loads per lane
  __shared__ float4 v_lds[8 * D / 4];               // fingerprints of the query heads of g
  __shared__ float red[kThreads / 64][8];
  const int g = blockIdx.x % num_kv_heads;
  const int rest = blockIdx.x / num_kv_heads;
  const int p = rest % parts;
  const int j = rest / parts;
  const ClusterGeo G = geo[j];
  const int chunks = (G.n_cand + kCandChunk - 1) / kCandChunk;
  if (p >= chunks) return;                          // uniform over the work-group
  const int group = num_q_heads / num_kv_heads;     // <= 8
  const float4* vsrc = reinterpret_cast<const float4*>(fingerprints + ((int64_t)j * num_q_heads + g * group) * D);
  for (int i = threadIdx.x; i < group * D / 4; i += kThreads) v_lds[i] = vsrc[i];
  __syncthreads();
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int q4 = lane & 3;
  for (int chunk = p; chunk < chunks; chunk += parts) {
    const int c = chunk * kCandChunk + wave * 16 + lane / 4;
    const bool valid = c < G.n_cand;
    float4 kv[kVec], kx[kBounds ? kVec : 1];
    const float4* kr = reinterpret_cast<const float4*>(
        k_rep + ((int64_t)(sink_blk + (valid ? c : 0)) * num_kv_heads + g) * (kBounds ? 2 * D : D));
#pragma unroll
    for (int i = 0; i < kVec; ++i) kv[i] = kr[4 * i + q4];               // mean, or the minima
    if constexpr (kBounds) {
#pragma unroll
      for (int i = 0; i < kVec; ++i) kx[i] = kr[D / 4 + 4 * i + q4];    // the maxima
    }
    float x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      x[u] = 0.f;
      if (u < group) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < kVec; ++i) {
          const float4 v = v_lds[u * (D / 4) + 4 * i + q4];
          if constexpr (kBounds) {
            acc += fmaxf(v.x * kv[i].x, v.x * kx[i].x);
            acc += fmaxf(v.y * kv[i].y, v.y * kx[i].y);
            acc += fmaxf(v.z * kv[i].z, v.z * kx[i].z);
            acc += fmaxf(v.w * kv[i].w, v.w * kx[i].w);
          } else {
            acc = fmaf(v.x, kv[i].x, acc);
            acc = fmaf(v.y, kv[i].y, acc);
            acc = fmaf(v.z, kv[i].z, acc);
            acc = fmaf(v.w, kv[i].w, acc);
          }
        }
        acc += __shfl_xor(acc, 1, 64);
        acc += __shfl_xor(acc, 2, 64);
        x[u] = score_scale * acc;
        if (valid && q4 == (u & 3))
          logits[((int64_t)j * num_q_heads + g * group + u) * cand_stride + c] = x[u];
      }
    }
    // softmax partials of this chunk per head: max over its candidates, then sum of exp(x - max)
    float m[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float t = valid ? x[u] : -FLT_MAX;
#pragma unroll
      for (int o = 4; o < 64; o <<= 1) t = fmaxf(t, __shfl_xor(t, o, 64));
      m[u] = t;
    }
    if (lane == 0)
      for (int u = 0; u < group; ++u) red[wave][u] = m[u];
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 8; ++u) m[u] = fmaxf(fmaxf(red[0][u], red[1][u]), fmaxf(red[2][u], red[3][u]));
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float t = (valid && u < group) ? expf(x[u] - m[u]) : 0.f;
#pragma unroll
      for (int o = 4; o < 64; o <<= 1) t += __shfl_xor(t, o, 64);
      if (lane == 0 && u < group) red[wave][u] = t;
    }
    __syncthreads();
    if (threadIdx.x < group) {
      const int u = threadIdx.x;
      const float s = (red[0][u] + red[1][u]) + (red[2][u] + red[3][u]);
      head_stats[((int64_t)j * num_q_heads + g * group + u) * n_chunks + chunk] = make_float2(m[u], s);
    }
    __syncthreads();
  }
}

// ---- vote_topk ----
constexpr int kVoteThreads = 1024;
constexpr int kVoteWaves = kVoteThreads / 64;
constexpr int kMaxLdsCand = 8192;        // scores of larger clusters live in the global spill row
constexpr int kHistBins = 4096;          // radix digits of the first two passes (12 bits)

// Exclusive prefix sum over the work-group's threads in thread order; the total through *total.
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
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kVoteWaves; ++w) {
    before += w < wave ? red[w] : 0;
    all += red[w];
  }
  *total = all;
  return before + incl - v;
}

// grid: output row = cluster, or (cluster, KV head) with one set per KV head (row j * Hkv + g,
// voted by the query heads of g only).
//  1. soft-voting: each head's softmax maximum and normaliser over all candidates, combined from
//     the chunk partials in chunk order; then per candidate the sum over heads, in head order.
//     Token mode (kTok): the per-KV-head partial sums of the token scoring kernel are added in
//     KV-head order instead.
//  2. threshold: the sel_cnt-th largest score, by radix selection on the score bits (scores are
//     >= 0, so their bit patterns order like their values and the sign bit is 0) in three passes
//     over bits 30-19, 18-7 and 6-0; wide first digits spread the scores of a cluster, which share
//     few exponents, over many histogram bins. The digit is found with a prefix sum over the
//     histogram in descending digit order.
//  3. selected = score above the threshold, or equal to it and among the first ties in index
//     order; written in ascending index order by an ordered compaction.
struct VoteArgs {
  const float* logits;         // block mode: [cluster][Hq][cand_stride]
  const float2* head_stats;    // block mode: [cluster][Hq][n_chunks]
  const float* partial;        // token mode: [cluster][Hkv][cand_stride]
  const ClusterGeo* geo;
  int n_chunks, num_q_heads, num_kv_heads, top_k;
  int64_t cand_stride;
  int first;                   // index of candidate 0 (sink_blk, or sink_blk * B for tokens)
  int n_out;                   // row length of scores_out
  int per_kv;                  // 1: one set per (cluster, KV head), voted by its own query heads
  float* spill;                // [output row][cand_stride]
  int32_t *sel_idx, *sel_cnt;
  float* scores_out;
};

template <bool kTok>
__global__ __launch_bounds__(kVoteThreads) void vote_topk_kernel(VoteArgs a) {
  __shared__ float score_lds[kMaxLdsCand];
  __shared__ int red_i[kVoteWaves];
  __shared__ unsigned hist[kHistBins];
  __shared__ int pick[2];
  extern __shared__ float head_lds[];               // [Hq] maxima, then [Hq] 1 / normaliser
  const int row = blockIdx.x;
  const int sets = a.per_kv ? a.num_kv_heads : 1;
  const int j = row / sets;
  const ClusterGeo G = a.geo[j];
  const int n = G.n_cand;
  const int cnt = G.sel_cnt;
  const int top_k = a.top_k;
  float* score = n <= kMaxLdsCand ? score_lds : a.spill + (int64_t)row * a.cand_stride;

  // 1.
  if constexpr (kTok) {
    // the KV head's own partial row, or the sum over KV heads written by token_sum_kernel
    score = a.per_kv ? const_cast<float*>(a.partial) + (int64_t)row * a.cand_stride
                     : a.spill + (int64_t)j * a.cand_stride;
  } else {
    const int num_q_heads = a.num_q_heads;
    const int group = num_q_heads / a.num_kv_heads;
    const int h0 = a.per_kv ? (row % sets) * group : 0;
    const int h1 = a.per_kv ? h0 + group : num_q_heads;
    const int64_t cand_stride = a.cand_stride;
    const float* x = a.logits + (int64_t)j * num_q_heads * cand_stride;
    const int used = (n + kCandChunk - 1) / kCandChunk;
    for (int h = h0 + (int)threadIdx.x; h < h1; h += kVoteThreads) {
      const float2* st = a.head_stats + ((int64_t)j * num_q_heads + h) * a.n_chunks;
      float m = -FLT_MAX;
      for (int k = 0; k < used; ++k) m = fmaxf(m, st[k].x);
      float s = 0.f;
      for (int k = 0; k < used; ++k) s += st[k].y * expf(st[k].x - m);
      head_lds[h] = m;
      head_lds[num_q_heads + h] = 1.0f / s;
    }
    __syncthreads();
    for (int c = threadIdx.x; c < n; c += kVoteThreads) {
      float acc = 0.f;
      int h = h0;
      for (; h + 16 <= h1; h += 16) {
        float xv[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) xv[u] = x[(int64_t)(h + u) * cand_stride + c];
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += expf(xv[u] - head_lds[h + u]) * head_lds[num_q_heads + h + u];
      }
      for (; h < h1; ++h)
        acc += expf(x[(int64_t)h * cand_stride + c] - head_lds[h]) * head_lds[num_q_heads + h];
      score[c] = acc;
    }
  }
  __syncthreads();
  if (a.scores_out) {
    float* so = a.scores_out + (int64_t)row * a.n_out;
    for (int b = threadIdx.x; b < a.n_out; b += kVoteThreads) {
      const int c = b - a.first;
      so[b] = (c >= 0 && c < n) ? score[c] : -1.0f;
    }
  }
  int32_t* out = a.sel_idx + (int64_t)row * top_k;
  if (threadIdx.x == 0) a.sel_cnt[row] = cnt;

  // f(score bits) for every candidate, in any order. Token mode reads the global score row as
  // float4s (n is a multiple of 64, the row 16-byte aligned) with four loads in flight per thread.
  auto sweep = [&](auto&& f) {
    if constexpr (kTok) {
      const float4* s4 = reinterpret_cast<const float4*>(score);
      const int n4 = n >> 2;
      for (int b = threadIdx.x; b < n4; b += 4 * kVoteThreads) {
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = s4[min(b + u * kVoteThreads, n4 - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (b + u * kVoteThreads < n4) {
            f(__float_as_uint(v[u].x));
            f(__float_as_uint(v[u].y));
            f(__float_as_uint(v[u].z));
            f(__float_as_uint(v[u].w));
          }
        }
      }
    } else {
      for (int c = threadIdx.x; c < n; c += kVoteThreads) f(__float_as_uint(score[c]));
    }
  };
  // f(index, score bits) for the candidates [c0, c1) in index order (token mode: c0, c1 multiples
  // of 4, float4 loads, four in flight).
  auto range_each = [&](int c0, int c1, auto&& f) {
    if constexpr (kTok) {
      const float4* s4 = reinterpret_cast<const float4*>(score);
      for (int c = c0; c < c1; c += 16) {
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = s4[min(c + 4 * u, c1 - 4) >> 2];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (c + 4 * u < c1) {
            f(c + 4 * u, __float_as_uint(v[u].x));
            f(c + 4 * u + 1, __float_as_uint(v[u].y));
            f(c + 4 * u + 2, __float_as_uint(v[u].z));
            f(c + 4 * u + 3, __float_as_uint(v[u].w));
          }
        }
      }
    } else {
      for (int c = c0; c < c1; ++c) f(c, __float_as_uint(score[c]));
    }
  };

  // 2.
  unsigned prefix = 0, prefix_mask = 0;
  int want = cnt;             // rank (1-based) of the threshold among the still-matching values
  if (cnt > 0 && cnt < n) {
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = pass == 0 ? 19 : (pass == 1 ? 7 : 0);
      const int nbins = pass == 2 ? 128 : kHistBins;
      const unsigned dmask = (unsigned)nbins - 1u;
      for (int b = threadIdx.x; b < nbins; b += kVoteThreads) hist[b] = 0;
      __syncthreads();
      sweep([&](unsigned u) {
        if ((u & prefix_mask) == prefix) atomicAdd(&hist[(u >> shift) & dmask], 1u);
      });
      __syncthreads();
      // thread t owns the `per` digits below nbins - 1 - t * per, in descending order
      const int per = (nbins + kVoteThreads - 1) / kVoteThreads;
      const int top = nbins - 1 - (int)threadIdx.x * per;
      int local = 0;
      for (int i = 0; i < per; ++i)
        if (top - i >= 0) local += (int)hist[top - i];
      int total = 0;
      const int above = block_exclusive_scan(local, red_i, &total);   // values with a larger digit
      if (above < want && above + local >= want) {
        int acc = above;
        for (int i = 0; i < per; ++i) {
          const int hc = (int)hist[top - i];
          if (acc + hc >= want) {
            pick[0] = top - i;
            pick[1] = acc;
            break;
          }
          acc += hc;
        }
      }
      __syncthreads();
      want -= pick[1];
      prefix |= (unsigned)pick[0] << shift;
      prefix_mask |= dmask << shift;
      __syncthreads();
    }
  }
  const unsigned thr = prefix;   // bit pattern of the threshold value (valid when 0 < cnt < n)

  // 3. thread t owns a contiguous index range, so prefix sums follow index order. The ties at
  //    the threshold taken are the first `want` in index order: this thread's ties are the
  //    global ties [tie_before, tie_before + n_tie).
  int per = (n + kVoteThreads - 1) / kVoteThreads;
  if (kTok) per = (per + 3) & ~3;
  const int c0 = min(n, (int)threadIdx.x * per), c1 = min(n, c0 + per);
  int n_tie = 0, n_gt = 0;
  if (cnt > 0 && cnt < n) {
    range_each(c0, c1, [&](int, unsigned u) {
      n_gt += u > thr;
      n_tie += u == thr;
    });
  }
  int tie_total = 0;
  const int tie_before = block_exclusive_scan(n_tie, red_i, &tie_total);
  const int n_sel_local = cnt >= n ? c1 - c0 : (cnt > 0 ? n_gt + min(max(want - tie_before, 0), n_tie) : 0);
  int sel_total = 0;
  int pos = block_exclusive_scan(n_sel_local, red_i, &sel_total);
  if (cnt >= n) {
    for (int c = c0; c < c1; ++c) out[pos++] = a.first + c;
  } else if (cnt > 0) {
    int ties_seen = tie_before;
    range_each(c0, c1, [&](int c, unsigned u) {
      const bool take = u > thr || (u == thr && ties_seen++ < want);
      if (take) out[pos++] = a.first + c;
    });
  }
  for (int i = cnt + threadIdx.x; i < top_k; i += kVoteThreads) out[i] = -1;
}

// grid: (1024-candidate slice, cluster). score[j][c] = sum over KV heads g, in order, of the
// partial scores of the token scoring kernel; four candidates per thread (n_cand is a multiple of
// 64 and the rows are 16-byte aligned).
__global__ __launch_bounds__(kThreads) void token_sum_kernel(const float* __restrict__ partial,
                                                             const ClusterGeo* __restrict__ geo, int64_t cand_stride,
                                                             int num_kv_heads, float* __restrict__ score) {
  const int j = blockIdx.y;
  const int c = (blockIdx.x * kThreads + threadIdx.x) * 4;
  if (c >= geo[j].n_cand) return;
  const float* part = partial + (int64_t)j * num_kv_heads * cand_stride + c;
  float4 acc = *reinterpret_cast<const float4*>(part);
  for (int g = 1; g < num_kv_heads; ++g) {
    const float4 v = *reinterpret_cast<const float4*>(part + (int64_t)g * cand_stride);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  *reinterpret_cast<float4*>(score + (int64_t)j * cand_stride + c) = acc;
}

struct LogitsArgs {
  const float *fingerprints, *k_rep;
  const ClusterGeo* geo;
  int parts, n_chunks, cand_stride, sink_blk, num_q_heads, num_kv_heads;
  float score_scale;
  float* logits;
  float2* head_stats;
};

template <int D, bool kBounds>
void launch_logits(dim3 grid, const LogitsArgs& a, hipStream_t stream) {
  block_logits_kernel<D, kBounds><<<grid, kThreads, 0, stream>>>(a.fingerprints, a.k_rep, a.geo, a.parts, a.n_chunks,
                                                                a.cand_stride, a.sink_blk, a.num_q_heads,
                                                                a.num_kv_heads, a.score_scale, a.logits, a.head_stats);
}

}  // namespace

hipError_t launch_fingerprints(const uint16_t* q, const ClusterGeo* geo, int n_clusters,
                               int num_q_heads, int head_dim, float* fingerprints, hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  const int row_elems = num_q_heads * head_dim;
  const dim3 grid((row_elems + kFpCols - 1) / kFpCols, n_clusters);
  fingerprint_kernel<<<grid, kFpThreads, 0, stream>>>(q, geo, row_elems, fingerprints);
  return hipGetLastError();
}

int selection_chunks(int max_cand) { return (max_cand + kCandChunk - 1) / kCandChunk; }

hipError_t launch_block_logits(const float* fingerprints, const float* k_rep, const ClusterGeo* geo,
                               int n_clusters, int max_cand, int cand_stride, int sink_blk,
                               int num_q_heads, int num_kv_heads, int head_dim, bool bounds, float score_scale,
                               float* logits, float2* head_stats, hipStream_t stream) {
  if (n_clusters <= 0 || max_cand <= 0) return hipSuccess;
  const int n_chunks = selection_chunks(max_cand);
  // enough work-groups to fill the chip, without launching many that find no chunk
  const int64_t base = (int64_t)n_clusters * num_kv_heads;
  const int parts = (int)std::min<int64_t>(n_chunks, std::max<int64_t>(1, (kLogitsTargetGroups + base - 1) / base));
  const dim3 grid((unsigned)(base * parts));
  const LogitsArgs a{fingerprints, k_rep, geo, parts, n_chunks, cand_stride, sink_blk, num_q_heads, num_kv_heads,
                     score_scale, logits, head_stats};
  if (head_dim == 128)
    bounds ? launch_logits<128, true>(grid, a, stream) : launch_logits<128, false>(grid, a, stream);
  else
    bounds ? launch_logits<64, true>(grid, a, stream) : launch_logits<64, false>(grid, a, stream);
  return hipGetLastError();
}

hipError_t launch_vote_topk(const float* logits, const float2* head_stats, const ClusterGeo* geo, int n_clusters,
                            int max_cand, int cand_stride, int sink_blk, int num_q_heads, int num_kv_heads,
                            bool per_kv, int top_k, int n_blocks, float* spill, int32_t* sel_idx, int32_t* sel_cnt,
                            float* scores_out, hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  VoteArgs a{};
  a.logits = logits;
  a.head_stats = head_stats;
  a.geo = geo;
  a.n_chunks = selection_chunks(max_cand);
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.per_kv = per_kv ? 1 : 0;
  a.top_k = top_k;
  a.cand_stride = cand_stride;
  a.first = sink_blk;
  a.n_out = n_blocks;
  a.spill = spill;
  a.sel_idx = sel_idx;
  a.sel_cnt = sel_cnt;
  a.scores_out = scores_out;
  const size_t lds = sizeof(float) * 2 * (size_t)num_q_heads;
  vote_topk_kernel<false><<<n_clusters * (per_kv ? num_kv_heads : 1), kVoteThreads, lds, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_vote_topk_tokens(const float* partial, const ClusterGeo* geo, int n_clusters, int64_t cand_stride,
                                   int max_cand, int first_token, int num_kv_heads, bool per_kv, int top_k,
                                   int n_tokens, float* spill, int32_t* sel_idx, int32_t* sel_cnt, float* scores_out,
                                   hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  if (max_cand > 0 && !per_kv) {
    const dim3 grid((unsigned)((max_cand + 4 * kThreads - 1) / (4 * kThreads)), (unsigned)n_clusters);
    token_sum_kernel<<<grid, kThreads, 0, stream>>>(partial, geo, cand_stride, num_kv_heads, spill);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  VoteArgs a{};
  a.partial = partial;
  a.geo = geo;
  a.num_kv_heads = num_kv_heads;
  a.top_k = top_k;
  a.cand_stride = cand_stride;
  a.first = first_token;
  a.n_out = n_tokens;
  a.per_kv = per_kv ? 1 : 0;
  a.spill = spill;
  a.sel_idx = sel_idx;
  a.sel_cnt = sel_cnt;
  a.scores_out = scores_out;
  vote_topk_kernel<true><<<n_clusters * (per_kv ? num_kv_heads : 1), kVoteThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace scale
