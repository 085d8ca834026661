// Cluster-level block selection: anchor fingerprints, per-head logits, head soft-voting and a
// deterministic top-k, once per cluster (paper Sec. 5.1.3, Eq. 9 and the head soft-voting
// instantiation of the selection function).
//
//  fingerprint   (column slice, cluster) -> mean of the anchor rows: fp64 sums, written in fp64
//                (for the logits) and rounded once to fp32 (for token scoring and the caller)
//  block_logits  (candidate tile, fingerprint-row tile, KV head) -> for the 64 rows (cluster j,
//                query head h of KV head g) x 64 candidates c of the tile, the fp64 logit
//                x = sigma * v[j][h] . k_rep[c][g] (bound form: sigma * sum_i max(v_i mn_i, v_i mx_i)),
//                then per row the tile's softmax partials: m = max_c x, the weights exp(x - m) and
//                their sum. A tile is one 64-candidate chunk; the k_rep tile staged in LDS serves
//                every cluster whose rows share the tile (up to 64 clusters), the fingerprint tile
//                every candidate of it
//  vote_topk     cluster (or (cluster, KV head) with one set per KV head) -> per head the softmax
//                maximum and normaliser from the chunk partials and one factor exp(m_k - M) / S per
//                chunk, score = sum over the voting heads of weight x factor (all fp64), rounded
//                once to fp32; top-k by (score desc, index asc), ascending; token mode takes the
//                scores of the token scoring kernels (select_tokens.hip)
//  token_sum     (candidate slice, cluster) -> token scores: the per-KV-head partial scores summed
//                in KV-head order
//
// The softmax of a head is split exactly: exp(x - M) / S = exp(x - m_k) * exp(m_k - M) / S for
// the chunk k holding x, with S = sum_k s_k exp(m_k - M). Every reduction has a fixed order, so two
// runs give identical bits.
#include <float.h>

#include <algorithm>

#include "common.h"

namespace scale {
namespace {

constexpr int kThreads = 256;
constexpr int kFpThreads = 512;          // fingerprint: 8 waves
constexpr int kFpCols = 512;             // columns of the Hq*d row per fingerprint work-group
constexpr int kFpRowsInFlight = 4;       // 16-byte loads in flight per lane
constexpr int kCandChunk = 64;           // candidates per logits tile = per softmax-partial chunk
constexpr int kLgRows = 64;              // fingerprint rows (cluster, query head) per logits tile
constexpr int kLgDk = 32;                // head-dim slice staged in LDS per step

// grid: (column slice, cluster). Lane l of wave w owns the 8 columns [slice*512 + 8l, +8) and
// sums anchor rows w, w+8, w+16, ... in fp64 (exact for bf16 inputs of moderate range); the 8
// waves' sums are combined in LDS in wave order and divided once.
__global__ __launch_bounds__(kFpThreads) void fingerprint_kernel(const uint16_t* __restrict__ q,
                                                                 const ClusterGeo* __restrict__ geo,
                                                                 int row_elems, float* __restrict__ fingerprints,
                                                                 double* __restrict__ fingerprints64) {
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
    const double mean = s / (double)n_rows;
    fingerprints[(int64_t)j * row_elems + c] = (float)mean;
    if (fingerprints64) fingerprints64[(int64_t)j * row_elems + c] = mean;
  }
}

// grid: linear over (candidate tile ct, row tile rt, KV head g), g fastest, so the 8 XCDs each
// serve KV heads of their own (one KV head's slice of k_rep per L2 when Hkv = 8). Rows of KV head g
// are r = j * G + u (cluster j, query head g * G + u); a work-group takes rows [64 rt, 64 rt + 64)
// and candidates [64 ct, 64 ct + 64) and skips the tile when no cluster of its rows has that many
// candidates. 256 threads as 16 x 16: thread (tr, tc) owns rows 4 tr .. 4 tr + 3 and candidates
// 4 tc .. 4 tc + 3 (tc in the low lane bits, so a row's 16 threads are 16 consecutive lanes). The
// head dim is staged through LDS in slices of 32, fingerprints and keys both as doubles stored
// [dim][row or candidate], so each step reads 4 fingerprint and 4 key values and does 16 fp64 fmas.
template <int D, bool kBounds>
__global__ __launch_bounds__(kThreads) void block_logits_kernel(
    const double* __restrict__ fingerprints, const float* __restrict__ k_rep, const ClusterGeo* __restrict__ geo,
    int n_clusters, int row_tiles, int n_chunks, int64_t cand_stride, int sink_blk, int num_q_heads,
    int num_kv_heads, double score_scale, double* __restrict__ weights, double2* __restrict__ stats) {
  constexpr int kKeys = kBounds ? 2 : 1;                  // mean key, or minima then maxima
  __shared__ double v_lds[kLgDk][kLgRows];
  __shared__ double k_lds[kKeys][kLgDk][kCandChunk];
  const int G = num_q_heads / num_kv_heads;
  const int g = blockIdx.x % num_kv_heads;
  const int rest = blockIdx.x / num_kv_heads;
  const int rt = rest % row_tiles;
  const int ct = rest / row_tiles;
  const int n_rows = n_clusters * G;
  const int r0 = rt * kLgRows, c0 = ct * kCandChunk;
  const int tid = threadIdx.x, lane = tid % 64;

  // candidates of the tile's clusters (at most 64 clusters: one per lane), reduced per wave
  const int j_first = r0 / G, j_last = (min(n_rows, r0 + kLgRows) - 1) / G;
  int nc = 0;
  if (j_first + lane <= j_last) nc = geo[j_first + lane].n_cand;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) nc = max(nc, __shfl_xor(nc, o, 64));
  if (c0 >= nc) return;                                   // uniform over the work-group

  const int tr = tid / 16, tc = tid % 16;
  // staging: thread t loads 8 consecutive dims of row / candidate t / 4
  const int ld_row = tid / 4, ld_part = (tid % 4) * 8;
  const int r_ld = r0 + ld_row;
  const double* v_src = nullptr;
  if (r_ld < n_rows)
    v_src = fingerprints + ((int64_t)(r_ld / G) * num_q_heads + g * G + r_ld % G) * D + ld_part;
  const int c_ld = c0 + ld_row;
  const float* k_src = nullptr;
  if (c_ld < nc) k_src = k_rep + ((int64_t)(sink_blk + c_ld) * num_kv_heads + g) * (kKeys * D) + ld_part;

  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[i][q] = 0.0;

  // The global loads of slice d0 + kLgDk are issued before slice d0 is multiplied, so their
  // latency hides under the fmas of the slice before.
  double vv[8];
  float kk[kKeys][8];
  auto load_slice = [&](int d0) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const double2 t = v_src ? *reinterpret_cast<const double2*>(v_src + d0 + e) : make_double2(0.0, 0.0);
      vv[e] = t.x;
      vv[e + 1] = t.y;
    }
#pragma unroll
    for (int m = 0; m < kKeys; ++m)
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        const float4 t = k_src ? *reinterpret_cast<const float4*>(k_src + m * D + d0 + e)
                               : make_float4(0.f, 0.f, 0.f, 0.f);
        kk[m][e] = t.x;
        kk[m][e + 1] = t.y;
        kk[m][e + 2] = t.z;
        kk[m][e + 3] = t.w;
      }
  };
  load_slice(0);
  for (int d0 = 0; d0 < D; d0 += kLgDk) {
    __syncthreads();                                      // the previous slice has been read
#pragma unroll
    for (int e = 0; e < 8; ++e) v_lds[ld_part + e][ld_row] = vv[e];
#pragma unroll
    for (int m = 0; m < kKeys; ++m)
#pragma unroll
      for (int e = 0; e < 8; ++e) k_lds[m][ld_part + e][ld_row] = (double)kk[m][e];
    __syncthreads();
    if (d0 + kLgDk < D) load_slice(d0 + kLgDk);
#pragma unroll 4
    for (int dd = 0; dd < kLgDk; ++dd) {
      const double2 va = *reinterpret_cast<const double2*>(&v_lds[dd][4 * tr]);
      const double2 vb = *reinterpret_cast<const double2*>(&v_lds[dd][4 * tr + 2]);
      const double v[4] = {va.x, va.y, vb.x, vb.y};
      double k[kKeys][4];
#pragma unroll
      for (int m = 0; m < kKeys; ++m) {
        const double2 ka = *reinterpret_cast<const double2*>(&k_lds[m][dd][4 * tc]);
        const double2 kb = *reinterpret_cast<const double2*>(&k_lds[m][dd][4 * tc + 2]);
        k[m][0] = ka.x;
        k[m][1] = ka.y;
        k[m][2] = kb.x;
        k[m][3] = kb.y;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if constexpr (kBounds)
            acc[i][q] += fmax(v[i] * k[0][q], v[i] * k[1][q]);
          else
            acc[i][q] = fma(v[i], k[0][q], acc[i][q]);
        }
    }
  }

  // per row: this tile's softmax partials over its valid candidates (16 lanes per row)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = r0 + 4 * tr + i;
    const int j = r / G;
    const int n_valid = r < n_rows ? geo[j].n_cand - c0 : 0;   // candidates of row r in this tile
    double x[4], m = -DBL_MAX;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[q] = score_scale * acc[i][q];
      if (4 * tc + q < n_valid) m = fmax(m, x[q]);
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) m = fmax(m, __shfl_xor(m, o, 64));
    double e[4], sum = 0.0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      e[q] = 4 * tc + q < n_valid ? exp(x[q] - m) : 0.0;
      sum += e[q];
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) sum += __shfl_xor(sum, o, 64);
    if (n_valid <= 0) continue;
    const int64_t row = (int64_t)j * num_q_heads + g * G + r % G;
    double* w = weights + row * cand_stride + c0 + 4 * tc;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (4 * tc + q < n_valid) w[q] = e[q];
    if (tc == 0) stats[row * n_chunks + ct] = make_double2(m, sum);
  }
}

// ---- vote_topk ----
constexpr int kVoteThreads = 1024;
constexpr int kVoteWaves = kVoteThreads / 64;
constexpr int kMaxLdsCand = 8192;        // scores of larger clusters live in the global spill row
constexpr int kHistBins = 4096;          // radix digits of the first two passes (12 bits)
constexpr int kFacLds = 2048;            // chunk factors (voting heads x chunks) kept in LDS
constexpr int kStatsCached = 1;          // chunk statistics a lane holds in registers (64 chunks per head)
constexpr int kWeightBatch = 8;          // weight loads in flight per candidate

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
//  1. soft-voting, in fp64: wave w takes heads w, w + 16, ...; each head's softmax maximum M and
//     normaliser S over all candidates come from the chunk partials (m_k, s_k) with a fixed lane
//     butterfly, and each chunk gets the factor exp(m_k - M) / S (written to the factor scratch);
//     then per candidate the sum over heads, in head order, of its weight exp(x - m_k) times the
//     factor of its chunk, rounded once to fp32. Token mode (kTok): the per-KV-head partial sums of
//     the token scoring kernel are added in KV-head order instead.
//  2. threshold: the sel_cnt-th largest score, by radix selection on the score bits (scores are
//     >= 0, so their bit patterns order like their values and the sign bit is 0) in three passes
//     over bits 30-19, 18-7 and 6-0; wide first digits spread the scores of a cluster, which share
//     few exponents, over many histogram bins. The digit is found with a prefix sum over the
//     histogram in descending digit order.
//  3. selected = score above the threshold, or equal to it and among the first ties in index
//     order; written in ascending index order by an ordered compaction.
struct VoteArgs {
  const double* weights;       // block mode: [cluster][Hq][cand_stride], exp(x - chunk max)
  const double2* stats;        // block mode: [cluster][Hq][n_chunks], (chunk max, chunk sum)
  double* factors;             // block mode: [cluster][Hq][n_chunks] scratch
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
  __shared__ double fac_lds[kTok ? 1 : kFacLds];
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
    const int n_chunks = a.n_chunks;
    const int used = (n + kCandChunk - 1) / kCandChunk;
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    // the factors of the voting heads stay in LDS when they fit, else in the global scratch
    const bool fac_in_lds = (h1 - h0) * used <= kFacLds;
    for (int h = h0 + wave; h < h1; h += kVoteWaves) {
      const int64_t hrow = (int64_t)j * num_q_heads + h;
      const double2* st = a.stats + hrow * n_chunks;
      // a lane's first kStatsCached chunks k = lane + 64 u are loaded once, together
      double2 sc[kStatsCached];
#pragma unroll
      for (int u = 0; u < kStatsCached; ++u)
        sc[u] = lane + 64 * u < used ? st[lane + 64 * u] : make_double2(-DBL_MAX, 0.0);
      double m = -DBL_MAX;
#pragma unroll
      for (int u = 0; u < kStatsCached; ++u) m = fmax(m, sc[u].x);
      for (int k = lane + 64 * kStatsCached; k < used; k += 64) m = fmax(m, st[k].x);
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) m = fmax(m, __shfl_xor(m, o, 64));
      // the lane's chunks in increasing order, then the fixed butterfly
      double e[kStatsCached];        // exp(m_k - M) of the cached chunks
#pragma unroll
      for (int u = 0; u < kStatsCached; ++u) e[u] = lane + 64 * u < used ? exp(sc[u].x - m) : 0.0;
      double sum = 0.0;
#pragma unroll
      for (int u = 0; u < kStatsCached; ++u)
        if (lane + 64 * u < used) sum += sc[u].y * e[u];
      for (int k = lane + 64 * kStatsCached; k < used; k += 64) sum += st[k].y * exp(st[k].x - m);
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) sum += __shfl_xor(sum, o, 64);
      const double inv = 1.0 / sum;
      double* f = fac_in_lds ? fac_lds + (h - h0) * used : a.factors + hrow * n_chunks;
#pragma unroll
      for (int u = 0; u < kStatsCached; ++u)
        if (lane + 64 * u < used) f[lane + 64 * u] = e[u] * inv;
      for (int k = lane + 64 * kStatsCached; k < used; k += 64) f[k] = exp(st[k].x - m) * inv;
    }
    __syncthreads();                                 // the factors are read by every thread below
    const double* wts = a.weights + (int64_t)j * num_q_heads * cand_stride;
    // per candidate: the sum over the voting heads, in head order, of weight x chunk factor
    auto vote = [&](auto&& fac) {
      for (int c = threadIdx.x; c < n; c += kVoteThreads) {
        const int k = c / kCandChunk;
        double acc = 0.0;
        int h = h0;
        for (; h + kWeightBatch <= h1; h += kWeightBatch) {
          double wv[kWeightBatch];
#pragma unroll
          for (int u = 0; u < kWeightBatch; ++u) wv[u] = wts[(int64_t)(h + u) * cand_stride + c];
#pragma unroll
          for (int u = 0; u < kWeightBatch; ++u) acc = fma(wv[u], fac(h + u, k), acc);
        }
        for (; h < h1; ++h) acc = fma(wts[(int64_t)h * cand_stride + c], fac(h, k), acc);
        score[c] = (float)acc;
      }
    };
    if (fac_in_lds) {
      vote([&](int h, int k) { return fac_lds[(h - h0) * used + k]; });
    } else {
      const double* fac = a.factors + (int64_t)j * num_q_heads * n_chunks;
      vote([&](int h, int k) { return fac[(int64_t)h * n_chunks + k]; });
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
  const double* fingerprints;
  const float* k_rep;
  const ClusterGeo* geo;
  int n_clusters, row_tiles, n_chunks;
  int64_t cand_stride;
  int sink_blk, num_q_heads, num_kv_heads;
  double score_scale;
  double* weights;
  double2* stats;
};

template <int D, bool kBounds>
void launch_logits(dim3 grid, const LogitsArgs& a, hipStream_t stream) {
  block_logits_kernel<D, kBounds><<<grid, kThreads, 0, stream>>>(
      a.fingerprints, a.k_rep, a.geo, a.n_clusters, a.row_tiles, a.n_chunks, a.cand_stride, a.sink_blk,
      a.num_q_heads, a.num_kv_heads, a.score_scale, a.weights, a.stats);
}

}  // namespace

hipError_t launch_fingerprints(const uint16_t* q, const ClusterGeo* geo, int n_clusters,
                               int num_q_heads, int head_dim, float* fingerprints, double* fingerprints64,
                               hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  const int row_elems = num_q_heads * head_dim;
  const dim3 grid((row_elems + kFpCols - 1) / kFpCols, n_clusters);
  fingerprint_kernel<<<grid, kFpThreads, 0, stream>>>(q, geo, row_elems, fingerprints, fingerprints64);
  return hipGetLastError();
}

int selection_chunks(int max_cand) { return (max_cand + kCandChunk - 1) / kCandChunk; }

hipError_t launch_block_logits(const double* fingerprints, const float* k_rep, const ClusterGeo* geo,
                               int n_clusters, int max_cand, int64_t cand_stride, int sink_blk,
                               int num_q_heads, int num_kv_heads, int head_dim, bool bounds, double score_scale,
                               double* weights, double2* stats, hipStream_t stream) {
  if (n_clusters <= 0 || max_cand <= 0) return hipSuccess;
  const int n_chunks = selection_chunks(max_cand);
  const int64_t rows = (int64_t)n_clusters * (num_q_heads / num_kv_heads);
  const int row_tiles = (int)((rows + kLgRows - 1) / kLgRows);
  const dim3 grid((unsigned)((int64_t)n_chunks * row_tiles * num_kv_heads));
  const LogitsArgs a{fingerprints, k_rep, geo, n_clusters, row_tiles, n_chunks, cand_stride, sink_blk,
                     num_q_heads, num_kv_heads, score_scale, weights, stats};
  if (head_dim == 128)
    bounds ? launch_logits<128, true>(grid, a, stream) : launch_logits<128, false>(grid, a, stream);
  else
    bounds ? launch_logits<64, true>(grid, a, stream) : launch_logits<64, false>(grid, a, stream);
  return hipGetLastError();
}

hipError_t launch_vote_topk(const double* weights, const double2* stats, double* factors, const ClusterGeo* geo,
                            int n_clusters, int max_cand, int64_t cand_stride, int sink_blk, int num_q_heads,
                            int num_kv_heads, bool per_kv, int top_k, int n_blocks, float* spill, int32_t* sel_idx,
                            int32_t* sel_cnt, float* scores_out, hipStream_t stream) {
  if (n_clusters <= 0) return hipSuccess;
  VoteArgs a{};
  a.weights = weights;
  a.stats = stats;
  a.factors = factors;
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
  vote_topk_kernel<false><<<n_clusters * (per_kv ? num_kv_heads : 1), kVoteThreads, 0, stream>>>(a);
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
