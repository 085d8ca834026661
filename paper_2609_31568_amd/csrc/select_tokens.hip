// Token-level selection: head soft-voting over single candidate tokens, each scored with its own
// key, once per cluster (paper Sec. 5.1.3, Eq. 9 at the granularity of individual tokens), and the
// gather of the selected keys and values for the cluster attention of Eq. 10.
//
// Per KV head g the logits of every cluster are one dense product: the fingerprint rows
// (cluster j, query head h of g), R of them, times the candidate keys, which is where the matrix
// cores belong. A fingerprint row is split into two bf16 pieces (hi = bf16(v), lo = bf16(v - hi),
// |v - hi - lo| <= 2^-18 |v|); bf16 keys are exact, so two v_mfma_f32_32x32x16_bf16 per 16-wide
// slice of d give fp32-class logits. Candidates are the tokens [T0, T0 + n_cand_j) with
// T0 = sink_blk * B; n_cand_j is a multiple of B, so every 64-token tile lies wholly inside or
// outside a cluster's candidates.
//
//  split          fingerprints -> bf16 pieces F[g][row][piece][d], row = j * GP + i (GP = the
//                 group size rounded up to a power of two; rows i >= G are zero)
//  token_logits   (KV head g, row group of 128 rows, chunk of tiles):
//                   stats pass   per (row, chunk): a reference m and s = sum of 2^(x - m) over the
//                                chunk's candidates (x = logit in base-2 units)
//                   scores pass  per (cluster, KV head, token): sum over the query heads of g of
//                                2^(x - lse_row), written as a partial score
//  token_lse      per row: log2 of the softmax normaliser from the chunk partials (fixed order)
//  gather         (tile of selected rows, KV head, cluster) -> the selected keys and values copied
//                 into [cluster][g][kpad][d] tiles; rows past the selection are zero
//
// The soft-voting sum over KV heads (token_sum) and the top-k (vote_topk) are in select.hip. Every
// reduction has a fixed order, so two runs give identical bits.
#include <math.h>

#include <algorithm>

#include "common.h"

namespace scale {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTokTile = kTokenTile;  // candidate tokens per step
constexpr int kTokThreads = 256;      // 4 waves, one 32-row block each
constexpr int kRowsPerGroup = 128;
constexpr int kGatherThreads = 256;
constexpr float kStatsHeadroom = 20.f;   // base-2 units a logit may exceed the stats reference by

__device__ __forceinline__ uint16_t bf16_rne(float v) {
  uint32_t u = __float_as_uint(v);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// grid: cluster. Writes the rows of cluster j for every KV head (zero rows for i >= G).
__global__ __launch_bounds__(256) void split_fingerprints_kernel(const float* __restrict__ fps, int num_q_heads,
                                                                 int num_kv_heads, int head_dim, int gp, int r_pad,
                                                                 uint16_t* __restrict__ F) {
  const int j = blockIdx.x;
  const int group = num_q_heads / num_kv_heads;
  const int n = num_kv_heads * gp * head_dim;
  for (int idx = threadIdx.x; idx < n; idx += blockDim.x) {
    const int c = idx % head_dim;
    const int i = (idx / head_dim) % gp;
    const int g = idx / (head_dim * gp);
    uint16_t hi = 0, lo = 0;
    if (i < group) {
      const float v = fps[((int64_t)j * num_q_heads + g * group + i) * head_dim + c];
      hi = bf16_rne(v);
      lo = bf16_rne(v - __uint_as_float((uint32_t)hi << 16));
    }
    uint16_t* dst = F + ((int64_t)(g * r_pad + j * gp + i) * 2) * head_dim + c;
    dst[0] = hi;
    dst[head_dim] = lo;
  }
}

struct TokArgs {
  const uint16_t* k_pages;
  const int32_t* block_table;
  const uint16_t* F;
  const ClusterGeo* geo;
  const float* lse2;     // scores pass: [g][row]
  float2* stats;         // stats pass: [g][row][chunk]
  float* partial;        // scores pass: [cluster][g][cand_stride]
  int64_t cand_stride;
  int n_clusters, group, r_pad, n_rowgroups, tiles_per_chunk, n_chunks;
  int first_token, num_kv_heads, log2_block;
  float scale2;          // sigma * log2(e)
};

// grid: linear over (chunk, row group, KV head) with the KV head fastest, so a KV head's keys and
// fingerprint rows stay in one XCD's L2. Wave w owns the 32 fingerprint rows of row block
// 4 * row group + w, held in registers as the MFMA A operand; the 64-token key tiles of the chunk
// stream through LDS (row stride d + 8 elements: conflict-free 16-byte operand reads) with one
// tile in flight. Accumulator e of lane l holds row 8 (e / 4) + 4 (l / 32) + e % 4 of the block
// and token l % 32 of the 32-token column block.
template <int D, int GP, bool kScores>
__global__ __launch_bounds__(kTokThreads) void token_logits_kernel(TokArgs a) {
  constexpr int kKStride = D + 8;
  constexpr int kPer = kTokTile * D / 8 / kTokThreads;
  __shared__ __attribute__((aligned(16))) uint16_t kl[2][kTokTile * kKStride];
  __shared__ int wave_nc[kTokThreads / 64];
  const int g = blockIdx.x % a.num_kv_heads;
  const int rest = blockIdx.x / a.num_kv_heads;
  const int rg = rest % a.n_rowgroups;
  const int chunk = rest / a.n_rowgroups;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, half = lane / 32, col = lane % 32;
  const int rb = rg * 4 + wave;

  // candidate count of each accumulator row (0 for padding rows and absent clusters)
  int nc[16];
  int wmax = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int row = rb * 32 + 8 * (e / 4) + 4 * half + (e % 4);
    const int j = row / GP, i = row % GP;
    nc[e] = (j < a.n_clusters && i < a.group) ? a.geo[j].n_cand : 0;
    wmax = max(wmax, nc[e]);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) wmax = max(wmax, __shfl_xor(wmax, o, 64));
  if (lane == 0) wave_nc[wave] = wmax;
  __syncthreads();
  const int gmax = max(max(wave_nc[0], wave_nc[1]), max(wave_nc[2], wave_nc[3]));
  const int c0 = chunk * a.tiles_per_chunk * kTokTile;
  if (c0 >= gmax) return;                                  // uniform over the work-group
  const int n_t = min(a.tiles_per_chunk, (gmax - c0) / kTokTile);

  bf16x8 fa[2][D / 16];
  if (wmax > c0) {
    const uint16_t* fr = a.F + ((int64_t)(g * a.r_pad + rb * 32 + col) * 2) * D + 8 * half;
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int c = 0; c < D / 16; ++c) fa[p][c] = *reinterpret_cast<const bf16x8*>(fr + p * D + 16 * c);
  }

  const int bmask = (1 << a.log2_block) - 1;
  auto tile_src = [&](int t) -> const uint16_t* {
    const int tok = a.first_token + c0 + t * kTokTile;
    const int blk = tok >> a.log2_block;
    const int page = a.block_table ? a.block_table[blk] : blk;
    return a.k_pages + ((((int64_t)page * a.num_kv_heads + g) << a.log2_block) + (tok & bmask)) * D;
  };
  u32x4 kr[kPer];
  auto load = [&](int t) {
    const uint16_t* src = tile_src(t);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = tid + i * kTokThreads;
      kr[i] = *reinterpret_cast<const u32x4*>(src + (idx / (D / 8)) * D + 8 * (idx % (D / 8)));
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = tid + i * kTokThreads;
      *reinterpret_cast<u32x4*>(&kl[buf][(idx / (D / 8)) * kKStride + 8 * (idx % (D / 8))]) = kr[i];
    }
  };

  float m[16], s[16], lse[16];
  if constexpr (kScores) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int row = rb * 32 + 8 * (e / 4) + 4 * half + (e % 4);
      lse[e] = nc[e] > 0 ? a.lse2[g * a.r_pad + row] : INFINITY;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      m[e] = -INFINITY;
      s[e] = 0.f;
    }
  }

  load(0);
  store(0);
  __syncthreads();
  for (int t = 0; t < n_t; ++t) {
    const int buf = t & 1;
    if (t + 1 < n_t) load(t + 1);
    const int tc = c0 + t * kTokTile;                       // candidate index of the tile's first token
    if (wmax > tc) {
      f32x16 acc[2] = {f32x16{}, f32x16{}};
      const uint16_t* kb = &kl[buf][col * kKStride + 8 * half];
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(kb + 16 * c);
        const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(kb + 32 * kKStride + 16 * c);
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][c], k0, acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][c], k1, acc[1], 0, 0, 0);
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][c], k0, acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][c], k1, acc[1], 0, 0, 0);
      }
      if constexpr (kScores) {
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
          float p[16];
#pragma unroll
          for (int e = 0; e < 16; ++e)
            p[e] = tc < nc[e] ? __builtin_amdgcn_exp2f(fmaf(acc[cb][e], a.scale2, -lse[e])) : 0.f;
          // sum over the query heads of each cluster: GP consecutive rows
          constexpr int kIn = GP < 4 ? GP : 4;
#pragma unroll
          for (int e = 0; e < 16; e += kIn) {
            float sum = p[e];
#pragma unroll
            for (int u = 1; u < kIn; ++u) sum += p[e + u];
            if constexpr (GP == 8) sum += __shfl_xor(sum, 32, 64);
            const int row0 = rb * 32 + 8 * (e / 4) + 4 * half + (e % 4);
            const int j = row0 / GP;
            if ((GP < 8 || half == 0) && tc < nc[e])
              a.partial[((int64_t)j * a.num_kv_heads + g) * a.cand_stride + tc + 32 * cb + col] = sum;
          }
        }
      } else {
        // s accumulates 2^(x - m) against a reference m that is only raised (exactly: s rescaled)
        // when a value would exceed it by more than 2^kStatsHeadroom; the first tile always does.
        bool up = false;
#pragma unroll
        for (int e = 0; e < 16; ++e)
          up |= tc < nc[e] && fmaxf(acc[0][e] * a.scale2, acc[1][e] * a.scale2) > m[e] + kStatsHeadroom;
        if (__any(up)) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            if (tc < nc[e]) {
              const float mx = fmaxf(fmaxf(acc[0][e] * a.scale2, acc[1][e] * a.scale2), m[e]);
              s[e] *= __builtin_amdgcn_exp2f(m[e] - mx);
              m[e] = mx;
            }
          }
        }
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (tc < nc[e])
            s[e] += __builtin_amdgcn_exp2f(fmaf(acc[0][e], a.scale2, -m[e])) +
                    __builtin_amdgcn_exp2f(fmaf(acc[1][e], a.scale2, -m[e]));
      }
    }
    if (t + 1 < n_t) store(buf ^ 1);
    __syncthreads();
  }

  if constexpr (!kScores) {
    // merge the 32 columns of each lane half, then lane 0 / 32 writes its 16 rows
#pragma unroll
    for (int e = 0; e < 16; ++e) {
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) {
        const float mo = __shfl_xor(m[e], o, 64), so = __shfl_xor(s[e], o, 64);
        const float M = fmaxf(m[e], mo);
        const float a0 = m[e] == -INFINITY ? 0.f : s[e] * __builtin_amdgcn_exp2f(m[e] - M);
        const float a1 = mo == -INFINITY ? 0.f : so * __builtin_amdgcn_exp2f(mo - M);
        s[e] = a0 + a1;
        m[e] = M;
      }
    }
    if (col == 0) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rb * 32 + 8 * (e / 4) + 4 * half + (e % 4);
        if (nc[e] > c0) a.stats[((int64_t)g * a.r_pad + row) * a.n_chunks + chunk] = make_float2(m[e], s[e]);
      }
    }
  }
}

// grid: ceil(Hkv * r_pad / 4), one wave per row. lse2[g][row] = M + log2(sum over chunks of
// s_k 2^(m_k - M)); lane l takes chunks l, l + 64, ... in order, and the 64 lane values are
// combined by a fixed butterfly. +inf for rows without candidates (their weights are then 0).
__global__ __launch_bounds__(256) void token_lse_kernel(const float2* __restrict__ stats, const ClusterGeo* __restrict__ geo,
                                                       int n_clusters, int group, int gp, int r_pad, int num_kv_heads,
                                                       int n_chunks, int chunk_tokens, float* __restrict__ lse2) {
  const int idx = blockIdx.x * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  if (idx >= num_kv_heads * r_pad) return;                 // uniform over the wave
  const int row = idx % r_pad;
  const int j = row / gp, i = row % gp;
  const int used = (j < n_clusters && i < group) ? (geo[j].n_cand + chunk_tokens - 1) / chunk_tokens : 0;
  if (used == 0) {
    if (lane == 0) lse2[idx] = INFINITY;
    return;
  }
  const float2* st = stats + (int64_t)idx * n_chunks;
  float m = -INFINITY;
  for (int k = lane; k < used; k += 64) m = fmaxf(m, st[k].x);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  float z = 0.f;
  for (int k = lane; k < used; k += 64) z += st[k].y * exp2f(st[k].x - m);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) z += __shfl_xor(z, o, 64);
  if (lane == 0) lse2[idx] = m + log2f(z);
}

// grid: (64-row tile of the selection, KV head, cluster). Copies rows [64 u, 64 u + 64) of
// cluster j's selection (selection row j, or j * Hkv + g with one set per KV head) for KV head g;
// rows at or past sel_cnt are written as zeros, tiles past the last partial one are not touched.
template <int D>
__global__ __launch_bounds__(kGatherThreads) void gather_kernel(const uint16_t* __restrict__ k_pages,
                                                                const uint16_t* __restrict__ v_pages,
                                                                const int32_t* __restrict__ block_table,
                                                                const int32_t* __restrict__ sel_idx,
                                                                const int32_t* __restrict__ sel_cnt, int per_kv,
                                                                int top_k, int kpad, int n_tokens, int num_kv_heads,
                                                                int log2_block, uint16_t* __restrict__ gk,
                                                                uint16_t* __restrict__ gv) {
  constexpr int kChunksPerRow = D / 8;
  const int u = blockIdx.x, g = blockIdx.y, j = blockIdx.z;
  const int srow = per_kv ? j * num_kv_heads + g : j;
  int cnt = sel_cnt[srow];
  cnt = cnt < 0 ? 0 : (cnt > top_k ? top_k : cnt);
  if (u * kTokTile >= cnt) return;
  const int32_t* sel = sel_idx + (int64_t)srow * top_k;
  const int64_t dst0 = (((int64_t)j * num_kv_heads + g) * kpad + u * kTokTile) * D;
  for (int idx = threadIdx.x; idx < kTokTile * kChunksPerRow; idx += kGatherThreads) {
    const int r = idx / kChunksPerRow, c = idx % kChunksPerRow;
    const int64_t dst = dst0 + (int64_t)r * D + 8 * c;
    u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
    if (u * kTokTile + r < cnt) {
      int t = sel[u * kTokTile + r];
      t = t < 0 ? 0 : (t >= n_tokens ? n_tokens - 1 : t);
      const int blk = t >> log2_block;
      const int page = block_table ? block_table[blk] : blk;
      const int64_t src = ((((int64_t)page * num_kv_heads + g) << log2_block) + (t & ((1 << log2_block) - 1))) * D + 8 * c;
      kv = *reinterpret_cast<const u32x4*>(k_pages + src);
      vv = *reinterpret_cast<const u32x4*>(v_pages + src);
    }
    *reinterpret_cast<u32x4*>(gk + dst) = kv;
    *reinterpret_cast<u32x4*>(gv + dst) = vv;
  }
}

template <int D, bool kScores>
hipError_t launch_logits_d(int gp, dim3 grid, const TokArgs& a, hipStream_t stream) {
  switch (gp) {
    case 1: token_logits_kernel<D, 1, kScores><<<grid, kTokThreads, 0, stream>>>(a); break;
    case 2: token_logits_kernel<D, 2, kScores><<<grid, kTokThreads, 0, stream>>>(a); break;
    case 4: token_logits_kernel<D, 4, kScores><<<grid, kTokThreads, 0, stream>>>(a); break;
    case 8: token_logits_kernel<D, 8, kScores><<<grid, kTokThreads, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int token_row_pad(int n_clusters, int group) {
  const int gp = token_group_pad(group);
  return (n_clusters * gp + kRowsPerGroup - 1) / kRowsPerGroup * kRowsPerGroup;
}

int token_group_pad(int group) { return group <= 1 ? 1 : group <= 2 ? 2 : group <= 4 ? 4 : 8; }

TokenPlan plan_token_selection(int n_clusters, int group, int, int max_cand) {
  TokenPlan p{};
  p.gp = token_group_pad(group);
  p.r_pad = token_row_pad(n_clusters, group);
  p.n_rowgroups = p.r_pad / kRowsPerGroup;
  // A fixed chunk: a cluster's statistics (and so its scores, bit for bit) do not depend on the
  // other clusters of the call, which keeps incremental calls equal to one-shot ones.
  const int n_tiles = (max_cand + kTokTile - 1) / kTokTile;
  p.tiles_per_chunk = kTokenChunkTiles;
  p.n_chunks = (n_tiles + p.tiles_per_chunk - 1) / p.tiles_per_chunk;
  p.chunk_tokens = p.tiles_per_chunk * kTokTile;
  return p;
}

hipError_t launch_token_selection(const float* fingerprints, const uint16_t* k_pages, const int32_t* block_table,
                                  const ClusterGeo* geo, int n_clusters, int max_cand, int first_token,
                                  int num_q_heads, int num_kv_heads, int head_dim, int block_size,
                                  float score_scale, int64_t cand_stride, uint16_t* F, float2* stats, float* lse2,
                                  float* partial, hipStream_t stream) {
  if (n_clusters <= 0 || max_cand <= 0) return hipSuccess;
  const int group = num_q_heads / num_kv_heads;
  const TokenPlan p = plan_token_selection(n_clusters, group, num_kv_heads, max_cand);
  split_fingerprints_kernel<<<n_clusters, 256, 0, stream>>>(fingerprints, num_q_heads, num_kv_heads, head_dim, p.gp,
                                                           p.r_pad, F);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  TokArgs a{};
  a.k_pages = k_pages;
  a.block_table = block_table;
  a.F = F;
  a.geo = geo;
  a.lse2 = lse2;
  a.stats = stats;
  a.partial = partial;
  a.cand_stride = cand_stride;
  a.n_clusters = n_clusters;
  a.group = group;
  a.r_pad = p.r_pad;
  a.n_rowgroups = p.n_rowgroups;
  a.tiles_per_chunk = p.tiles_per_chunk;
  a.n_chunks = p.n_chunks;
  a.first_token = first_token;
  a.num_kv_heads = num_kv_heads;
  a.log2_block = block_size == 128 ? 7 : 6;
  a.scale2 = score_scale * 1.4426950408889634f;
  const dim3 grid((unsigned)((int64_t)p.n_chunks * p.n_rowgroups * num_kv_heads));
  e = head_dim == 128 ? launch_logits_d<128, false>(p.gp, grid, a, stream) : launch_logits_d<64, false>(p.gp, grid, a, stream);
  if (e != hipSuccess) return e;
  const int n_rows = num_kv_heads * p.r_pad;
  token_lse_kernel<<<(n_rows + 3) / 4, 256, 0, stream>>>(stats, geo, n_clusters, group, p.gp, p.r_pad,
                                                              num_kv_heads, p.n_chunks, p.chunk_tokens, lse2);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return head_dim == 128 ? launch_logits_d<128, true>(p.gp, grid, a, stream) : launch_logits_d<64, true>(p.gp, grid, a, stream);
}

hipError_t launch_gather_selected(const uint16_t* k_pages, const uint16_t* v_pages, const int32_t* block_table,
                                  const int32_t* sel_idx, const int32_t* sel_cnt, bool per_kv, int n_clusters,
                                  int top_k, int kpad, int n_tokens, int num_kv_heads, int head_dim, int block_size,
                                  uint16_t* gk, uint16_t* gv, hipStream_t stream) {
  if (n_clusters <= 0 || top_k <= 0) return hipSuccess;
  const dim3 grid((unsigned)(kpad / kTokTile), (unsigned)num_kv_heads, (unsigned)n_clusters);
  const int lb = block_size == 128 ? 7 : 6;
  if (head_dim == 128)
    gather_kernel<128><<<grid, kGatherThreads, 0, stream>>>(k_pages, v_pages, block_table, sel_idx, sel_cnt,
                                                            per_kv ? 1 : 0, top_k, kpad, n_tokens, num_kv_heads, lb,
                                                            gk, gv);
  else
    gather_kernel<64><<<grid, kGatherThreads, 0, stream>>>(k_pages, v_pages, block_table, sel_idx, sel_cnt,
                                                           per_kv ? 1 : 0, top_k, kpad, n_tokens, num_kv_heads, lb,
                                                           gk, gv);
  return hipGetLastError();
}

}  // namespace scale
