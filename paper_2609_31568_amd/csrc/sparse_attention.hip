// Gathered block-sparse flash attention for cluster-level sparse prefill (paper Sec. 5.1.3,
// Eq. 10; Algorithm 2, "compute cluster attention ... with causal mask").
//
// Work item = (cluster j, KV head g, tile of up to 32 query positions). The work-group has one
// wave per query head of the group (G = Hq / Hkv waves); all of them share every K/V tile that
// is staged in LDS. The tile sequence of an item is: the sink blocks, the cluster's selected
// blocks, then the local window [lo_blk * B, last position] in 64-key tiles; only the tile that
// reaches the item's own positions needs the causal mask.
//
// Per 64-key tile and wave (d = head dim, 32 query rows of one head):
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = Q held in registers
//   online softmax  fp32, base-2 exponent with the softmax scale folded into log2(e)
//   O^T += V^T P^T  v_mfma_f32_32x32x16_bf16, A = V^T from LDS, B = P straight from the S^T
//                   accumulators (bf16)
// Computing the transposed products keeps query row (lane % 32) in the same lanes for S, the
// running max / sum and the O accumulators, so no LDS round trip is needed between the two
// products. The key order inside a 16-key MFMA step is permuted consistently on both operands
// (lane half 0 holds keys {0-3, 8-11}, lane half 1 keys {4-7, 12-15}), which is what the
// accumulator layout of the first product hands to the second.
#include <math.h>

#include "common.h"

namespace scale {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kKeyTile = 64;                 // keys per LDS tile
constexpr int kVtPad = 4;                    // V^T row padding (elements)
constexpr int kKPad = 8;                     // K row padding (elements)

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void sparse_attention_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_pages,
    const uint16_t* __restrict__ v_pages, const int32_t* __restrict__ block_table,
    const ClusterGeo* __restrict__ geo, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ sel_idx, const int32_t* __restrict__ sel_cnt, int top_k,
    int num_q_heads, int num_kv_heads, int block_size, int n_blocks, float qk_scale_log2,
    int out_bf16, void* __restrict__ out) {
  constexpr int kThreads = NW * 64;
  constexpr int kKStride = D + kKPad;
  constexpr int kVtStride = kKeyTile + kVtPad;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kKeyTile * kKStride];
  __shared__ __attribute__((aligned(16))) uint16_t vt_lds[D * kVtStride];

  const WorkItem it = items[blockIdx.x];
  const ClusterGeo cg = geo[it.cluster];
  const int g = it.kv_head;
  const int wave = threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  const int half = lane / 32;
  const int row = lane % 32;
  const int h = g * NW + wave;
  const int p0 = it.p0;
  const int p = p0 + row;
  const bool row_valid = row < it.n_rows;

  // Q fragments: B operand of S^T = K Q^T for each 16-wide slice of d.
  bf16x8 qf[D / 16];
  {
    const int pr = row_valid ? p : p0;
    const uint16_t* qrow = q + ((int64_t)pr * num_q_heads + h) * D + 8 * half;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) qf[c] = *reinterpret_cast<const bf16x8*>(qrow + 16 * c);
  }

  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[db][e] = 0.f;
  float m_run = -INFINITY;
  float l_run = 0.f;

  const int tiles_per_block = block_size / kKeyTile;
  int n_sel = sel_cnt[it.cluster];
  n_sel = n_sel < 0 ? 0 : (n_sel > top_k ? top_k : n_sel);
  const int n_sink_tiles = cg.sink_eff * tiles_per_block;
  const int n_sel_tiles = n_sel * tiles_per_block;
  const int local0 = cg.lo_blk * block_size;
  const int local_end = p0 + it.n_rows;            // keys [local0, local_end) of the window
  const int n_local_tiles = (local_end - local0 + kKeyTile - 1) / kKeyTile;
  const int n_tiles = n_sink_tiles + n_sel_tiles + n_local_tiles;
  const int32_t* sel = sel_idx + (int64_t)it.cluster * top_k;

  for (int t = 0; t < n_tiles; ++t) {
    int key0;
    if (t < n_sink_tiles) {
      key0 = t * kKeyTile;
    } else if (t < n_sink_tiles + n_sel_tiles) {
      const int u = t - n_sink_tiles;
      int blk = sel[u / tiles_per_block];
      blk = blk < 0 ? 0 : (blk >= n_blocks ? n_blocks - 1 : blk);
      key0 = blk * block_size + (u % tiles_per_block) * kKeyTile;
    } else {
      key0 = local0 + (t - n_sink_tiles - n_sel_tiles) * kKeyTile;
    }
    const int blk = key0 / block_size;
    const int page = block_table ? block_table[blk] : blk;
    const int64_t base = (((int64_t)page * num_kv_heads + g) * block_size + (key0 - blk * block_size)) * D;
    const uint16_t* kt = k_pages + base;
    const uint16_t* vt = v_pages + base;

    __syncthreads();   // every wave is done with the previous tile
    // K tile: [key][d] rows of 16-byte chunks.
    for (int i = threadIdx.x; i < kKeyTile * D / 8; i += kThreads) {
      const int r = i / (D / 8), c = i % (D / 8);
      *reinterpret_cast<uint4*>(k_lds + r * kKStride + 8 * c) =
          *reinterpret_cast<const uint4*>(kt + (int64_t)r * D + 8 * c);
    }
    // V tile transposed: [d][key], two keys per 32-bit store.
    for (int i = threadIdx.x; i < (kKeyTile / 2) * (D / 8); i += kThreads) {
      const int c = i % (D / 8), kp = i / (D / 8);
      const uint4 a = *reinterpret_cast<const uint4*>(vt + (int64_t)(2 * kp) * D + 8 * c);
      const uint4 b = *reinterpret_cast<const uint4*>(vt + (int64_t)(2 * kp + 1) * D + 8 * c);
      const uint32_t wa[4] = {a.x, a.y, a.z, a.w};
      const uint32_t wb[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint32_t* dst0 = reinterpret_cast<uint32_t*>(vt_lds + (8 * c + 2 * e) * kVtStride + 2 * kp);
        uint32_t* dst1 = reinterpret_cast<uint32_t*>(vt_lds + (8 * c + 2 * e + 1) * kVtStride + 2 * kp);
        *dst0 = (wa[e] & 0xFFFFu) | (wb[e] << 16);
        *dst1 = (wa[e] >> 16) | (wb[e] & 0xFFFF0000u);
      }
    }
    __syncthreads();

    // S^T for the two 32-key halves of the tile.
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[kb][e] = 0.f;
      const uint16_t* krow = k_lds + (32 * kb + row) * kKStride + 8 * half;
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + 16 * c);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[c], s[kb], 0, 0, 0);
      }
    }

    // Scale into base 2, causal mask on the tile that reaches this item's positions.
    const bool diag = key0 + kKeyTile > p0;
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float x = s[kb][e] * qk_scale_log2;
        if (diag) {
          const int key = key0 + 32 * kb + 8 * (e / 4) + 4 * half + (e % 4);
          if (key > p) x = -INFINITY;
        }
        s[kb][e] = x;
        mt = fmaxf(mt, x);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float pv = fast_exp2(s[kb][e] - m_use);
        s[kb][e] = pv;
        psum += pv;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[db][e] *= alpha;

    // P fragments: key chunk kc = 2 kb + u takes accumulator entries [8u, 8u + 8) of s[kb].
    bf16x8 pf[4];
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[kc][e] = (__bf16)s[kc / 2][8 * (kc % 2) + e];

    // O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const uint16_t* vrow = vt_lds + (32 * db + row) * kVtStride + 4 * half;
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow + 16 * kc);
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 16 * kc + 8);
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kc], o[db], 0, 0, 0);
      }
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  if (!row_valid) return;
  const int64_t obase = ((int64_t)p * num_q_heads + h) * D;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int dcol = 32 * db + 8 * i + 4 * half;
      const float r0 = o[db][4 * i + 0] * inv, r1 = o[db][4 * i + 1] * inv;
      const float r2 = o[db][4 * i + 2] * inv, r3 = o[db][4 * i + 3] * inv;
      if (out_bf16) {
        const bf16x4 v = {(__bf16)r0, (__bf16)r1, (__bf16)r2, (__bf16)r3};
        *reinterpret_cast<bf16x4*>(reinterpret_cast<uint16_t*>(out) + obase + dcol) = v;
      } else {
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(out) + obase + dcol) = make_float4(r0, r1, r2, r3);
      }
    }
}

template <int D, int NW>
hipError_t launch_nw(const uint16_t* q, const uint16_t* k_pages, const uint16_t* v_pages,
                     const int32_t* block_table, const ClusterGeo* geo, const WorkItem* items,
                     int n_items, const int32_t* sel_idx, const int32_t* sel_cnt, int top_k,
                     int num_q_heads, int num_kv_heads, int block_size, int n_blocks,
                     float qk_scale_log2, int out_bf16, void* out, hipStream_t stream) {
  sparse_attention_kernel<D, NW><<<n_items, NW * 64, 0, stream>>>(
      q, k_pages, v_pages, block_table, geo, items, sel_idx, sel_cnt, top_k, num_q_heads, num_kv_heads,
      block_size, n_blocks, qk_scale_log2, out_bf16, out);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(int group, const uint16_t* q, const uint16_t* k_pages, const uint16_t* v_pages,
                    const int32_t* block_table, const ClusterGeo* geo, const WorkItem* items, int n_items,
                    const int32_t* sel_idx, const int32_t* sel_cnt, int top_k, int num_q_heads,
                    int num_kv_heads, int block_size, int n_blocks, float qk_scale_log2, int out_bf16,
                    void* out, hipStream_t stream) {
#define SCALE_NW_CASE(NWV)                                                                              \
  case NWV:                                                                                            \
    return launch_nw<D, NWV>(q, k_pages, v_pages, block_table, geo, items, n_items, sel_idx, sel_cnt,  \
                             top_k, num_q_heads, num_kv_heads, block_size, n_blocks, qk_scale_log2,    \
                             out_bf16, out, stream);
  switch (group) {
    SCALE_NW_CASE(1)
    SCALE_NW_CASE(2)
    SCALE_NW_CASE(3)
    SCALE_NW_CASE(4)
    SCALE_NW_CASE(5)
    SCALE_NW_CASE(6)
    SCALE_NW_CASE(7)
    SCALE_NW_CASE(8)
    default:
      return hipErrorInvalidValue;
  }
#undef SCALE_NW_CASE
}

}  // namespace

hipError_t launch_sparse_attention(const uint16_t* q, const uint16_t* k_pages, const uint16_t* v_pages,
                                   const int32_t* block_table, const ClusterGeo* geo,
                                   const WorkItem* items, int n_items, const int32_t* sel_idx,
                                   const int32_t* sel_cnt, int top_k, int num_q_heads,
                                   int num_kv_heads, int head_dim, int block_size, int n_blocks,
                                   float qk_scale_log2, int out_bf16, void* out, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  const int group = num_q_heads / num_kv_heads;
  if (head_dim == 128)
    return launch_d<128>(group, q, k_pages, v_pages, block_table, geo, items, n_items, sel_idx, sel_cnt, top_k,
                         num_q_heads, num_kv_heads, block_size, n_blocks, qk_scale_log2, out_bf16, out, stream);
  return launch_d<64>(group, q, k_pages, v_pages, block_table, geo, items, n_items, sel_idx, sel_cnt, top_k,
                      num_q_heads, num_kv_heads, block_size, n_blocks, qk_scale_log2, out_bf16, out, stream);
}

}  // namespace scale
