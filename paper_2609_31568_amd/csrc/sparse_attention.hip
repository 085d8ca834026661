// Gathered block-sparse flash attention for cluster-level sparse prefill (paper Sec. 5.1.3,
// Eq. 10; the cluster attention step of Algorithm 2, causal).
//
// Work item = (cluster j, KV head g, head group, tile of up to 32 * RB query positions). The
// work-group has GH * RB waves: one per (query head of the head group, 32-position row block); 8
// waves at d = 128 and 12 at d = 64 (two or three per SIMD, as the registers allow), the G query
// heads of a KV head split into G / GH head groups so that every SIMD gets the same number. All of
// them share the K/V tiles staged in LDS, so one 64-key tile fetched from L2 feeds GH * RB * 32
// query rows. The tile sequence of an item is: the sink blocks, the cluster's selected blocks, then
// the local window [lo_blk * B, last position] in 64-key tiles; only tiles reaching a wave's own
// positions need the causal mask. The page of every tile is resolved once per item into an LDS
// table. The selected set is the cluster's row of sel_idx, or the (cluster, KV head) row with one
// set per KV head. Token-level selection (TOK) reads the selected keys from the rows gathered per
// (cluster, KV head); their tiles are marked by negative table entries, and the padding rows of a
// partial last gathered tile are masked like the causal mask.
//
// The launch is persistent: one work-group per CU runs item after item, taking them in work-list
// order from eight queue counters (one per XCD, the others once its own is empty), so no item
// waits for a work-group launch and the CUs end within about one item of each other.
//
// Per 64-key tile and wave (d = head dim, 32 query rows of one head):
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = Q held in registers
//   online softmax  fp32 in base 2 with the softmax scale folded into one fma per score. A
//                   row keeps a reference max that is only raised when a half tile's weights
//                   against it would sum past 2^20 (exact: numerator and denominator share the
//                   reference); no per-tile max is taken, the bf16 weight sum is the check, and
//                   the O rescale is rare
//   O^T += V^T P^T  v_mfma_f32_32x32x16_bf16, A = V^T from LDS (ds_read_b128), B = P straight
//                   from the S^T accumulators (bf16)
// Computing the transposed products keeps query row (lane % 32) in the same lanes for S, the
// running max / sum and the O accumulators, so no LDS round trip is needed between the two
// products. K rows are stored in LDS in a permuted order so that the S^T accumulators of lane half
// h hold the 16 consecutive keys [16h, 16h + 16) of each 32-key block; a 16-key PV step then takes
// 8 consecutive keys from each lane half, which the V^T operand reads as one 16-byte chunk.
//
// Order inside a tile: S(keys 0-31); S(keys 32-63) interleaved with the softmax of keys 0-31;
// PV(0-31) interleaved with the softmax of keys 32-63; PV(32-63) with the stores of the next tile
// into LDS. Each softmax shares a scheduling region with the MFMAs it overlaps (LLVM's
// MFMA / exponential interleave strategy places them), and the stores are unconditional (past the
// last tile they write the idle buffer), so no branch separates them from the last MFMAs.
//
// Pipelining: LDS holds two tile buffers, and two register sets stage the global loads. A tile's
// loads are issued two tiles ahead; they are written to LDS at the end of the tile before it, and
// one barrier per tile separates the phases.
//
// LDS layouts:
//   K   [row][d], row stride d + 8 elements; row 32 b + 8 i + 4 h + j holds key 32 b + 16 h + 4 i + j
//       (operand reads conflict-free)
//   V^T [d][key], row stride 80 dwords; the 32 key-pair dwords of row d start at dword
//       4 ((d / 8) % 8). gfx950 serves a ds_read_b128 in 16-lane passes over 64 banks of 4 bytes,
//       a pass being the four lane quads of one half-wave whose quad index has the same bit
//       parity, and a ds_write_b32 in 32-lane passes over 32 banks (both measured with bank
//       conflict counters). Under that model the stride and rotation make both the operand reads
//       (rows 4q..4q+3 of a pass land on distinct 4-bank groups) and the transposing tile writes
//       (the 8 d-chunks of a pass on distinct bank groups mod 32) conflict-free.
// (ds_read_b64_tr_b16 would avoid the transposing writes, but it sustains well under half the
// bytes per clock of ds_read_b128, and the V operand reads dominate the LDS traffic.)
#include <math.h>

#include <algorithm>

#include "common.h"

namespace scale {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kKeyTile = 64;
constexpr int kQueues = kAttentionQueues;   // work queues, one per XCD of the round-robin placement
constexpr int kDescBatch = 256;       // tile descriptors resolved per batch
constexpr float kWeightSumLimit = 1048576.0f;   // 2^20: bound on a lane's weight sum per half tile

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Weights of one 32-key half against reference mc (= m_ref * c): p = 2^(s c - mc) rounded to
// bf16 into the two P fragments of the half; returns the lane's sum of the bf16 weights.
__device__ __forceinline__ float half_weights(const f32x16& s, float mc, float c, bf16x8 (&pf)[2]) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
  for (int e = 0; e < 16; e += 2) {
    const bf16x2 w = {(__bf16)fast_exp2(fmaf(s[e], c, -mc)), (__bf16)fast_exp2(fmaf(s[e + 1], c, -mc))};
    pf[e / 8][e % 8] = w[0];
    pf[e / 8][e % 8 + 1] = w[1];
    if (e & 2) acc1 = __builtin_amdgcn_fdot2_f32_bf16(w, ones, acc1, false);
    else acc0 = __builtin_amdgcn_fdot2_f32_bf16(w, ones, acc0, false);
  }
  return acc0 + acc1;
}

template <int D, int GH, int RB>
struct AttnShape {
  static constexpr int kWaves = GH * RB;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kKStride = D + 8;                   // elements
  static constexpr int kVtStrideDw = 80;                   // dwords per V^T row
  static constexpr int kKElems = kKeyTile * kKStride;
  static constexpr int kVElems = D * kVtStrideDw * 2;
  static constexpr int kBufElems = kKElems + kVElems;
  static constexpr int kChunks = kKeyTile * D / 8;         // 16-byte chunks of one K tile
  static constexpr int kPer = (kChunks + kThreads - 1) / kThreads;
  static constexpr int kVUnits = (kKeyTile / 2) * (D / 8); // (key pair, 8-wide d chunk) units
  static constexpr int kVPer = (kVUnits + kThreads - 1) / kThreads;
};

// LDS row of tile key r: the permutation that makes lane half h of the S^T accumulators hold
// keys [16h, 16h + 16) of its 32-key block.
__device__ __forceinline__ int k_lds_row(int r) {
  const int k = r & 31;
  return (r & 32) + 8 * ((k >> 2) & 3) + 4 * (k >> 4) + (k & 3);
}

// V unit u = (key pair kp, d chunk c): lanes of a 32-lane group cover 8 consecutive chunks of 4 key
// pairs (coalesced 128-byte global reads, conflict-free transposing LDS writes).
template <int D>
__device__ __forceinline__ void v_unit(int u, int& kp, int& c) {
  const int rest = u >> 5;
  c = (u & 7) + 8 * (rest % (D / 64));
  kp = 4 * (rest / (D / 64)) + ((u >> 3) & 3);
}

template <class S, int D>
__device__ __forceinline__ void load_tile(u32x4 (&kreg)[S::kPer], u32x4 (&vreg)[2 * S::kVPer],
                                          const uint16_t* __restrict__ k_pages,
                                          const uint16_t* __restrict__ v_pages, int64_t base, int tid) {
#pragma unroll
  for (int i = 0; i < S::kPer; ++i) {
    const int idx = tid + i * S::kThreads;
    if (S::kChunks % S::kThreads == 0 || idx < S::kChunks)
      kreg[i] = *reinterpret_cast<const u32x4*>(k_pages + base + (int64_t)(idx / (D / 8)) * D + 8 * (idx % (D / 8)));
  }
#pragma unroll
  for (int i = 0; i < S::kVPer; ++i) {
    const int u = tid + i * S::kThreads;
    if (S::kVUnits % S::kThreads == 0 || u < S::kVUnits) {
      int kp, c;
      v_unit<D>(u, kp, c);
      const uint16_t* src = v_pages + base + (int64_t)(2 * kp) * D + 8 * c;
      vreg[2 * i] = *reinterpret_cast<const u32x4*>(src);
      vreg[2 * i + 1] = *reinterpret_cast<const u32x4*>(src + D);
    }
  }
}

template <class S, int D>
__device__ __forceinline__ void store_tile(const u32x4 (&kreg)[S::kPer], const u32x4 (&vreg)[2 * S::kVPer],
                                           uint16_t* kl, int tid) {
  uint32_t* vt = reinterpret_cast<uint32_t*>(kl + S::kKElems);
#pragma unroll
  for (int i = 0; i < S::kPer; ++i) {
    const int idx = tid + i * S::kThreads;
    if (S::kChunks % S::kThreads == 0 || idx < S::kChunks) {
      const int r = idx / (D / 8), c = idx % (D / 8);
      *reinterpret_cast<u32x4*>(kl + k_lds_row(r) * S::kKStride + 8 * c) = kreg[i];
    }
  }
#pragma unroll
  for (int i = 0; i < S::kVPer; ++i) {
    const int u = tid + i * S::kThreads;
    if (S::kVUnits % S::kThreads == 0 || u < S::kVUnits) {
      int kp, c;
      v_unit<D>(u, kp, c);
      const u32x4 a = vreg[2 * i], b = vreg[2 * i + 1];   // keys 2kp and 2kp+1, d = 8c .. 8c+7
      uint32_t* dst = vt + (8 * c) * S::kVtStrideDw + 4 * (c & 7) + kp;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        dst[(2 * e) * S::kVtStrideDw] = __builtin_amdgcn_perm(b[e], a[e], 0x05040100u);   // low halves
        dst[(2 * e + 1) * S::kVtStrideDw] = __builtin_amdgcn_perm(b[e], a[e], 0x07060302u); // high halves
      }
    }
  }
}

template <int D, int GH, int RB, int LOG2B, bool TOK>
__global__ __launch_bounds__(GH * RB * 64) void sparse_attention_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_pages,
    const uint16_t* __restrict__ v_pages, const int32_t* __restrict__ block_table,
    const ClusterGeo* __restrict__ geo, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ sel_idx, const int32_t* __restrict__ sel_cnt, int per_kv, int top_k,
    int num_q_heads, int num_kv_heads, int n_blocks, float qk_scale_log2, int out_bf16,
    void* __restrict__ out, const uint16_t* __restrict__ gk, const uint16_t* __restrict__ gv, int kpad,
    int n_items, uint32_t* __restrict__ queue) {
  using S = AttnShape<D, GH, RB>;
  constexpr int B = 1 << LOG2B;
  constexpr int kTilesPerBlock = B / kKeyTile;
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * S::kBufElems];
  __shared__ int32_t tile_row[2][kDescBatch];   // first cache row ((page * Hkv + g) * B + off)

  // Persistent work-groups: work-group b serves queue b % kQueues (with the hardware's round-robin
  // placement, one queue per XCD), taking the items b % kQueues, + kQueues, + 2 kQueues, ... of the
  // work list in order from the queue's counter until they run out. A work-group runs item after
  // item without leaving the CU, so no item waits for the launch of a new work-group; a queue
  // balances the CUs that serve it to within one item, and taking from the other queues once its
  // own is empty (below) balances the XCDs.
  // Each item's successor is taken from the queue when the item starts and published at the end of
  // its prologue, so the atomic's latency hides under the prologue's loads; the two slots
  // alternate, and every wave reads a slot (at the end of an item) before the barriers of the next
  // item precede its reuse.
  __shared__ int item_slot[2];
  const int queue_id = blockIdx.x & (kQueues - 1);
  // A take tries the work-group's own queue first and, once that is empty, the others in turn, so
  // CUs of a faster XCD finish the items a slower XCD has left (the stolen items lose their L2
  // locality, which only the last items of a launch pay); n_items when every queue is empty.
  auto take = [&]() {
    for (int i = 0; i < kQueues; ++i) {
      const int qq = (queue_id + i) & (kQueues - 1);
      const int v = qq + kQueues * (int)atomicAdd(&queue[qq], 1u);
      if (v < n_items) return v;
    }
    return n_items;
  };
  if (threadIdx.x == 0) item_slot[0] = take();
  __syncthreads();
  int cur_item = item_slot[0];
  for (int k = 0; cur_item < n_items; ++k) {
    // the successor's atomic is issued here and its result stored at the end of the prologue
    const int successor = threadIdx.x == 0 ? take() : 0;
    const WorkItem it = items[cur_item];
    const ClusterGeo cg = geo[it.cluster];
    const int g = it.kv_head & 0xFFFF;
    // The thread index passes through an empty asm once per item, so nothing derived from it (the
    // operand and staging offsets) is hoisted out of the item loop: kept live across every item,
    // they took registers the prefetch sets need, and the compiler then waited on the prefetches.
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int wave = tid / 64;
    const int lane = tid % 64;
    const int half = lane / 32;
    const int row = lane % 32;
    // query head: KV head g's group of num_q_heads / num_kv_heads heads, head group it.kv_head >> 16
    // of GH of them, then this wave's head in the head group
    const int h = g * (num_q_heads / num_kv_heads) + (it.kv_head >> 16) * GH + wave % GH;
    const int rb = wave / GH;
    const int p0 = it.p0;
    const int wave_p0 = p0 + 32 * rb;
    const int p = wave_p0 + row;
    const bool row_valid = 32 * rb + row < it.n_rows;

    // ---- tile sequence: sink blocks, selected blocks, local window ----
    const int srow = per_kv ? it.cluster * num_kv_heads + g : it.cluster;   // selection row
    int n_sel = sel_cnt[srow];
    n_sel = n_sel < 0 ? 0 : (n_sel > top_k ? top_k : n_sel);
    const int n_sink_tiles = cg.sink_eff * kTilesPerBlock;
    // token-level selection: the selected keys are n_sel gathered rows, the last tile padded
    const int n_fixed = n_sink_tiles + (TOK ? (n_sel + kKeyTile - 1) / kKeyTile : n_sel * kTilesPerBlock);
    const int sel_rem = TOK ? n_sel % kKeyTile : 0;
    const int local0 = cg.lo_blk << LOG2B;
    const int local_end = p0 + it.n_rows;            // keys [local0, local_end) of the window
    const int n_tiles = n_fixed + (local_end - local0 + kKeyTile - 1) / kKeyTile;
    const int32_t* sel = sel_idx + (int64_t)srow * top_k;

    auto fill_batch = [&](int batch) {
      const int t0 = batch * kDescBatch;
      const int cnt = min(kDescBatch, n_tiles - t0);
      for (int i = tid; i < cnt; i += S::kThreads) {
        const int t = t0 + i;
        int key0;
        if (t < n_sink_tiles) {
          key0 = t * kKeyTile;
        } else if (TOK && t < n_fixed) {
          // gathered row of the selection, marked by a negative entry
          tile_row[batch & 1][i] = -1 - ((it.cluster * num_kv_heads + g) * kpad + (t - n_sink_tiles) * kKeyTile);
          continue;
        } else if (t < n_fixed) {
          const int u = t - n_sink_tiles;
          int blk = sel[u / kTilesPerBlock];
          blk = blk < 0 ? 0 : (blk >= n_blocks ? n_blocks - 1 : blk);
          key0 = (blk << LOG2B) + (u % kTilesPerBlock) * kKeyTile;
        } else {
          key0 = local0 + (t - n_fixed) * kKeyTile;
        }
        const int blk = key0 >> LOG2B;
        const int page = block_table ? block_table[blk] : blk;
        tile_row[batch & 1][i] = ((page * num_kv_heads + g) << LOG2B) + (key0 & (B - 1));
      }
    };

    // ---- per-thread prefetch registers: two sets, each one K and one V tile ----
    u32x4 kreg0[S::kPer], vreg0[2 * S::kVPer], kreg1[S::kPer], vreg1[2 * S::kVPer];
    auto load_at = [&](int t, u32x4 (&kr)[S::kPer], u32x4 (&vr)[2 * S::kVPer]) {
      const int r = tile_row[(t / kDescBatch) & 1][t % kDescBatch];
      const uint16_t* kp = k_pages;
      const uint16_t* vp = v_pages;
      int64_t row = r;
      if constexpr (TOK) {
        if (r < 0) {
          kp = gk;
          vp = gv;
          row = -1 - (int64_t)r;
        }
      }
      load_tile<S, D>(kr, vr, kp, vp, row * D, tid);
    };

    // ---- Q fragments: B operand of S^T = K Q^T for each 16-wide slice of d ----
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
    float m_ref = -1e30f;      // reference max (raw score units) of this lane's row
    float l_run = 0.f;         // this lane's share of the row's softmax denominator

    // Per-lane LDS element offsets of the operand reads (immediate offsets add the rest).
    const int k_off = row * S::kKStride + 8 * half;
    // V^T row 32 db + row starts its keys at dword 4 ((32 db + row) / 8 % 8); lane half h reads keys
    // 16h + [0, 16) of each 32-key block, the 16-byte chunk of keys 32 kb + 16 h + 8 u at dword
    // offset 16 kb + 8 h + 4 u.
    int vt_off[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
      vt_off[db] = 2 * ((32 * db + row) * S::kVtStrideDw + 4 * ((4 * db + row / 8) & 7) + 8 * half);

    fill_batch(0);
    __syncthreads();
    if (n_tiles > kDescBatch) fill_batch(1);
    // Tile j's global loads are issued two tiles ahead, in iteration j - 2, into register set j % 2,
    // and stored into LDS buffer j % 2 at the end of iteration j - 1. Loads past the last tile
    // re-read the last tile (never stored), which keeps the wait counts static.
    if (n_tiles > 0) {
      load_at(0, kreg0, vreg0);
      store_tile<S, D>(kreg0, vreg0, lds, tid);
      load_at(min(1, n_tiles - 1), kreg1, vreg1);
    }
    if (threadIdx.x == 0) item_slot[(k + 1) & 1] = successor;
    __syncthreads();

    auto body = [&](int t, u32x4 (&kl)[S::kPer], u32x4 (&vl)[2 * S::kVPer], u32x4 (&ks)[S::kPer],
                    u32x4 (&vs)[2 * S::kVPer]) {
      const int buf = t & 1;
      if (t > 0 && t % kDescBatch == 0 && t + kDescBatch < n_tiles) fill_batch(t / kDescBatch + 1);
      load_at(min(t + 2, n_tiles - 1), kl, vl);

      const uint16_t* k_lds = lds + buf * S::kBufElems;
      const uint16_t* v_lds = k_lds + S::kKElems;

      // S^T of half 0, then S^T of half 1 interleaved with the softmax of half 0, then PV of half 0
      // interleaved with the softmax of half 1, then PV of half 1.
      auto s_half = [&](int kb, f32x16& acc) {
        const uint16_t* krow = k_lds + k_off + 32 * kb * S::kKStride;
        bf16x8 kf[D / 16];
#pragma unroll
        for (int c = 0; c < D / 16; ++c) kf[c] = *reinterpret_cast<const bf16x8*>(krow + 16 * c);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[0], qf[0], f32x16{}, 0, 0, 0);
#pragma unroll
        for (int c = 1; c < D / 16; ++c) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[c], qf[c], acc, 0, 0, 0);
      };
      auto mask_half = [&](int kb, f32x16& sc) {
        if constexpr (TOK) {
          // One branch for both masks: a local tile masks the keys after the row's own position, the
          // last gathered tile its padding after the last selected row. A separate branch for the
          // padding lets the compiler hoist its 16 lane masks into scalar registers, which spill,
          // and splits the MFMA chains it sits between.
          bool need = false;
          int last = 0;   // last visible key of the tile, relative to the tile's first key
          if (t >= n_fixed) {
            const int key0 = local0 + (t - n_fixed) * kKeyTile;
            need = key0 + kKeyTile > wave_p0;
            last = p - key0;
          } else if (sel_rem != 0 && t == n_fixed - 1) {
            need = true;
            last = sel_rem - 1;
          }
          if (need) {
            const int lim = last - 16 * half;
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (32 * kb + e > lim) sc[e] = -INFINITY;
          }
        } else if (t >= n_fixed) {
          const int key0 = local0 + (t - n_fixed) * kKeyTile;
          if (key0 + kKeyTile > wave_p0) {
            const int lim = p - key0 - 16 * half;
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (32 * kb + e > lim) sc[e] = -INFINITY;
          }
        }
      };
      auto finish = [&](const f32x16& sc, float lsum, bf16x8 (&pf)[2]) {
        if (__any(!(lsum <= kWeightSumLimit))) {
          float mt = fmaxf(sc[0], sc[1]);
#pragma unroll
          for (int e = 2; e < 16; ++e) mt = fmaxf(mt, sc[e]);
          mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
          const float m_new = fmaxf(m_ref, mt);
          const float alpha = fast_exp2((m_ref - m_new) * qk_scale_log2);
          l_run *= alpha;
#pragma unroll
          for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[db][e] *= alpha;
          m_ref = m_new;
          lsum = half_weights(sc, m_ref * qk_scale_log2, qk_scale_log2, pf);
        }
        l_run += lsum;
      };
      auto pv_half = [&](int kb, const bf16x8 (&pf)[2]) {
        bf16x8 vf[D / 32][2];
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int u = 0; u < 2; ++u) vf[db][u] = *reinterpret_cast<const bf16x8*>(v_lds + vt_off[db] + 2 * (16 * kb + 4 * u));
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int u = 0; u < 2; ++u) o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db][u], pf[u], o[db], 0, 0, 0);
      };
      f32x16 s0, s1;
      bf16x8 pf0[2], pf1[2];
      s_half(0, s0);
      mask_half(0, s0);
      {
        s_half(1, s1);
        const float l0 = half_weights(s0, m_ref * qk_scale_log2, qk_scale_log2, pf0);
        __builtin_amdgcn_iglp_opt(2);   // interleave the exponentials with the MFMAs
        finish(s0, l0, pf0);
      }
      mask_half(1, s1);
      {
        pv_half(0, pf0);
        const float l1 = half_weights(s1, m_ref * qk_scale_log2, qk_scale_log2, pf1);
        __builtin_amdgcn_iglp_opt(2);
        finish(s1, l1, pf1);
      }
      pv_half(1, pf1);

      // Past the last tile this stores the re-read last tile into the idle buffer: unconditional, so
      // the stores share a scheduling region with the last PV MFMAs.
      store_tile<S, D>(ks, vs, lds + (buf ^ 1) * S::kBufElems, tid);
      __syncthreads();
    };
    for (int t = 0; t < n_tiles; t += 2) {
      body(t, kreg0, vreg0, kreg1, vreg1);
      if (t + 1 < n_tiles) body(t + 1, kreg1, vreg1, kreg0, vreg0);
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    const float inv = 1.0f / l_tot;
    if (row_valid) {
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
    cur_item = item_slot[(k + 1) & 1];   // written before this item's last prologue barrier
  }
  // The last work-group to leave clears the counters for the next launch on the stream: every other
  // work-group made its last grab before its own increment of the leave counter.
  if (threadIdx.x == 0) {
    __threadfence();
    if (atomicAdd(&queue[kQueues], 1u) == gridDim.x - 1)
      for (int i = 0; i <= kQueues; ++i) atomicExch(&queue[i], 0u);
  }
}

// Shape of the work-group: GH query heads (a head group of the G heads of a KV head) times RB row
// blocks, one wave each, one work-group per CU (its LDS). At d = 128 a wave needs 224-232 VGPRs,
// so two waves share a SIMD and a work-group has 8; at d = 64 it needs about 140, so three share a
// SIMD and a work-group has 12. GH is the largest divisor of G that fills the waves exactly (8 at
// d = 128: GH = 1 for G = 3, 5, 7, GH = 2 for G = 6; 12 at d = 64: GH = 1 for G = 5, 7, GH = 4
// for G = 8), so every SIMD carries the same number of waves.
constexpr int waves_per_group(int d) { return d == 64 ? 12 : 8; }
constexpr int heads_per_group(int group, int d) {
  for (int gh = group; gh > 1; --gh)
    if (group % gh == 0 && waves_per_group(d) % gh == 0) return gh;
  return 1;
}
constexpr int row_blocks(int gh, int d) { return waves_per_group(d) / gh; }

struct LaunchArgs {
  const uint16_t *q, *k_pages, *v_pages;
  const int32_t* block_table;
  const ClusterGeo* geo;
  const WorkItem* items;
  int n_items;
  const int32_t *sel_idx, *sel_cnt;
  int per_kv, top_k, num_q_heads, num_kv_heads, n_blocks;
  float qk_scale_log2;
  int out_bf16;
  void* out;
  const uint16_t *gk, *gv;
  int kpad;
  uint32_t* queue;
  hipStream_t stream;
};

// Work-groups of a persistent launch: as many as fit on the device at once (one per CU for every
// shape here), at least one per queue that holds an item, never more than there are items.
template <class K>
int persistent_grid(K kernel, int threads, int n_items) {
  // the kernel's resident work-groups per CU (the same on every gfx950 device), found once
  // (initialisation of a local static is thread-safe)
  static const int per_cu = [&]() {
    int n = 0;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) == hipSuccess && n >= 1 ? n : 1;
  }();
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess || cus < 1)
    cus = 1;
  return std::min(n_items, std::max(cus * per_cu, kQueues));
}

template <int D, int GH, int LOG2B, bool TOK>
hipError_t launch_dgbt(const LaunchArgs& a) {
  constexpr int RB = row_blocks(GH, D);
  constexpr int kThreads = GH * RB * 64;
  auto kernel = sparse_attention_kernel<D, GH, RB, LOG2B, TOK>;
  kernel<<<persistent_grid(kernel, kThreads, a.n_items), kThreads, 0, a.stream>>>(
      a.q, a.k_pages, a.v_pages, a.block_table, a.geo, a.items, a.sel_idx, a.sel_cnt, a.per_kv, a.top_k,
      a.num_q_heads, a.num_kv_heads, a.n_blocks, a.qk_scale_log2, a.out_bf16, a.out, TOK ? a.gk : nullptr,
      TOK ? a.gv : nullptr, TOK ? a.kpad : 0, a.n_items, a.queue);
  return hipGetLastError();
}

template <int D, int GH, int LOG2B>
hipError_t launch_dgb(const LaunchArgs& a) {
  return a.gk ? launch_dgbt<D, GH, LOG2B, true>(a) : launch_dgbt<D, GH, LOG2B, false>(a);
}

template <int D, int GH>
hipError_t launch_dg(int block_size, const LaunchArgs& a) {
  return block_size == 128 ? launch_dgb<D, GH, 7>(a) : launch_dgb<D, GH, 6>(a);
}

template <int D>
hipError_t launch_d(int group, int block_size, const LaunchArgs& a) {
  switch (heads_per_group(group, D)) {
    case 1: return launch_dg<D, 1>(block_size, a);
    case 2: return launch_dg<D, 2>(block_size, a);
    case 3: if constexpr (D == 64) return launch_dg<D, 3>(block_size, a); else return hipErrorInvalidValue;
    case 4: return launch_dg<D, 4>(block_size, a);
    case 6: if constexpr (D == 64) return launch_dg<D, 6>(block_size, a); else return hipErrorInvalidValue;
    case 8: if constexpr (D == 128) return launch_dg<D, 8>(block_size, a); else return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int attention_tile_positions(int group, int head_dim) {
  return 32 * (head_dim == 64 ? row_blocks(heads_per_group(group, 64), 64)
                              : row_blocks(heads_per_group(group, 128), 128));
}
int attention_head_groups(int group, int head_dim) {
  return group / (head_dim == 64 ? heads_per_group(group, 64) : heads_per_group(group, 128));
}

hipError_t launch_sparse_attention(const uint16_t* q, const uint16_t* k_pages, const uint16_t* v_pages,
                                   const int32_t* block_table, const ClusterGeo* geo,
                                   const WorkItem* items, int n_items, const int32_t* sel_idx,
                                   const int32_t* sel_cnt, bool per_kv, int top_k, int num_q_heads,
                                   int num_kv_heads, int head_dim, int block_size, int n_blocks,
                                   float qk_scale_log2, int out_bf16, void* out, const uint16_t* gk,
                                   const uint16_t* gv, int kpad, uint32_t* queue, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  LaunchArgs a{};
  a.q = q;
  a.k_pages = k_pages;
  a.v_pages = v_pages;
  a.block_table = block_table;
  a.geo = geo;
  a.items = items;
  a.n_items = n_items;
  a.sel_idx = sel_idx;
  a.sel_cnt = sel_cnt;
  a.per_kv = per_kv ? 1 : 0;
  a.top_k = top_k;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.n_blocks = n_blocks;
  a.qk_scale_log2 = qk_scale_log2;
  a.out_bf16 = out_bf16;
  a.out = out;
  a.gk = gk;
  a.gv = gv;
  a.kpad = kpad;
  a.queue = queue;
  a.stream = stream;
  const int group = num_q_heads / num_kv_heads;
  return head_dim == 128 ? launch_d<128>(group, block_size, a) : launch_d<64>(group, block_size, a);
}

}  // namespace scale
