// Host-code sanitizer run: drives every entry point of libscale on random inputs, in the four
// modes (block; block with bound keys and per-KV-head sets; tokens; tokens with per-KV-head sets),
// with more calls per handle than its staging slots, incremental cluster sets and an invalid call;
// checks statuses and that outputs are finite. Only the host code is instrumented:
//
//   hipcc --offload-arch=gfx950 -O1 -g -std=c++17 -fPIC -Xclang -target-feature -Xclang -packed-fp32-ops \
//     -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -shared -I include \
//     paper_2609_31568_amd/csrc/*.hip -x hip paper_2609_31568_amd/csrc/scale_api.cpp -o libscale_asan.so
//   amdclang++ -O1 -g -std=c++17 -D__HIP_PLATFORM_AMD__ -I/opt/rocm/include -I include \
//     -fsanitize=address,undefined -static-libsan tests/c/host_sanitize_driver.cpp ./libscale_asan.so \
//     -L/opt/rocm/lib -lamdhip64 -Wl,-rpath,'$ORIGIN' -o host_sanitize_driver
//   ASAN_OPTIONS=detect_leaks=0 UBSAN_OPTIONS=halt_on_error=1 ./host_sanitize_driver     (on a GPU)
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "scale.h"

#define CHECK(x)                                                           \
  do {                                                                     \
    int _s = (int)(x);                                                     \
    if (_s != 0) {                                                         \
      std::printf("FAIL %s -> %d at line %d\n", #x, _s, __LINE__);         \
      std::fflush(stdout);                                                 \
      std::exit(1);                                                        \
    }                                                                      \
  } while (0)

static uint16_t bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFF + ((u >> 16) & 1);
  return (uint16_t)(u >> 16);
}

int main() {
  const int Hq = 8, Hkv = 2, D = 128, B = 64, L = 256, N = 8192, M = N / L;
  std::mt19937 rng(7);
  std::normal_distribution<float> nd(0.f, 1.f);
  std::vector<uint16_t> hq((size_t)N * Hq * D), hk((size_t)N * Hkv * D), hv((size_t)N * Hkv * D);
  for (auto& x : hq) x = bf16(nd(rng));
  for (auto& x : hk) x = bf16(nd(rng));
  for (auto& x : hv) x = bf16(nd(rng));
  std::vector<int32_t> bt(N / B);
  for (int i = 0; i < N / B; ++i) bt[i] = (i * 7) % (N / B);   // a page permutation
  uint16_t *q, *kp, *vp;
  int32_t *dbt, *sel, *cnt;
  float *krep, *out, *scores;
  CHECK(hipMalloc(&q, hq.size() * 2));
  CHECK(hipMalloc(&kp, hk.size() * 2));
  CHECK(hipMalloc(&vp, hv.size() * 2));
  CHECK(hipMalloc(&dbt, bt.size() * 4));
  CHECK(hipMalloc(&krep, (size_t)(N / B) * Hkv * 2 * D * 4));
  CHECK(hipMalloc(&sel, (size_t)M * Hkv * 4096 * 4));
  CHECK(hipMalloc(&cnt, (size_t)M * Hkv * 4));
  CHECK(hipMalloc(&out, (size_t)N * Hq * D * 4));
  CHECK(hipMalloc(&scores, (size_t)M * Hkv * N * 4));
  CHECK(hipMemcpy(q, hq.data(), hq.size() * 2, hipMemcpyHostToDevice));
  CHECK(hipMemcpy(kp, hk.data(), hk.size() * 2, hipMemcpyHostToDevice));
  CHECK(hipMemcpy(vp, hv.data(), hv.size() * 2, hipMemcpyHostToDevice));
  CHECK(hipMemcpy(dbt, bt.data(), bt.size() * 4, hipMemcpyHostToDevice));
  std::vector<float> hout((size_t)N * Hq * D);

  auto finite = [&](const char* what) {
    CHECK(hipMemcpy(hout.data(), out, hout.size() * 4, hipMemcpyDeviceToHost));
    for (float x : hout)
      if (!std::isfinite(x)) {
        std::printf("FAIL %s: non-finite output\n", what);
        std::exit(1);
      }
    std::printf("ok %s\n", what);
    std::fflush(stdout);
  };

  for (int mode = 0; mode < 4; ++mode) {   // block, block + variants, tokens, tokens + per-KV sets
    scale_config c;
    std::memset(&c, 0, sizeof c);
    c.num_q_heads = Hq;
    c.num_kv_heads = Hkv;
    c.head_dim = D;
    c.block_size = B;
    c.sub_chunk = L;
    c.top_k = mode >= 2 ? 700 : 6;
    c.sink_tokens = 64;
    c.local_window = 512;
    c.max_tokens = N;
    c.max_clusters = M;
    c.select_tokens = mode >= 2;
    c.rep_kind = mode == 1 ? SCALE_REP_BOUNDS : SCALE_REP_MEAN;
    c.kv_head_sets = mode == 1 || mode == 3;
    scale_handle h = nullptr;
    CHECK(scale_init(&c, nullptr, &h));
    CHECK(scale_enable_timing(h, 1));
    for (int rep = 0; rep < 6; ++rep) {   // more calls than the handle's staging slots
      std::vector<int32_t> cs(M + 1);
      int32_t n = 0;
      std::vector<double> band((size_t)M * 7);
      CHECK(scale_cluster_subchunks(h, q, N, 0, 0.2 + 0.1 * rep, 8 * L, 0, cs.data(), &n, band.data()));
      if (c.select_tokens) {
        CHECK(scale_select_cluster_tokens(h, q, N, kp, dbt, cs.data(), n, sel, cnt, scores, nullptr));
      } else {
        CHECK(scale_rep_keys(h, kp, dbt, N, krep));
        CHECK(scale_select_cluster(h, q, N, krep, cs.data(), n, sel, cnt, scores, nullptr));
      }
      CHECK(scale_sparse_prefill(h, q, kp, vp, dbt, N, cs.data(), n, sel, cnt, out));
      // incremental: the second half of the sub-chunks against the whole cache
      std::vector<int32_t> tail = {M / 2, M / 2 + 3, M};
      if (!c.select_tokens) {
        CHECK(scale_rep_keys_range(h, kp, dbt, (M / 2) * L / B, N, krep));
        CHECK(scale_select_cluster(h, q, N, krep, tail.data(), 2, sel, cnt, nullptr, nullptr));
      } else {
        CHECK(scale_select_cluster_tokens(h, q, N, kp, dbt, tail.data(), 2, sel, cnt, nullptr, nullptr));
      }
      CHECK(scale_sparse_prefill(h, q, kp, vp, dbt, N, tail.data(), 2, sel, cnt, out));
    }
    double ms[SCALE_NUM_STAGES];
    int64_t launches[SCALE_NUM_STAGES];
    CHECK(scale_stage_times(h, ms, launches, 1));
    int64_t calls = 0;
    CHECK(scale_retrieval_calls(h, &calls));
    CHECK(hipDeviceSynchronize());
    char what[64];
    std::snprintf(what, sizeof what, "mode %d (%lld calls)", mode, (long long)calls);
    finite(what);
    // errors leave the handle usable
    int32_t bad[3] = {0, 0, M};
    if (scale_sparse_prefill(h, q, kp, vp, dbt, N, bad, 2, sel, cnt, out) != SCALE_ERR_INVALID_ARG) {
      std::printf("FAIL malformed clusters accepted\n");
      return 1;
    }
    scale_free(h);
  }
  CHECK(hipFree(q));
  CHECK(hipFree(kp));
  CHECK(hipFree(vp));
  CHECK(hipFree(dbt));
  CHECK(hipFree(krep));
  CHECK(hipFree(sel));
  CHECK(hipFree(cnt));
  CHECK(hipFree(out));
  CHECK(hipFree(scores));
  std::printf("ok all\n");
  return 0;
}
