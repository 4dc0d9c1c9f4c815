// Memory-safety run of libzf's host code under AddressSanitizer and
// UndefinedBehaviorSanitizer (built host-only by tests/test_host_asan.py; no
// GPU is touched).  Exercises the multithreaded deferred update on
// exact-size heap buffers in both layouts, padded strides and thread counts,
// and the host-side validation of every entry point that must reject bad
// arguments before any HIP call.  Values are checked against a plain loop
// here (the numerics themselves are pinned against the oracle elsewhere).
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "zf.h"

static int failures = 0;
#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      std::fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #c); \
      ++failures;                                                  \
    }                                                              \
  } while (0)

static uint16_t rne_bf16(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// one case: exact-size heap buffers so that any overrun is reported
static void run_case(int64_t n, int64_t m, int64_t k, int32_t layout, int pad, int threads,
                     unsigned seed) {
  std::mt19937 rng(seed);
  std::normal_distribution<float> nd(0.0f, 1.0f);
  const int64_t u = m - k;
  const bool cm = layout == ZF_LAYOUT_CHANNEL_MAJOR;
  const int64_t ar = cm ? u : n, aw = cm ? n : u, sr = cm ? m : n, sw = cm ? n : m;
  const int64_t lda = aw + pad, lds = sw + pad, ldw = aw + pad;
  const size_t na = ar ? static_cast<size_t>((ar - 1) * lda + aw) : 0;
  const size_t ns = sr ? static_cast<size_t>((sr - 1) * lds + sw) : 0;
  float* acc = static_cast<float*>(std::malloc(std::max<size_t>(na, 1) * 4));
  float* P = static_cast<float*>(std::malloc(std::max<size_t>(ns, 1) * 4));
  float* M = static_cast<float*>(std::malloc(std::max<size_t>(ns, 1) * 4));
  float* V = static_cast<float*>(std::malloc(std::max<size_t>(ns, 1) * 4));
  uint16_t* W = static_cast<uint16_t*>(std::malloc(std::max<size_t>(na, 1) * 2));
  std::vector<int32_t> perm(m);
  for (int64_t j = 0; j < m; ++j) perm[j] = static_cast<int32_t>(j);
  std::shuffle(perm.begin(), perm.end(), rng);
  std::vector<char> is_sel(m, 0);
  for (int64_t r = 0; r < k; ++r) is_sel[perm[r]] = 1;
  std::vector<int32_t> unsel;
  for (int64_t j = 0; j < m; ++j)
    if (!is_sel[j]) unsel.push_back(static_cast<int32_t>(j));
  for (size_t e = 0; e < na; ++e) acc[e] = nd(rng);
  for (size_t e = 0; e < ns; ++e) {
    P[e] = 0.02f * nd(rng);
    M[e] = 1e-3f * nd(rng);
    V[e] = 1e-6f * std::fabs(nd(rng));
  }
  std::vector<float> P0(P, P + ns), M0(M, M + ns), V0(V, V + ns);
  const zf_adam_hparams hp{1e-3, 0.9, 0.999, 1e-8, 0.01};
  const float scale = 0.25f;
  const int st = zf_host_adam_unselected(acc, lda, unsel.empty() ? nullptr : unsel.data(), n, m,
                                         k, layout, scale, P, M, V, lds, W, ldw, &hp, 3, threads);
  CHECK(st == ZF_OK);
  // plain loop of the same element sequence
  const float b1 = 0.9f, b2 = 0.999f, c1 = static_cast<float>(1.0 - 0.9),
              c2 = static_cast<float>(1.0 - 0.999), lr = 1e-3f, eps = 1e-8f,
              wd = static_cast<float>(1e-3 * 0.01);
  const float ib1 = static_cast<float>(1.0 / (1.0 - std::pow(0.9, 3.0)));
  const float ib2 = static_cast<float>(1.0 / (1.0 - std::pow(0.999, 3.0)));
  for (int64_t i = 0; i < n; ++i) {
    for (int64_t q = 0; q < u; ++q) {
      const int64_t j = unsel[q];
      const int64_t ai = cm ? q * lda + i : i * lda + q;
      const int64_t si = cm ? j * lds + i : i * lds + j;
      const float g = acc[ai] * scale;
      float m1 = b1 * M0[si] + c1 * g;
      float v1 = b2 * V0[si] + c2 * (g * g);
      const float d = std::sqrt(v1 * ib2) + eps;
      const float up = (m1 * ib1) / d;
      float p = P0[si] - wd * P0[si];
      p = p - lr * up;
      CHECK(P[si] == p && M[si] == m1 && V[si] == v1);
      CHECK(W[cm ? q * ldw + i : i * ldw + q] == rne_bf16(p));
      if (failures > 20) std::exit(1);
    }
  }
  // selected columns untouched
  for (int64_t r = 0; r < k; ++r) {
    const int64_t j = perm[r];
    for (int64_t i = 0; i < n; ++i) {
      const int64_t si = cm ? j * lds + i : i * lds + j;
      CHECK(P[si] == P0[si] && M[si] == M0[si] && V[si] == V0[si]);
    }
  }
  std::free(acc);
  std::free(P);
  std::free(M);
  std::free(V);
  std::free(W);
}

int main() {
  // k from ratio
  CHECK(zf_k_from_ratio(0.1, 4096) == 410);
  CHECK(zf_k_from_ratio(0.1, 28672) == 2867);
  CHECK(zf_k_from_ratio(1.5, 10) == -1);
  CHECK(zf_k_from_ratio(NAN, 10) == -1);
  for (int s = 0; s <= 4; ++s) CHECK(std::strlen(zf_status_string(s)) > 0);
  CHECK(std::strlen(zf_status_string(99)) > 0);

  // the deferred update, both layouts, ragged shapes, strides, threads
  const int64_t shapes[][3] = {{1, 1, 0}, {1, 1, 1}, {3, 7, 2}, {17, 64, 6}, {64, 130, 13},
                               {257, 33, 3}, {40, 1000, 50}, {9, 9, 9}, {5, 3, 0}};
  unsigned seed = 1;
  for (const auto& s : shapes)
    for (int32_t layout = 0; layout < 2; ++layout)
      for (int pad : {0, 5})
        for (int threads : {1, 3, 16}) run_case(s[0], s[1], s[2], layout, pad, threads, seed++);

  // host-side rejection before any HIP call
  const zf_adam_hparams hp{1e-3, 0.9, 0.999, 1e-8, 0.0};
  const zf_adam_hparams bad{1e-3, 1.0, 0.999, 1e-8, 0.0};
  float buf[64] = {0};
  uint16_t wb[64] = {0};
  int32_t idx[2] = {1, 0};  // not ascending
  CHECK(zf_host_adam_unselected(buf, 2, idx, 2, 4, 2, 0, 1.0f, buf + 8, buf + 16, buf + 24, 4,
                                wb, 2, &hp, 1, 1) == ZF_EINVAL);
  int32_t ok_idx[2] = {0, 1};
  CHECK(zf_host_adam_unselected(buf, 2, ok_idx, 2, 4, 2, 0, 1.0f, buf + 8, buf + 16, buf + 24, 4,
                                wb, 2, &bad, 1, 1) == ZF_EINVAL);
  CHECK(zf_host_adam_unselected(buf, 2, ok_idx, 2, 4, 2, 0, 1.0f, buf + 8, buf + 16, buf + 24, 4,
                                wb, 2, &hp, 0, 1) == ZF_EINVAL);
  CHECK(zf_host_adam_unselected(buf, 2, ok_idx, 2, 4, 2, 0, 1.0f, buf + 8, buf + 16, buf + 24, 4,
                                wb, 2, &hp, 1, -1) == ZF_EINVAL);
  CHECK(zf_colnorm(nullptr, 4, 4, 4, 0, nullptr, nullptr, 0, nullptr) == ZF_EINVAL);
  CHECK(zf_topk_select(nullptr, 4, 0.5, nullptr, nullptr, nullptr) == ZF_EINVAL);
  zf_plan* plan = nullptr;
  size_t plan_bytes = 0;
  CHECK(zf_plan_query(nullptr, 1, &plan_bytes) == ZF_EINVAL);
  CHECK(zf_plan_create(nullptr, 1, nullptr, 0, nullptr, &plan) == ZF_EINVAL);
  {
    // valid (empty) descriptors: sized on the host; create rejects too
    // little memory before any device call
    zf_matrix d[2];
    std::memset(d, 0, sizeof(d));
    d[0].m = 4;
    d[0].k = 1;
    d[1].m = 9;
    d[1].k = 2;
    CHECK(zf_plan_query(d, 2, &plan_bytes) == ZF_OK && plan_bytes >= 256);
    void* fake = reinterpret_cast<void*>(uintptr_t(1) << 40);
    CHECK(zf_plan_create(d, 2, fake, plan_bytes - 1, nullptr, &plan) == ZF_EWORKSPACE);
    CHECK(plan == nullptr);
  }
  CHECK(zf_plan_update(nullptr, &hp, 1, 0, 1, 1, 1, 1, nullptr) == ZF_EINVAL);
  CHECK(zf_plan_update_zen(nullptr, &hp, 1, 0, 1, 4, 1.0, nullptr, nullptr) == ZF_EINVAL);
  CHECK(zf_plan_update_handover(nullptr, &hp, 1, 0, 1, 4, 1.0f, nullptr) == ZF_EINVAL);
  CHECK(zf_plan_scatter_weights(nullptr, nullptr) == ZF_EINVAL);
  zf_plan_destroy(nullptr);

  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("host code clean under the sanitizers\n");
  return 0;
}
