// A C++ consumer of libzf that uses only include/zf.h and the HIP runtime
// (no Python, no torch): device buffers from hipMalloc, one stream, the
// single-matrix calls and a two-matrix plan, in both layouts.  Checks what
// the definitions fix, computed here on the host:
//   * scores: s_j = sum_i g_ij^2 (fp64 sum of exact squares, compared within
//     1e-5 relative);
//   * selection: sel / unsel partition [0, m) in ascending order, |sel| = k,
//     every selected score >= every unselected score, mask / prefix
//     consistent with sel;
//   * update at step 1 (fresh states from W) followed by the last step of an
//     interval with the fused hand-over (scale 0.5): the hand-over is +0.0
//     at selected channels and 0.5 * (g1 + g2) at the others (exact fp32
//     operations), the packed buffer keeps g1;
//   * the plan over two matrices gives the same bits as the single calls;
//   * so do plans with deferred packing (zf_plan_update_handover_deferred)
//     and, channel-major, Zen-auto on the device with deferred packing
//     (zf_plan_update_zen_deferred ending the interval by force at step 2,
//     zf_plan_handover_zen_deferred then writing nothing).
// Built by __graft_entry__.build() next to this file; run by
// tests/test_gpu_abi_native.py.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>
#include <random>
#include <vector>

#include "zf.h"

#define HIP_OK(x)                                                              \
  do {                                                                         \
    hipError_t e_ = (x);                                                       \
    if (e_ != hipSuccess) {                                                    \
      std::fprintf(stderr, "HIP error %d at %s:%d\n", int(e_), __FILE__, __LINE__); \
      std::exit(2);                                                            \
    }                                                                          \
  } while (0)
#define ZF_OK_(x)                                                              \
  do {                                                                         \
    int s_ = (x);                                                              \
    if (s_ != ZF_OK) {                                                         \
      std::fprintf(stderr, "%s at %s:%d\n", zf_status_string(s_), __FILE__, __LINE__); \
      std::exit(3);                                                            \
    }                                                                          \
  } while (0)

static int failures = 0;
#define CHECK(c)                                                               \
  do {                                                                         \
    if (!(c)) {                                                                \
      if (failures < 20) std::fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #c); \
      ++failures;                                                              \
    }                                                                          \
  } while (0)

static float widen(uint16_t b) {
  const uint32_t u = static_cast<uint32_t>(b) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

static uint16_t to_bf16(float x) {  // round to nearest even (finite inputs)
  uint32_t u;
  std::memcpy(&u, &x, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T>
static T* dev_alloc(size_t count) {
  void* p = nullptr;
  HIP_OK(hipMalloc(&p, std::max<size_t>(count, 1) * sizeof(T)));
  return static_cast<T*>(p);
}

template <typename T>
static std::vector<T> down(const T* d, size_t count) {
  std::vector<T> h(count);
  if (count) HIP_OK(hipMemcpy(h.data(), d, count * sizeof(T), hipMemcpyDeviceToHost));
  return h;
}

template <typename T>
static bool same_bits(const std::vector<T>& a, const std::vector<T>& b) {
  return a.size() == b.size() && (a.empty() || std::memcmp(a.data(), b.data(), a.size() * sizeof(T)) == 0);
}

template <typename T>
static void up(T* d, const std::vector<T>& h) {
  if (!h.empty()) HIP_OK(hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
}

struct Mat {
  int64_t n, m, k;
  int32_t layout;
  std::vector<uint16_t> g1, g2, w;  // logical [n][m], stored in `layout`
  uint16_t *G1, *G2, *W;
  float *P, *M, *V, *A, *D, *norms;
  zf_selection sel;
  int64_t ld_g() const { return layout == ZF_LAYOUT_ROW_MAJOR ? m : n; }
  int64_t ld_s() const { return layout == ZF_LAYOUT_ROW_MAJOR ? k : n; }
  int64_t ld_a() const { return layout == ZF_LAYOUT_ROW_MAJOR ? m - k : n; }
  size_t at(int64_t i, int64_t j) const {  // storage index of logical (i, j)
    return layout == ZF_LAYOUT_ROW_MAJOR ? size_t(i * m + j) : size_t(j * n + i);
  }
};

static Mat make(int64_t n, int64_t m, double ratio, int32_t layout, unsigned seed) {
  Mat x;
  x.n = n;
  x.m = m;
  x.k = zf_k_from_ratio(ratio, m);
  x.layout = layout;
  std::mt19937 rng(seed);
  std::normal_distribution<float> nd(0.0f, 1.0f);
  std::vector<float> scale(m);
  for (auto& s : scale) s = std::exp(1.5f * nd(rng));
  x.g1.resize(n * m);
  x.g2.resize(n * m);
  x.w.resize(n * m);
  for (int64_t i = 0; i < n; ++i)
    for (int64_t j = 0; j < m; ++j) {
      x.g1[x.at(i, j)] = to_bf16(nd(rng) * scale[j]);
      x.g2[x.at(i, j)] = to_bf16(nd(rng) * scale[j]);
      x.w[x.at(i, j)] = to_bf16(0.02f * nd(rng));
    }
  x.G1 = dev_alloc<uint16_t>(n * m);
  x.G2 = dev_alloc<uint16_t>(n * m);
  x.W = dev_alloc<uint16_t>(n * m);
  up(x.G1, x.g1);
  up(x.G2, x.g2);
  up(x.W, x.w);
  x.P = dev_alloc<float>(n * x.k);
  x.M = dev_alloc<float>(n * x.k);
  x.V = dev_alloc<float>(n * x.k);
  x.A = dev_alloc<float>(n * (m - x.k));
  x.D = dev_alloc<float>(n * m);
  x.norms = dev_alloc<float>(m);
  const int64_t words = (m + 63) / 64;
  x.sel.sel_idx = dev_alloc<int32_t>(x.k);
  x.sel.unsel_idx = dev_alloc<int32_t>(m - x.k);
  x.sel.sel_mask = dev_alloc<uint64_t>(words);
  x.sel.sel_prefix = dev_alloc<int32_t>(words);
  return x;
}

static void release(Mat& x) {
  for (void* p : {static_cast<void*>(x.G1), static_cast<void*>(x.G2), static_cast<void*>(x.W),
                  static_cast<void*>(x.P), static_cast<void*>(x.M), static_cast<void*>(x.V),
                  static_cast<void*>(x.A), static_cast<void*>(x.D), static_cast<void*>(x.norms),
                  static_cast<void*>(x.sel.sel_idx), static_cast<void*>(x.sel.unsel_idx),
                  static_cast<void*>(x.sel.sel_mask), static_cast<void*>(x.sel.sel_prefix)})
    HIP_OK(hipFree(p));
}

static const zf_adam_hparams kHp{1e-3, 0.9, 0.999, 1e-8, 0.0};

// scores, selection, step 1 (INIT), step 2 (hand-over) with the single calls
static void run_single(Mat& x, hipStream_t s) {
  const size_t wsb = zf_colnorm_workspace_bytes(x.n, x.m, x.layout);
  void* dws = nullptr;
  if (wsb) HIP_OK(hipMalloc(&dws, wsb));
  ZF_OK_(zf_colnorm(x.G1, x.n, x.m, x.ld_g(), x.layout, x.norms, dws, wsb, s));
  int64_t k = -1;
  ZF_OK_(zf_topk_select(x.norms, x.m, double(x.k) / double(x.m), &x.sel, &k, s));
  CHECK(k == x.k);
  ZF_OK_(zf_update_fused(x.G1, x.n, x.m, x.ld_g(), x.layout, &x.sel, x.k, x.P, x.M, x.V,
                         x.ld_s(), x.W, x.ld_g(), &kHp, 1, ZF_STATES_INIT, nullptr, x.A,
                         x.ld_a(), 1, 2, s));
  ZF_OK_(zf_update_fused_handover(x.G2, x.n, x.m, x.ld_g(), x.layout, &x.sel, x.k, x.P, x.M,
                                  x.V, x.ld_s(), x.W, x.ld_g(), &kHp, 2, ZF_STATES_INPLACE,
                                  nullptr, x.A, x.ld_a(), 2, 2, 0.5f, x.D, x.ld_g(), s));
  HIP_OK(hipStreamSynchronize(s));
  if (dws) HIP_OK(hipFree(dws));
}

static void check(const Mat& x) {
  const auto norms = down(x.norms, x.m);
  const auto sel = down(x.sel.sel_idx, x.k);
  const auto unsel = down(x.sel.unsel_idx, x.m - x.k);
  const int64_t words = (x.m + 63) / 64;
  const auto mask = down(x.sel.sel_mask, words);
  const auto prefix = down(x.sel.sel_prefix, words);
  // scores
  for (int64_t j = 0; j < x.m; ++j) {
    double s = 0.0;
    for (int64_t i = 0; i < x.n; ++i) {
      const double g = widen(x.g1[x.at(i, j)]);
      s += g * g;
    }
    CHECK(std::fabs(norms[j] - s) <= 1e-5 * s);
  }
  // selection
  std::vector<int> seen(x.m, 0);
  for (int64_t r = 0; r < x.k; ++r) {
    CHECK(sel[r] >= 0 && sel[r] < x.m);
    if (r) CHECK(sel[r] > sel[r - 1]);
    if (sel[r] >= 0 && sel[r] < x.m) seen[sel[r]] += 1;
  }
  for (int64_t u = 0; u < x.m - x.k; ++u) {
    CHECK(unsel[u] >= 0 && unsel[u] < x.m);
    if (u) CHECK(unsel[u] > unsel[u - 1]);
    if (unsel[u] >= 0 && unsel[u] < x.m) seen[unsel[u]] += 2;
  }
  for (int64_t j = 0; j < x.m; ++j) CHECK(seen[j] == 1 || seen[j] == 2);
  float min_sel = INFINITY, max_unsel = -INFINITY;
  for (auto j : sel) min_sel = std::min(min_sel, norms[j]);
  for (auto j : unsel) max_unsel = std::max(max_unsel, norms[j]);
  if (x.k && x.k < x.m) CHECK(min_sel >= max_unsel);
  int32_t count = 0;
  for (int64_t w = 0; w < words; ++w) {
    CHECK(prefix[w] == count);
    count += __builtin_popcountll(mask[w]);
  }
  CHECK(count == x.k);
  for (auto j : sel) CHECK((mask[j >> 6] >> (j & 63)) & 1ull);
  // hand-over and packed buffer
  const auto D = down(x.D, x.n * x.m);
  const auto A = down(x.A, x.n * (x.m - x.k));
  for (int64_t i = 0; i < x.n; ++i) {
    for (auto j : sel) {
      const float d = D[x.at(i, j)];
      CHECK(d == 0.0f && !std::signbit(d));
    }
    for (int64_t u = 0; u < x.m - x.k; ++u) {
      const int64_t j = unsel[u];
      const float g1 = widen(x.g1[x.at(i, j)]), g2 = widen(x.g2[x.at(i, j)]);
      const float want = (g1 + g2) * 0.5f;
      CHECK(std::memcmp(&D[x.at(i, j)], &want, 4) == 0);
      const size_t ai = x.layout == ZF_LAYOUT_ROW_MAJOR ? size_t(i * (x.m - x.k) + u)
                                                        : size_t(u * x.n + i);
      CHECK(std::memcmp(&A[ai], &g1, 4) == 0);  // only read by the hand-over step
    }
  }
}

int main() {
  int ndev = 0;
  HIP_OK(hipGetDeviceCount(&ndev));
  if (ndev < 1) {
    std::fprintf(stderr, "no GPU\n");
    return 2;
  }
  hipStream_t s;
  HIP_OK(hipStreamCreate(&s));
  for (int32_t layout : {ZF_LAYOUT_ROW_MAJOR, ZF_LAYOUT_CHANNEL_MAJOR}) {
    // single calls on two matrices, then the same work as one plan
    Mat a = make(264, 300, 0.1, layout, 11), b = make(43, 77, 0.2, layout, 12);
    run_single(a, s);
    run_single(b, s);
    check(a);
    check(b);
    const auto Da = down(a.D, a.n * a.m), Db = down(b.D, b.n * b.m);
    const auto Wa = down(a.W, a.n * a.m), Wb = down(b.W, b.n * b.m);
    Mat pa = make(264, 300, 0.1, layout, 11), pb = make(43, 77, 0.2, layout, 12);
    zf_matrix desc[2];
    std::memset(desc, 0, sizeof(desc));
    Mat* ms[2] = {&pa, &pb};
    for (int q = 0; q < 2; ++q) {
      Mat& x = *ms[q];
      zf_matrix& d = desc[q];
      d.n = x.n;
      d.m = x.m;
      d.k = x.k;
      d.layout = layout;
      d.grad = x.G1;
      d.ld_grad = x.ld_g();
      d.weight = x.W;
      d.ld_weight = x.ld_g();
      d.master = x.P;
      d.exp_avg = x.M;
      d.exp_avg_sq = x.V;
      d.ld_state = x.ld_s();
      d.acc = x.A;
      d.ld_acc = x.ld_a();
      d.norms_sq = x.norms;
      d.sel = x.sel;
      d.unpacked = x.D;
      d.ld_unpacked = x.ld_g();
    }
    // the plans' tables and workspaces in memory this program allocates
    size_t bytes1 = 0, bytes2 = 0;
    ZF_OK_(zf_plan_query(desc, 2, &bytes1));
    void* mem1 = nullptr;
    HIP_OK(hipMalloc(&mem1, bytes1));
    zf_plan* plan1 = nullptr;
    ZF_OK_(zf_plan_create(desc, 2, mem1, bytes1, s, &plan1));
    CHECK(zf_plan_device_bytes(plan1) == bytes1);
    desc[0].grad = pa.G2;
    desc[1].grad = pb.G2;
    ZF_OK_(zf_plan_query(desc, 2, &bytes2));
    void* mem2 = nullptr;
    HIP_OK(hipMalloc(&mem2, bytes2));
    zf_plan* plan2 = nullptr;
    ZF_OK_(zf_plan_create(desc, 2, mem2, bytes2, s, &plan2));
    ZF_OK_(zf_plan_colnorm(plan1, s));
    ZF_OK_(zf_plan_topk_select(plan1, s));
    ZF_OK_(zf_plan_update(plan1, &kHp, 1, ZF_STATES_INIT, 1, 2, 1, 1, s));
    ZF_OK_(zf_plan_update_handover(plan2, &kHp, 2, ZF_STATES_INPLACE, 2, 2, 0.5f, s));
    HIP_OK(hipStreamSynchronize(s));
    CHECK(same_bits(down(pa.D, pa.n * pa.m), Da) && same_bits(down(pb.D, pb.n * pb.m), Db));
    CHECK(same_bits(down(pa.W, pa.n * pa.m), Wa) && same_bits(down(pb.W, pb.n * pb.m), Wb));
    zf_plan_destroy(plan1);
    zf_plan_destroy(plan2);
    HIP_OK(hipFree(mem1));  // the stream was synchronised above
    HIP_OK(hipFree(mem2));
    // deferred packing: no packed buffer; step 1 runs Adam alone, step 2
    // sums both steps' gradients into the hand-over -- the same bits
    Mat da = make(264, 300, 0.1, layout, 11), db = make(43, 77, 0.2, layout, 12);
    Mat* dm[2] = {&da, &db};
    for (int q = 0; q < 2; ++q) {
      desc[q].grad = dm[q]->G1;
      desc[q].weight = dm[q]->W;
      desc[q].master = dm[q]->P;
      desc[q].exp_avg = dm[q]->M;
      desc[q].exp_avg_sq = dm[q]->V;
      desc[q].acc = nullptr;
      desc[q].ld_acc = 0;
      desc[q].norms_sq = dm[q]->norms;
      desc[q].sel = dm[q]->sel;
      desc[q].unpacked = dm[q]->D;
    }
    size_t bytes3 = 0, bytes4 = 0;
    ZF_OK_(zf_plan_query(desc, 2, &bytes3));
    void* mem3 = nullptr;
    HIP_OK(hipMalloc(&mem3, bytes3));
    zf_plan* plan3 = nullptr;
    ZF_OK_(zf_plan_create(desc, 2, mem3, bytes3, s, &plan3));
    desc[0].grad = da.G2;
    desc[1].grad = db.G2;
    ZF_OK_(zf_plan_query(desc, 2, &bytes4));
    void* mem4 = nullptr;
    HIP_OK(hipMalloc(&mem4, bytes4));
    zf_plan* plan4 = nullptr;
    ZF_OK_(zf_plan_create(desc, 2, mem4, bytes4, s, &plan4));
    ZF_OK_(zf_plan_colnorm(plan3, s));
    ZF_OK_(zf_plan_topk_select(plan3, s));
    ZF_OK_(zf_plan_update(plan3, &kHp, 1, ZF_STATES_INIT, 1, 2, 1, 0, s));
    // packing every step needs the packed buffer these plans do not have
    CHECK(zf_plan_update(plan3, &kHp, 1, ZF_STATES_INPLACE, 2, 2, 1, 1, s) == ZF_EINVAL);
    const zf_plan* earlier[1] = {plan3};
    ZF_OK_(zf_plan_update_handover_deferred(plan4, &kHp, 2, earlier, 1, 0.5f, s));
    HIP_OK(hipStreamSynchronize(s));
    CHECK(same_bits(down(da.D, da.n * da.m), Da) && same_bits(down(db.D, db.n * db.m), Db));
    CHECK(same_bits(down(da.W, da.n * da.m), Wa) && same_bits(down(db.W, db.n * db.m), Wb));
    zf_plan_destroy(plan3);
    zf_plan_destroy(plan4);
    HIP_OK(hipFree(mem3));
    HIP_OK(hipFree(mem4));
    if (layout == ZF_LAYOUT_CHANNEL_MAJOR) {
      // Zen-auto on the device with deferred packing: step 1 refreshes (no
      // end: tau = inf never triggers), step 2 ends the interval by force
      // with the hand-over fused -- again the single calls' bits; the gated
      // hand-over then writes nothing
      Mat za = make(264, 300, 0.1, layout, 11), zb = make(43, 77, 0.2, layout, 12);
      Mat* zm[2] = {&za, &zb};
      std::vector<float*> stats;
      for (int q = 0; q < 2; ++q) {
        desc[q].grad = zm[q]->G1;
        desc[q].weight = zm[q]->W;
        desc[q].master = zm[q]->P;
        desc[q].exp_avg = zm[q]->M;
        desc[q].exp_avg_sq = zm[q]->V;
        desc[q].norms_sq = zm[q]->norms;
        desc[q].sel = zm[q]->sel;
        desc[q].unpacked = zm[q]->D;
        desc[q].sel_sq = dev_alloc<float>(zm[q]->k);
        desc[q].acc_sq = dev_alloc<float>(zm[q]->m - zm[q]->k);
        stats.push_back(desc[q].sel_sq);
        stats.push_back(desc[q].acc_sq);
      }
      size_t bytes5 = 0, bytes6 = 0;
      ZF_OK_(zf_plan_query(desc, 2, &bytes5));
      void* mem5 = nullptr;
      HIP_OK(hipMalloc(&mem5, bytes5));
      zf_plan* plan5 = nullptr;
      ZF_OK_(zf_plan_create(desc, 2, mem5, bytes5, s, &plan5));
      desc[0].grad = za.G2;
      desc[1].grad = zb.G2;
      ZF_OK_(zf_plan_query(desc, 2, &bytes6));
      void* mem6 = nullptr;
      HIP_OK(hipMalloc(&mem6, bytes6));
      zf_plan* plan6 = nullptr;
      ZF_OK_(zf_plan_create(desc, 2, mem6, bytes6, s, &plan6));
      zf_zen_totals* tot = dev_alloc<zf_zen_totals>(1);
      zf_zen_state* st = dev_alloc<zf_zen_state>(1);
      const zf_zen_state st0{0, 1};
      HIP_OK(hipMemcpy(st, &st0, sizeof st0, hipMemcpyHostToDevice));
      const double inf = std::numeric_limits<double>::infinity();
      ZF_OK_(zf_plan_colnorm(plan5, s));
      ZF_OK_(zf_plan_topk_select(plan5, s));
      ZF_OK_(zf_plan_update_zen_deferred(plan5, &kHp, 1, ZF_STATES_INIT, 4, nullptr, 0, 0, inf,
                                         tot, st, s));
      ZF_OK_(zf_plan_handover_zen_deferred(plan5, nullptr, 0, st, s));
      const zf_plan* zearlier[1] = {plan5};
      ZF_OK_(zf_plan_update_zen_deferred(plan6, &kHp, 2, ZF_STATES_INPLACE, 4, zearlier, 1, 2,
                                         inf, tot, st, s));
      ZF_OK_(zf_plan_handover_zen_deferred(plan6, zearlier, 1, st, s));
      HIP_OK(hipStreamSynchronize(s));
      zf_zen_state st2{};
      HIP_OK(hipMemcpy(&st2, st, sizeof st2, hipMemcpyDeviceToHost));
      CHECK(st2.length == 2 && st2.ended == 2);
      CHECK(same_bits(down(za.D, za.n * za.m), Da) && same_bits(down(zb.D, zb.n * zb.m), Db));
      CHECK(same_bits(down(za.W, za.n * za.m), Wa) && same_bits(down(zb.W, zb.n * zb.m), Wb));
      zf_plan_destroy(plan5);
      zf_plan_destroy(plan6);
      HIP_OK(hipFree(mem5));
      HIP_OK(hipFree(mem6));
      HIP_OK(hipFree(tot));
      HIP_OK(hipFree(st));
      for (float* p : stats) HIP_OK(hipFree(p));
      for (int q = 0; q < 2; ++q) desc[q].sel_sq = desc[q].acc_sq = nullptr;
      release(za);
      release(zb);
    }
    for (Mat* x : {&a, &b, &pa, &pb, &da, &db}) release(*x);
  }
  HIP_OK(hipStreamDestroy(s));
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("abi smoke ok: both layouts, single calls, plans, deferred packing, "
              "Zen-auto with deferred packing\n");
  return 0;
}
