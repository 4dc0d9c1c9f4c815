// Host (CPU) side of libzf: the deferred update of the unselected columns.
//
// ZenFlow applies the accumulated unimportant gradients with an optimizer
// that runs on the host over the offloaded optimizer states (Asynchronous
// Offloading Workflow; Implementation, "Concurrent CPU-side Optimizer"): at
// the end of an accumulation interval, every unselected column j = unsel[u]
// takes one Adam/AdamW step with the interval's mean gradient
//   g = A[i][u] * scale            (scale = 1/S: the mean of the S-step rule
//                                   of the Convergence Analysis)
// on its (p, m, v) in the host-resident full-state store, and its new bf16
// weights are produced for the device (zf_scatter_weights writes them into
// W).  The element sequence is the selective optimizer's, one IEEE fp32
// operation per line (the library is compiled without contraction or fast
// math), so the host and the device updates agree bit for bit.
//
// Work is split over threads by whole columns (channel-major: a column is
// one contiguous row of every buffer) or by rows (row-major); unsel must be
// strictly ascending, so no two threads write the same element.  In the
// row-major layout a row's unselected columns come in runs of consecutive
// indices (the same runs in every row): each run is one contiguous stretch of
// the states and of the accumulated row, updated by the same element loop.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "zf.h"
#include "zf_internal.hpp"

namespace {

inline uint16_t host_round_bf16(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// One element: the same operations, in the same order, as the device's
// selective Adam step.
inline void host_adam_elem(float g, float& p, float& m, float& v, const zf::AdamK& c) {
  m = c.b1 * m + c.c1 * g;
  v = c.b2 * v + c.c2 * (g * g);
  const float den = std::sqrt(v * c.ib2) + c.eps;
  const float u = (m * c.ib1) / den;
  if (c.wd != 0.0f) p = p - c.wd * p;
  p = p - c.lr * u;
}

// A contiguous run of `len` elements: gradient a * scale, states p/m/v,
// bf16 output w.  Written as independent element loops so that the
// compiler vectorises them (every vector lane is the same IEEE operation).
void host_adam_run(const float* __restrict__ a, float scale, float* __restrict__ p,
                   float* __restrict__ m, float* __restrict__ v, uint16_t* __restrict__ w,
                   int64_t len, const zf::AdamK& c) {
  for (int64_t e = 0; e < len; ++e) {
    const float g = a[e] * scale;
    float pe = p[e], me = m[e], ve = v[e];
    host_adam_elem(g, pe, me, ve, c);
    p[e] = pe;
    m[e] = me;
    v[e] = ve;
    w[e] = host_round_bf16(pe);
  }
}

struct HostSpan {
  uintptr_t lo = 0, hi = 0;
};

HostSpan host_span(const void* p, int64_t rows, int64_t width, int64_t ld, size_t elem) {
  HostSpan s;
  if (p == nullptr || rows <= 0 || width <= 0) return s;
  s.lo = reinterpret_cast<uintptr_t>(p);
  s.hi = s.lo + static_cast<uintptr_t>((rows - 1) * ld + width) * elem;
  return s;
}

bool host_overlap(const HostSpan& a, const HostSpan& b) {
  return a.hi > a.lo && b.hi > b.lo && a.lo < b.hi && b.lo < a.hi;
}

bool host_mat_ok(const void* p, int64_t rows, int64_t width, int64_t ld, size_t elem) {
  if (rows < 0 || width < 0 || ld < width) return false;
  if (rows == 0 || width == 0) return true;
  return p != nullptr && reinterpret_cast<uintptr_t>(p) % elem == 0;
}

}  // namespace

extern "C" {

zf_status zf_host_adam_unselected(const float* acc, int64_t ld_acc, const int32_t* unsel_idx,
                                  int64_t n, int64_t m, int64_t k, int32_t layout, float scale,
                                  float* master, float* exp_avg, float* exp_avg_sq,
                                  int64_t ld_state, uint16_t* weight_cols, int64_t ld_wcols,
                                  const zf_adam_hparams* hp, int64_t step, int32_t nthreads) {
  if (layout != ZF_LAYOUT_ROW_MAJOR && layout != ZF_LAYOUT_CHANNEL_MAJOR) return ZF_EINVAL;
  if (n < 0 || m < 0 || k < 0 || k > m || n >= (int64_t(1) << 30) || m >= (int64_t(1) << 30))
    return ZF_EINVAL;
  if (!zf::hparams_ok(hp) || step < 1 || !std::isfinite(scale) || nthreads < 0) return ZF_EINVAL;
  const int64_t u = m - k;
  const bool cm = layout == ZF_LAYOUT_CHANNEL_MAJOR;
  // storage extents: (rows, width) of A / weight_cols (n x u) and the states (n x m)
  const int64_t ar = cm ? u : n, aw = cm ? n : u;
  const int64_t sr = cm ? m : n, sw = cm ? n : m;
  if (!host_mat_ok(acc, ar, aw, ld_acc, 4) || !host_mat_ok(weight_cols, ar, aw, ld_wcols, 2) ||
      !host_mat_ok(master, sr, sw, ld_state, 4) || !host_mat_ok(exp_avg, sr, sw, ld_state, 4) ||
      !host_mat_ok(exp_avg_sq, sr, sw, ld_state, 4))
    return ZF_EINVAL;
  if (n == 0 || u == 0) return ZF_OK;  // nothing to update
  if (unsel_idx == nullptr) return ZF_EINVAL;
  for (int64_t q = 0; q < u; ++q) {
    const int32_t j = unsel_idx[q];
    if (j < 0 || j >= m || (q > 0 && j <= unsel_idx[q - 1])) return ZF_EINVAL;
  }
  const HostSpan spans[5] = {host_span(acc, ar, aw, ld_acc, 4),
                             host_span(weight_cols, ar, aw, ld_wcols, 2),
                             host_span(master, sr, sw, ld_state, 4),
                             host_span(exp_avg, sr, sw, ld_state, 4),
                             host_span(exp_avg_sq, sr, sw, ld_state, 4)};
  for (int a = 0; a < 5; ++a)
    for (int b = a + 1; b < 5; ++b)
      if (host_overlap(spans[a], spans[b])) return ZF_EINVAL;

  const zf::AdamK c = zf::adam_consts(*hp, step);
  const int64_t units = cm ? u : n;  // columns (channel-major) or rows
  // row-major: runs (first slot, first column, length) of consecutive columns
  struct Run {
    int64_t q, j, len;
  };
  std::vector<Run> runs;
  if (!cm) {
    for (int64_t q = 0; q < u;) {
      int64_t e = q + 1;
      while (e < u && unsel_idx[e] == unsel_idx[e - 1] + 1) ++e;
      runs.push_back(Run{q, unsel_idx[q], e - q});
      q = e;
    }
  }
  int64_t threads = nthreads > 0 ? nthreads : std::max<int64_t>(1, std::thread::hardware_concurrency());
  threads = std::max<int64_t>(1, std::min<int64_t>(threads, units));

  auto work = [&](int64_t t0, int64_t t1) {
    if (cm) {
      for (int64_t q = t0; q < t1; ++q) {
        const int64_t j = unsel_idx[q];
        host_adam_run(acc + q * ld_acc, scale, master + j * ld_state, exp_avg + j * ld_state,
                      exp_avg_sq + j * ld_state, weight_cols + q * ld_wcols, n, c);
      }
    } else {
      for (int64_t i = t0; i < t1; ++i) {
        const float* a = acc + i * ld_acc;
        float* p = master + i * ld_state;
        float* mm = exp_avg + i * ld_state;
        float* vv = exp_avg_sq + i * ld_state;
        uint16_t* w = weight_cols + i * ld_wcols;
        for (const Run& r : runs)
          host_adam_run(a + r.q, scale, p + r.j, mm + r.j, vv + r.j, w + r.q, r.len, c);
      }
    }
  };
  if (threads == 1) {
    work(0, units);
    return ZF_OK;
  }
  std::vector<std::thread> pool;
  pool.reserve(static_cast<size_t>(threads - 1));
  const int64_t per = units / threads, extra = units % threads;
  int64_t start = 0;
  int64_t first_end = 0;
  for (int64_t t = 0; t < threads; ++t) {
    const int64_t end = start + per + (t < extra ? 1 : 0);
    if (t == 0) {
      first_end = end;
    } else {
      try {
        pool.emplace_back(work, start, end);
      } catch (...) {
        work(start, end);  // no thread available: run this share here
      }
    }
    start = end;
  }
  work(0, first_end);
  for (auto& th : pool) th.join();
  return ZF_OK;
}

}  // extern "C"
