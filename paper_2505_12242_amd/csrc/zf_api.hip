// Host entry points of libzf: argument validation, launch geometry, Adam
// constants and the batched plan.  Every check runs before the first HIP
// call, so invalid arguments enqueue nothing (and never touch a device).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "zf.h"
#include "zf_internal.hpp"
#include "zf_measure.h"

namespace zf {

bool hparams_ok(const zf_adam_hparams* hp) {
  if (hp == nullptr) return false;
  const auto fin = [](double x) { return std::isfinite(x); };
  return fin(hp->lr) && hp->lr >= 0.0 && fin(hp->eps) && hp->eps >= 0.0 && fin(hp->beta1) &&
         hp->beta1 >= 0.0 && hp->beta1 < 1.0 && fin(hp->beta2) && hp->beta2 >= 0.0 &&
         hp->beta2 < 1.0 && fin(hp->weight_decay) && hp->weight_decay >= 0.0;
}

AdamK adam_consts(const zf_adam_hparams& hp, int64_t step) {
  const double t = static_cast<double>(step);
  AdamK c;
  c.b1 = static_cast<float>(hp.beta1);
  c.b2 = static_cast<float>(hp.beta2);
  c.c1 = static_cast<float>(1.0 - hp.beta1);
  c.c2 = static_cast<float>(1.0 - hp.beta2);
  c.lr = static_cast<float>(hp.lr);
  c.eps = static_cast<float>(hp.eps);
  c.wd = static_cast<float>(hp.lr * hp.weight_decay);
  c.ib1 = static_cast<float>(1.0 / (1.0 - std::pow(hp.beta1, t)));
  c.ib2 = static_cast<float>(1.0 / (1.0 - std::pow(hp.beta2, t)));
  return c;
}

}  // namespace zf

using zf::adam_consts;
using zf::hparams_ok;
using zf::AdamK;
using zf::DevMat;
using zf::Table;

namespace {

thread_local int g_last_hip_error = 0;

zf_status hip_fail(hipError_t e) {
  g_last_hip_error = static_cast<int>(e);
  return ZF_EHIP;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// A row-major [rows][ld] buffer of `width` used elements per row must have
// ld >= width, be present when it holds data, and be element-aligned.
bool matrix_ok(const void* p, int64_t rows, int64_t width, int64_t ld, size_t elem) {
  if (rows < 0 || width < 0 || ld < width) return false;
  if (rows == 0 || width == 0) return true;
  return p != nullptr && aligned(p, elem);
}

bool vector_ok(const void* p, int64_t count, size_t elem) {
  if (count < 0) return false;
  if (count == 0) return true;
  return p != nullptr && aligned(p, elem);
}

struct Span {
  uintptr_t lo = 0, hi = 0;
};

Span span_of(const void* p, int64_t rows, int64_t width, int64_t ld, size_t elem) {
  Span s;
  if (p == nullptr || rows <= 0 || width <= 0) return s;
  s.lo = reinterpret_cast<uintptr_t>(p);
  s.hi = s.lo + static_cast<uintptr_t>(((rows - 1) * ld + width)) * elem;
  return s;
}

bool overlaps(const Span& a, const Span& b) {
  return a.hi > a.lo && b.hi > b.lo && a.lo < b.hi && b.lo < a.hi;
}

// ---- geometry -------------------------------------------------------------

constexpr int64_t kMinBlocks = 2048;          // enough blocks to fill 256 CUs
constexpr int64_t kMaxBlocks = int64_t(1) << 23;  // grid x block stays < 2^32

int64_t colnorm_blocks(int64_t n, int64_t m, int rpb) {
  if (n <= 0 || m <= 0) return 0;
  return ceil_div(m, zf::kColnormCols) * ceil_div(n, rpb);
}

int64_t update_blocks(int64_t n, int64_t m, int rows) {
  if (n <= 0 || m <= 0) return 0;
  return ceil_div(m, zf::kUpdateCols) * ceil_div(n, rows);
}

// Rows per colnorm block: 256 (partials cost 8 B per column per 256 rows,
// ~1.6% of G), halved down to 16 while the whole grid is too small.
int pick_colnorm_rows(const std::vector<std::pair<int64_t, int64_t>>& shapes) {
  int rpb = 256;
  for (;;) {
    int64_t total = 0;
    for (auto& s : shapes) total += colnorm_blocks(s.first, s.second, rpb);
    if (total >= kMinBlocks || rpb <= 16) return rpb;
    rpb >>= 1;
  }
}

#ifndef ZF_UPDATE_ROWS
#define ZF_UPDATE_ROWS 8
#endif

int pick_update_rows(const std::vector<std::pair<int64_t, int64_t>>& shapes) {
  int rows = ZF_UPDATE_ROWS;
  for (;;) {
    int64_t total = 0;
    for (auto& s : shapes) total += update_blocks(s.first, s.second, rows);
    if (total > kMaxBlocks && rows < (1 << 20)) {
      rows <<= 1;
      continue;
    }
    if (total >= kMinBlocks || rows <= 4) return rows;
    rows >>= 1;
  }
}

// Row-major update with 16-byte accesses: equal-width column tiles of at
// most kRvMaxCols columns (multiples of 8, so that 16-byte G loads and
// hand-over stores stay aligned) and rv_rows rows per block.
#ifndef ZF_RV_ROWS
#define ZF_RV_ROWS 16
#endif
#ifndef ZF_RV_ENABLE
#define ZF_RV_ENABLE 1
#endif

int32_t rv_width(int64_t m) {
  const int64_t tiles = std::max<int64_t>(1, ceil_div(m, zf::kRvMaxCols));
  return static_cast<int32_t>(8 * ceil_div(std::max<int64_t>(m, 1), 8 * tiles));
}

int64_t rv_blocks(int64_t n, int64_t m, int rows) {
  if (n <= 0 || m <= 0) return 0;
  return ceil_div(m, rv_width(m)) * ceil_div(n, rows);
}

int pick_rv_rows(const std::vector<std::pair<int64_t, int64_t>>& shapes) {
  int rows = ZF_RV_ROWS;
  for (;;) {
    int64_t total = 0;
    for (auto& s : shapes) total += rv_blocks(s.first, s.second, rows);
    if (total > kMaxBlocks && rows < (1 << 20)) {
      rows <<= 1;
      continue;
    }
    if (total >= kMinBlocks || rows <= 4) return rows;
    rows >>= 1;
  }
}

void set_geometry(DevMat& d, int cn_rows, int up_rows) {
  d.cn_rpb = cn_rows;
  d.cn_cb = static_cast<int32_t>(ceil_div(d.m, zf::kColnormCols));
  d.cn_rb = d.n > 0 ? static_cast<int32_t>(ceil_div(d.n, cn_rows)) : 0;
  d.up_rows = up_rows;
  d.up_cb = static_cast<int32_t>(ceil_div(d.m, zf::kUpdateCols));
  d.up_rb = d.n > 0 ? static_cast<int32_t>(ceil_div(d.n, up_rows)) : 0;
  d.vec = (d.grad != nullptr && aligned(d.grad, 16) && d.ld_grad % 8 == 0) ? 1 : 0;
}

DevMat blank() {
  DevMat d;
  std::memset(&d, 0, sizeof(d));
  return d;
}

Table single_table() { return Table{nullptr, nullptr, 1}; }

hipStream_t as_stream(zf_stream s) { return reinterpret_cast<hipStream_t>(s); }

// ---- per-matrix validation -------------------------------------------------

// Storage extent of a logical [rows_l][cols_l] matrix: row-major keeps
// [rows_l][ld], channel-major stores the transpose [cols_l][ld].
struct Ext {
  int64_t rows, width;
};

Ext ext(int32_t layout, int64_t rows_l, int64_t cols_l) {
  return layout == zf::kChannelMajor ? Ext{cols_l, rows_l} : Ext{rows_l, cols_l};
}

bool mat_ok(const void* p, Ext e, int64_t ld, size_t elem) {
  return matrix_ok(p, e.rows, e.width, ld, elem);
}

Span span(const void* p, Ext e, int64_t ld, size_t elem) {
  return span_of(p, e.rows, e.width, ld, elem);
}

bool layout_ok(int32_t layout) {
  return layout == zf::kRowMajor || layout == zf::kChannelMajor;
}

bool selection_ok(const zf_selection* s, int64_t m, int64_t k, bool need_idx) {
  if (s == nullptr) return false;
  const int64_t words = ceil_div(m, 64);
  if (!vector_ok(s->sel_mask, words, 8) || !vector_ok(s->sel_prefix, words, 4)) return false;
  if (need_idx && (!vector_ok(s->sel_idx, k, 4) || !vector_ok(s->unsel_idx, m - k, 4)))
    return false;
  return true;
}

bool shape_ok(int64_t n, int64_t m, int64_t k) {
  return n >= 0 && m >= 0 && k >= 0 && k <= m && n < (int64_t(1) << 30) &&
         m < (int64_t(1) << 30);
}

// Buffers that the kernels may find in pinned host memory (the full-state
// store, the host-produced weight columns) must be device memory or host
// memory mapped at the same address for the device; anything else (pageable
// host memory, an address HIP does not know) is rejected before it can reach
// a kernel.  Queries the runtime; enqueues nothing.
bool device_accessible(const void* p) {
  if (p == nullptr) return true;
  hipPointerAttribute_t a;
  std::memset(&a, 0, sizeof(a));
  const hipError_t e = hipPointerGetAttributes(&a, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // leave no sticky error behind
    return false;
  }
  if (a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged) return true;
  // pinned host memory: usable in place when the device maps it at the host
  // address (both pointers refer to the same spot of the allocation)
  if (a.type == hipMemoryTypeHost) return a.devicePointer != nullptr && a.devicePointer == a.hostPointer;
  return false;
}

bool store_accessible(const DevMat& d) {
  return device_accessible(d.st_P) && device_accessible(d.st_M) && device_accessible(d.st_V);
}

// Checks of one Adam step's buffers (selection mask/prefix already checked).
bool adam_args_ok(const DevMat& d, int32_t mode, Span g) {
  const int64_t n = d.n, m = d.m, k = d.k;
  const int32_t L = d.layout;
  if (!mat_ok(d.P, ext(L, n, k), d.ld_state, 4) || !mat_ok(d.M, ext(L, n, k), d.ld_state, 4) ||
      !mat_ok(d.V, ext(L, n, k), d.ld_state, 4) ||
      !mat_ok(d.weight, ext(L, n, m), d.ld_weight, 2))
    return false;
  if (mode != zf::kInplace && mode != zf::kRemap && mode != zf::kInit) return false;
  if (mode == zf::kRemap) {
    const int64_t words = ceil_div(m, 64);
    if (!vector_ok(d.prev_mask, words, 8) || !vector_ok(d.prev_prefix, words, 4)) return false;
    // The previous states hold as many slots as the previous selection has
    // columns (device data); only presence, alignment and stride are checked.
    // They are read for the selected columns and, with a store, for the
    // columns that leave the selection (swap-out), whatever k is.
    if (n > 0 && (k > 0 || d.st_P != nullptr) &&
        (d.prev_P == nullptr || d.prev_M == nullptr || d.prev_V == nullptr ||
         !aligned(d.prev_P, 4) || !aligned(d.prev_M, 4) || !aligned(d.prev_V, 4) ||
         d.ld_prev < (L == zf::kChannelMajor ? n : 0)))
      return false;
  }
  if (mode != zf::kInplace && d.init_P != nullptr &&
      !mat_ok(d.init_P, ext(L, n, m), d.ld_init, 4))
    return false;
  const bool store = mode != zf::kInplace && d.st_P != nullptr;
  if (store && (!store_accessible(d) || !mat_ok(d.st_P, ext(L, n, m), d.ld_store, 4) ||
                !mat_ok(d.st_M, ext(L, n, m), d.ld_store, 4) ||
                !mat_ok(d.st_V, ext(L, n, m), d.ld_store, 4) ||
                (n > 0 && m > 0 && (d.st_M == nullptr || d.st_V == nullptr))))
    return false;
  const Span outs[7] = {span(d.P, ext(L, n, k), d.ld_state, 4),
                        span(d.M, ext(L, n, k), d.ld_state, 4),
                        span(d.V, ext(L, n, k), d.ld_state, 4),
                        span(d.weight, ext(L, n, m), d.ld_weight, 2),
                        store ? span(d.st_P, ext(L, n, m), d.ld_store, 4) : Span{},
                        store ? span(d.st_M, ext(L, n, m), d.ld_store, 4) : Span{},
                        store ? span(d.st_V, ext(L, n, m), d.ld_store, 4) : Span{}};
  for (int a = 0; a < 7; ++a) {
    if (overlaps(outs[a], g)) return false;
    for (int b = a + 1; b < 7; ++b)
      if (overlaps(outs[a], outs[b])) return false;
  }
  return true;
}

// The full-state store (if any) against another buffer.
bool store_overlaps(const DevMat& d, Span other) {
  if (d.st_P == nullptr) return false;
  const Ext e = ext(d.layout, d.n, d.m);
  return overlaps(span(d.st_P, e, d.ld_store, 4), other) ||
         overlaps(span(d.st_M, e, d.ld_store, 4), other) ||
         overlaps(span(d.st_V, e, d.ld_store, 4), other);
}

bool pack_args_ok(const DevMat& d, int64_t sii, int64_t S, Span g) {
  if (S < 1 || sii < 1 || sii > S) return false;
  const Ext e = ext(d.layout, d.n, d.m - d.k);
  if (!mat_ok(d.acc, e, d.ld_acc, 4)) return false;
  return !overlaps(span(d.acc, e, d.ld_acc, 4), g);
}

DevMat base_mat(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad, int32_t layout,
                const zf_selection* sel, int64_t k) {
  DevMat d = blank();
  d.n = n;
  d.m = m;
  d.k = k;
  d.grad = grad;
  d.ld_grad = ld_grad;
  d.layout = layout;
  if (sel != nullptr) {
    d.sel_idx = sel->sel_idx;
    d.unsel_idx = sel->unsel_idx;
    d.mask = sel->sel_mask;
    d.prefix = sel->sel_prefix;
  }
  return d;
}

void apply_source(DevMat& d, const zf_state_source* src) {
  if (src == nullptr) return;
  d.prev_mask = src->prev_mask;
  d.prev_prefix = src->prev_prefix;
  d.prev_P = src->prev_master;
  d.prev_M = src->prev_exp_avg;
  d.prev_V = src->prev_exp_avg_sq;
  d.ld_prev = src->ld_prev;
  d.init_P = src->init_master;
  d.ld_init = src->ld_init;
  d.st_P = src->store_master;
  d.st_M = src->store_exp_avg;
  d.st_V = src->store_exp_avg_sq;
  d.ld_store = src->ld_store;
  d.pend_acc = src->pend_acc;
  d.ld_pend = src->ld_pend;
}

// Channel-major vector path: n a multiple of 8 and every present row start
// 16-byte aligned.
bool cm_vec_ok(const DevMat& d) {
  if (d.n % 8 != 0) return false;
  const auto ok = [](const void* p, int64_t ld, int64_t per16) {
    return p == nullptr || (aligned(p, 16) && ld % per16 == 0);
  };
  return ok(d.grad, d.ld_grad, 8) && ok(d.weight, d.ld_weight, 8) && ok(d.P, d.ld_state, 4) &&
         ok(d.M, d.ld_state, 4) && ok(d.V, d.ld_state, 4) && ok(d.acc, d.ld_acc, 4) &&
         ok(d.out, d.ld_out, 4) && ok(d.prev_P, d.ld_prev, 4) && ok(d.prev_M, d.ld_prev, 4) &&
         ok(d.prev_V, d.ld_prev, 4) && ok(d.init_P, d.ld_init, 4) && ok(d.st_P, d.ld_store, 4) &&
         ok(d.st_M, d.ld_store, 4) && ok(d.st_V, d.ld_store, 4) && ok(d.pend_acc, d.ld_pend, 4) &&
         ok(d.acc1, d.ld_acc1, 8);
}

// Row-major 16-byte update: G rows 16-byte aligned (8 bf16), and every
// fp32 buffer moved in slot quads or column quads (A, P/M/V, the hand-over
// output) 16-byte aligned per row.  Other buffers are accessed by element.
bool rv_ok(const DevMat& d) {
  if (!ZF_RV_ENABLE || d.layout != zf::kRowMajor) return false;
  // (a single row never uses its stride)
  const bool one_row = d.n <= 1;
  const auto ok = [one_row](const void* p, int64_t ld, int64_t per16) {
    return p == nullptr || (aligned(p, 16) && (one_row || ld % per16 == 0));
  };
  return d.grad != nullptr && aligned(d.grad, 16) && (one_row || d.ld_grad % 8 == 0) &&
         ok(d.acc, d.ld_acc, 4) && ok(d.P, d.ld_state, 4) && ok(d.M, d.ld_state, 4) &&
         ok(d.V, d.ld_state, 4) && ok(d.out, d.ld_out, 4);
}

// Geometry of the row-major 16-byte update; used when `allow` (all matrices
// of a plan qualify) and this matrix qualifies.
// Row-major update/unpack blocks address `rows` rows through 32-bit buffer
// offsets: every row stride times the rows of a block must stay below 2^31
// bytes.
bool strides_fit(const DevMat& d, int64_t rows) {
  const int64_t lim = (int64_t(1) << 31) / std::max<int64_t>(rows, 1);
  return d.ld_grad * 2 < lim && d.ld_weight * 2 < lim && d.ld_state * 4 < lim &&
         d.ld_acc * 4 < lim && d.ld_out * 4 < lim && d.ld_prev * 4 < lim && d.ld_init * 4 < lim &&
         d.ld_store * 4 < lim;
}

bool rm_strides_ok(const DevMat& d) { return strides_fit(d, d.up_rows); }

void set_rv(DevMat& d, int rows, bool allow) {
  d.rv_w = rv_width(d.m);
  d.rv_cb = d.m > 0 ? static_cast<int32_t>(ceil_div(d.m, d.rv_w)) : 0;
  d.rv_rows = rows;
  d.rv = (allow && rv_ok(d) && strides_fit(d, rows)) ? 1 : 0;
}

void finish_geometry(DevMat& d, int cn_rows, int up_rows, bool zen = false) {
  set_geometry(d, cn_rows, up_rows);
  if (d.layout == zf::kChannelMajor) {
    // quads per thread in the full-grid passes: kCmQpt when it fills at
    // least as many lanes of the last chunk as kCmQpt / 2 does (fewer,
    // fuller blocks), else kCmQpt / 2; the selected-only Adam grid takes one
    // quad per thread.  Plans with the Zen-auto statistics take kCmQpt
    // whatever the fill: their updates ran faster with more bytes in flight
    // per lane than with fuller blocks (13B set: 10% shorter steps with
    // deferred packing, 6% packing every step; 5120-row channels then leave
    // 37% of the last chunk's lanes idle).
    const auto fill = [&](int v) {
      const int64_t chunk = static_cast<int64_t>(v) * zf::kThreads * 4;
      const int64_t nch = std::max<int64_t>(1, ceil_div(d.n, chunk));
      return static_cast<double>(d.n) / static_cast<double>(nch * chunk);
    };
    const int best = (zen || fill(zf::kCmQpt) >= fill(zf::kCmQpt / 2) - 1e-12) ? zf::kCmQpt
                                                                              : zf::kCmQpt / 2;
    d.cm_qpt = best;
    d.cm_nch = d.n > 0 ? static_cast<int32_t>(ceil_div(d.n, int64_t(best) * zf::kThreads * 4)) : 0;
    d.cm_snch = d.n > 0 ? static_cast<int32_t>(ceil_div(d.n, int64_t(zf::kCmSelChunk))) : 0;
    d.cm_unch = d.n > 0 ? static_cast<int32_t>(ceil_div(d.n, zf::kCmUnpackChunk)) : 0;
    d.vec = cm_vec_ok(d) ? 1 : 0;
    const auto al16 = [](const void* p, int64_t ld) {
      return p != nullptr && aligned(p, 16) && ld % 8 == 0;
    };
    d.scat_vec = (d.n % 8 == 0 && al16(d.wcols, d.ld_wcols) && al16(d.weight, d.ld_weight)) ? 1 : 0;
  }
}

int64_t colnorm_grid(const DevMat& d) {
  if (d.layout == zf::kChannelMajor) return ceil_div(d.m, zf::kCmColnormCols);
  return colnorm_blocks(d.n, d.m, d.cn_rpb);
}

int64_t update_grid(const DevMat& d) {
  if (d.layout == zf::kChannelMajor) return d.m * d.cm_nch;
  return update_blocks(d.n, d.m, d.up_rows);
}

int64_t unpack_grid(const DevMat& d) {
  if (d.layout == zf::kChannelMajor) return d.m * d.cm_unch;
  return update_blocks(d.n, d.m, d.up_rows);
}

// Row-major: the 16-byte kernel serves the steps without a refresh (states in
// place, or no Adam); a refresh step (remap / init, whose per-column sources
// it would read element by element behind a chain of dependent index loads)
// runs the per-column kernel, which measured faster there.  Both give the
// same bits.
bool use_rv(const DevMat& one, int32_t mode, bool adam) {
  return one.layout == zf::kRowMajor && one.rv && (!adam || mode == zf::kInplace);
}

int64_t rv_grid(const DevMat& d) { return rv_blocks(d.n, d.m, d.rv_rows); }

// `rv` selects the row-major 16-byte kernel; t / blocks are then its table
// and grid.
hipError_t launch_update_any(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                             int32_t mode, int32_t first, bool adam, bool pack, int32_t layout,
                             hipStream_t s, bool handover, float scale, bool rv) {
  if (layout == zf::kChannelMajor)
    return zf::launch_cm_update(t, one, blocks, c, mode, first, adam, pack, nullptr, handover,
                                scale, s);
  if (rv) return zf::launch_rv_update(t, one, blocks, c, mode, first, adam, pack, handover, scale, s);
  return zf::launch_update(t, one, blocks, c, mode, first, adam, pack, handover, scale, s);
}

hipError_t launch_unpack_any(const Table& t, const DevMat& one, int64_t blocks, float scale,
                             int32_t layout, hipStream_t s) {
  return layout == zf::kChannelMajor ? zf::launch_cm_unpack(t, one, blocks, scale, s)
                                     : zf::launch_unpack(t, one, blocks, scale, s);
}

zf_status run_update(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad, int32_t layout,
                     const zf_selection* sel, int64_t k, float* master, float* exp_avg,
                     float* exp_avg_sq, int64_t ld_state, uint16_t* weight, int64_t ld_weight,
                     const zf_adam_hparams* hp, int64_t step, int32_t mode,
                     const zf_state_source* src, float* acc, int64_t ld_acc, int64_t sii,
                     int64_t S, bool adam, bool pack, zf_stream stream, float* out = nullptr,
                     int64_t ld_out = 0, float scale = 1.0f) {
  const bool handover = out != nullptr;
  if (!layout_ok(layout) || !shape_ok(n, m, k) ||
      !mat_ok(grad, ext(layout, n, m), ld_grad, 2))
    return ZF_EINVAL;
  if (!selection_ok(sel, m, k, true)) return ZF_EINVAL;
  DevMat d = base_mat(grad, n, m, ld_grad, layout, sel, k);
  const Span g = span(grad, ext(layout, n, m), ld_grad, 2);
  AdamK c{};
  if (adam) {
    if (!hparams_ok(hp) || step < 1) return ZF_EINVAL;
    if (mode == zf::kRemap && src == nullptr) return ZF_EINVAL;
    d.P = master;
    d.M = exp_avg;
    d.V = exp_avg_sq;
    d.ld_state = ld_state;
    d.weight = weight;
    d.ld_weight = ld_weight;
    apply_source(d, src);
    if (!adam_args_ok(d, mode, g)) return ZF_EINVAL;
    c = adam_consts(*hp, step);
  }
  if (pack) {
    d.acc = acc;
    d.ld_acc = ld_acc;
    if (!pack_args_ok(d, sii, S, g)) return ZF_EINVAL;
    if (adam) {
      const Span a = span(acc, ext(layout, n, m - k), ld_acc, 4);
      const Ext es = ext(layout, n, k);
      if (overlaps(a, span(master, es, ld_state, 4)) ||
          overlaps(a, span(exp_avg, es, ld_state, 4)) ||
          overlaps(a, span(exp_avg_sq, es, ld_state, 4)) ||
          overlaps(a, span(weight, ext(layout, n, m), ld_weight, 2)) || store_overlaps(d, a))
        return ZF_EINVAL;
    }
  }
  if (handover) {
    // the hand-over buffer is written: it must not overlap anything the pass reads or writes
    const Ext eo = ext(layout, n, m);
    if (!mat_ok(out, eo, ld_out, 4)) return ZF_EINVAL;
    const Span o = span(out, eo, ld_out, 4);
    const Ext es = ext(layout, n, k);
    if (overlaps(o, g) || overlaps(o, span(acc, ext(layout, n, m - k), ld_acc, 4)) ||
        overlaps(o, span(master, es, ld_state, 4)) || overlaps(o, span(exp_avg, es, ld_state, 4)) ||
        overlaps(o, span(exp_avg_sq, es, ld_state, 4)) ||
        overlaps(o, span(weight, ext(layout, n, m), ld_weight, 2)) || store_overlaps(d, o))
      return ZF_EINVAL;
    d.out = out;
    d.ld_out = ld_out;
  }
  // nothing to touch: no selected column to update, no leaving column to swap
  // out, no unselected column to pack
  const bool swap_out = adam && mode == zf::kRemap && d.st_P != nullptr;
  if (!handover && (!adam || k == 0) && !swap_out && (!pack || k == m)) return ZF_OK;
  finish_geometry(d, 256, pick_update_rows({{n, m}}));
  set_rv(d, pick_rv_rows({{n, m}}), true);
  if (layout == zf::kRowMajor && !rm_strides_ok(d)) return ZF_EINVAL;
  const bool rv = use_rv(d, mode, adam);
  const int64_t blocks = rv ? rv_grid(d) : update_grid(d);
  if (blocks == 0) return ZF_OK;
  const hipError_t e = launch_update_any(single_table(), d, blocks, c, adam ? mode : 0,
                                         sii == 1 ? 1 : 0, adam, pack, layout,
                                         as_stream(stream), handover, scale, rv);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================

extern "C" {

const char* zf_status_string(int status) {
  switch (status) {
    case ZF_OK: return "ZF_OK";
    case ZF_EINVAL: return "ZF_EINVAL: invalid argument";
    case ZF_EWORKSPACE: return "ZF_EWORKSPACE: workspace too small";
    case ZF_EHIP: return "ZF_EHIP: HIP call failed";
    case ZF_ENOMEM: return "ZF_ENOMEM: host allocation failed";
    default: return "unknown zf status";
  }
}

int zf_last_hip_error(void) { return g_last_hip_error; }

int64_t zf_k_from_ratio(double ratio, int64_t m) {
  if (!(ratio >= 0.0 && ratio <= 1.0) || m < 0) return -1;
  const double k = std::floor(ratio * static_cast<double>(m) + 0.5);
  return std::max<int64_t>(0, std::min<int64_t>(m, static_cast<int64_t>(k)));
}

size_t zf_colnorm_workspace_bytes(int64_t n, int64_t m, int32_t layout) {
  if (n <= 0 || m <= 0 || layout == zf::kChannelMajor) return 0;
  const int rpb = pick_colnorm_rows({{n, m}});
  return static_cast<size_t>(ceil_div(n, rpb)) * static_cast<size_t>(m) * sizeof(double);
}

zf_status zf_colnorm(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                     int32_t layout, float* norms_sq, void* ws, size_t ws_bytes,
                     zf_stream stream) {
  if (!layout_ok(layout) || !shape_ok(n, m, 0) ||
      !mat_ok(grad, ext(layout, n, m), ld_grad, 2) || !vector_ok(norms_sq, m, 4))
    return ZF_EINVAL;
  if (overlaps(span(grad, ext(layout, n, m), ld_grad, 2), span_of(norms_sq, 1, m, m, 4)))
    return ZF_EINVAL;
  const size_t need = zf_colnorm_workspace_bytes(n, m, layout);
  if (need > 0 && (ws == nullptr || ws_bytes < need || !aligned(ws, 8))) return ZF_EWORKSPACE;
  if (need > 0 && overlaps(Span{reinterpret_cast<uintptr_t>(ws),
                                reinterpret_cast<uintptr_t>(ws) + need},
                           span_of(norms_sq, 1, m, m, 4)))
    return ZF_EINVAL;
  if (m == 0) return ZF_OK;
  DevMat d = base_mat(grad, n, m, ld_grad, layout, nullptr, 0);
  d.norms = norms_sq;
  finish_geometry(d, n > 0 ? pick_colnorm_rows({{n, m}}) : 256, 64);
  d.cn_ws = 0;
  hipError_t e;
  if (layout == zf::kChannelMajor)
    e = zf::launch_cm_colnorm(single_table(), d, colnorm_grid(d), as_stream(stream));
  else
    e = zf::launch_colnorm(single_table(), d, colnorm_grid(d), single_table(),
                           ceil_div(m, zf::kFinalizeCols), static_cast<double*>(ws),
                           as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

}  // extern "C"

// ---- allocation-free column scores -----------------------------------------
// The workspace of zf_colnorm_noalloc: one array per GPU, part of this
// library's device code object (it lives as long as the process).  In host
// code `scratch` only names the symbol; its device address comes from
// hipGetSymbolAddress, once per device.
static __device__ __align__(256) double scratch[ZF_STATIC_SCRATCH_BYTES / sizeof(double)];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of `scratch` on the device `stream` belongs to (the
// current device for the null stream).  The first call for a device looks
// it up with that device current.
zf_status scratch_for(hipStream_t stream, void** out) {
  int dev = 0;
  hipError_t e = stream != nullptr ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  if (dev < 0 || dev >= kMaxDevices) return ZF_EINVAL;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      int cur = 0;
      e = hipGetDevice(&cur);
      if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
      if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (cur != dev) (void)hipSetDevice(cur);
      if (e != hipSuccess) return hip_fail(e);
      if (p == nullptr) return hip_fail(hipErrorInvalidSymbol);
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return ZF_OK;
}

}  // namespace

extern "C" {

zf_status zf_colnorm_noalloc(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                             int32_t layout, float* norms_sq, zf_stream stream) {
  // the same host validation as zf_colnorm, before the scratch is looked up
  if (!layout_ok(layout) || !shape_ok(n, m, 0) ||
      !mat_ok(grad, ext(layout, n, m), ld_grad, 2) || !vector_ok(norms_sq, m, 4))
    return ZF_EINVAL;
  const size_t need = zf_colnorm_workspace_bytes(n, m, layout);
  if (need > ZF_STATIC_SCRATCH_BYTES) return ZF_EWORKSPACE;
  void* ws = nullptr;
  if (need > 0) {
    const zf_status st = scratch_for(as_stream(stream), &ws);
    if (st != ZF_OK) return st;
  }
  return zf_colnorm(grad, n, m, ld_grad, layout, norms_sq, ws, need, stream);
}

zf_status zf_stream_probe(int32_t kind, const void* src, void* dst, size_t bytes, uint32_t key,
                          zf_stream stream) {
  if (kind < 0 || kind > 2 || bytes == 0 || bytes % 16 != 0 ||
      bytes > static_cast<size_t>(INT64_MAX / 2) || dst == nullptr)
    return ZF_EINVAL;
  const int64_t nb = static_cast<int64_t>(bytes);
  // one launch: at most 2^32 - 1 work-items
  if (zf::stream_probe_blocks(nb) > ((int64_t(1) << 32) - 1) / zf::kThreads) return ZF_EINVAL;
  if (kind == 0 && !aligned(dst, 4)) return ZF_EINVAL;
  if (kind != 0 && !aligned(dst, 16)) return ZF_EINVAL;
  if (kind != 2 && (src == nullptr || !aligned(src, 16))) return ZF_EINVAL;
  if (kind == 1 && overlaps(span_of(src, 1, nb, nb, 1), span_of(dst, 1, nb, nb, 1)))
    return ZF_EINVAL;
  const hipError_t e = zf::launch_stream_probe(kind, src, dst, nb, key, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_topk_select(const float* norms_sq, int64_t m, double ratio, const zf_selection* out,
                         int64_t* k_out, zf_stream stream) {
  const int64_t k = zf_k_from_ratio(ratio, m);
  if (k < 0 || !shape_ok(0, m, k) || !vector_ok(norms_sq, m, 4) ||
      !selection_ok(out, m, k, true))
    return ZF_EINVAL;
  const Span in = span_of(norms_sq, 1, m, m, 4);
  const Span outs[4] = {span_of(out->sel_idx, 1, k, k, 4), span_of(out->unsel_idx, 1, m - k, m - k, 4),
                        span_of(out->sel_mask, 1, ceil_div(m, 64), ceil_div(m, 64), 8),
                        span_of(out->sel_prefix, 1, ceil_div(m, 64), ceil_div(m, 64), 4)};
  for (int a = 0; a < 4; ++a) {
    if (overlaps(outs[a], in)) return ZF_EINVAL;
    for (int b = a + 1; b < 4; ++b)
      if (overlaps(outs[a], outs[b])) return ZF_EINVAL;
  }
  if (k_out != nullptr) *k_out = k;
  if (m == 0) return ZF_OK;
  DevMat d = base_mat(nullptr, 0, m, m, zf::kRowMajor, out, k);
  d.norms = const_cast<float*>(norms_sq);
  const hipError_t e = zf::launch_topk(single_table(), d, 1, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_adam_selected(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                           int32_t layout, const zf_selection* sel, int64_t k, float* master,
                           float* exp_avg, float* exp_avg_sq, int64_t ld_state, uint16_t* weight,
                           int64_t ld_weight, const zf_adam_hparams* hp, int64_t step,
                           int32_t mode, const zf_state_source* src, zf_stream stream) {
  return run_update(grad, n, m, ld_grad, layout, sel, k, master, exp_avg, exp_avg_sq, ld_state,
                    weight, ld_weight, hp, step, mode, src, nullptr, 0, 1, 1, true, false,
                    stream);
}

zf_status zf_pack_accumulate(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                             int32_t layout, const zf_selection* sel, int64_t k, float* acc,
                             int64_t ld_acc, int64_t step_in_interval, int64_t accum_interval,
                             zf_stream stream) {
  return run_update(grad, n, m, ld_grad, layout, sel, k, nullptr, nullptr, nullptr, 0, nullptr,
                    0, nullptr, 1, 0, nullptr, acc, ld_acc, step_in_interval, accum_interval,
                    false, true, stream);
}

zf_status zf_update_fused(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                          int32_t layout, const zf_selection* sel, int64_t k, float* master,
                          float* exp_avg, float* exp_avg_sq, int64_t ld_state, uint16_t* weight,
                          int64_t ld_weight, const zf_adam_hparams* hp, int64_t step,
                          int32_t mode, const zf_state_source* src, float* acc, int64_t ld_acc,
                          int64_t step_in_interval, int64_t accum_interval, zf_stream stream) {
  return run_update(grad, n, m, ld_grad, layout, sel, k, master, exp_avg, exp_avg_sq, ld_state,
                    weight, ld_weight, hp, step, mode, src, acc, ld_acc, step_in_interval,
                    accum_interval, true, true, stream);
}

zf_status zf_update_fused_handover(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                                   int32_t layout, const zf_selection* sel, int64_t k,
                                   float* master, float* exp_avg, float* exp_avg_sq,
                                   int64_t ld_state, uint16_t* weight, int64_t ld_weight,
                                   const zf_adam_hparams* hp, int64_t step, int32_t mode,
                                   const zf_state_source* src, const float* acc, int64_t ld_acc,
                                   int64_t step_in_interval, int64_t accum_interval, float scale,
                                   float* out, int64_t ld_out, zf_stream stream) {
  if (out == nullptr && n > 0 && m > 0) return ZF_EINVAL;
  if (out == nullptr) return ZF_OK;
  return run_update(grad, n, m, ld_grad, layout, sel, k, master, exp_avg, exp_avg_sq, ld_state,
                    weight, ld_weight, hp, step, mode, src, const_cast<float*>(acc), ld_acc,
                    step_in_interval, accum_interval, true, true, stream, out, ld_out, scale);
}

zf_status zf_unpack(const float* acc, int64_t ld_acc, const zf_selection* sel, int64_t k,
                    int64_t n, int64_t m, int32_t layout, float scale, float* out, int64_t ld_out,
                    zf_stream stream) {
  if (!layout_ok(layout) || !shape_ok(n, m, k) || !selection_ok(sel, m, k, false) ||
      !mat_ok(acc, ext(layout, n, m - k), ld_acc, 4) ||
      !mat_ok(out, ext(layout, n, m), ld_out, 4))
    return ZF_EINVAL;
  if (overlaps(span(acc, ext(layout, n, m - k), ld_acc, 4), span(out, ext(layout, n, m), ld_out, 4)))
    return ZF_EINVAL;
  DevMat d = base_mat(nullptr, n, m, 0, layout, sel, k);
  d.acc = const_cast<float*>(acc);
  d.ld_acc = ld_acc;
  d.out = out;
  d.ld_out = ld_out;
  finish_geometry(d, 256, pick_update_rows({{n, m}}));
  if (layout == zf::kRowMajor && !rm_strides_ok(d)) return ZF_EINVAL;
  const int64_t blocks = unpack_grid(d);
  if (blocks == 0) return ZF_OK;
  const hipError_t e =
      launch_unpack_any(single_table(), d, blocks, scale, layout, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_scatter_weights(const uint16_t* weight_cols, int64_t ld_wcols,
                             const zf_selection* sel, int64_t k, int64_t n, int64_t m,
                             int32_t layout, uint16_t* weight, int64_t ld_weight,
                             zf_stream stream) {
  if (!layout_ok(layout) || !shape_ok(n, m, k) || !selection_ok(sel, m, k, false) ||
      !mat_ok(weight_cols, ext(layout, n, m - k), ld_wcols, 2) ||
      !mat_ok(weight, ext(layout, n, m), ld_weight, 2))
    return ZF_EINVAL;
  if (overlaps(span(weight_cols, ext(layout, n, m - k), ld_wcols, 2),
               span(weight, ext(layout, n, m), ld_weight, 2)))
    return ZF_EINVAL;
  if (n > 0 && m > k && !device_accessible(weight_cols)) return ZF_EINVAL;
  DevMat d = base_mat(nullptr, n, m, 0, layout, sel, k);
  d.wcols = weight_cols;
  d.ld_wcols = ld_wcols;
  d.weight = weight;
  d.ld_weight = ld_weight;
  finish_geometry(d, 256, pick_update_rows({{n, m}}));
  const int64_t blocks = unpack_grid(d);
  if (blocks == 0 || k == m) return ZF_OK;
  const hipError_t e = zf::launch_scatter(single_table(), d, blocks, layout, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

}  // extern "C"

// ===========================================================================
// Plans
// ===========================================================================

struct zf_plan {
  int32_t nmats = 0;
  int32_t layout = 0;
  std::vector<DevMat> mats;
  void* dev = nullptr;     // caller-provided device memory (tables, then workspaces)
  size_t dev_bytes = 0;    // bytes of it the plan uses
  size_t head_bytes = 0;   // descriptor tables at the start of dev
  std::vector<char> image;  // host image of the tables, the source of the upload
  int64_t ws_doubles = 0, zs_doubles = 0, zb_doubles = 0;
  DevMat* d_mats = nullptr;
  int64_t* d_off_cn = nullptr;
  int64_t* d_off_fin = nullptr;
  int64_t* d_off_top = nullptr;
  int64_t* d_off_up = nullptr;
  int64_t* d_off_unp = nullptr;
  int64_t* d_off_zen = nullptr;
  int64_t* d_off_zp = nullptr;  // row-major Zen-auto partial pass
  int64_t* d_off_upv = nullptr;  // row-major 16-byte update
  int64_t* d_off_sel = nullptr;  // channel-major Adam over the selected channels only
  double* d_ws = nullptr;
  double* d_zs = nullptr;  // Zen-auto per-wave partials
  double* d_zb = nullptr;  // Zen-auto per-finalize-block sums
  int64_t blk_cn = 0, blk_fin = 0, blk_top = 0, blk_up = 0, blk_unp = 0, blk_zen = 0, blk_zp = 0,
          blk_upv = 0, blk_sel = 0;
  int64_t k_total = 0, u_total = 0;
  bool can_colnorm = true, can_topk = true, can_adam = true, can_remap = true, can_pack = true,
       can_unpack = true, can_zen = true, can_scatter = true, can_handover = true,
       can_pending = true, can_scatter_skip = true;
  bool has_acc1 = false;  // some descriptor gives the bf16 first-step stage
  bool all_acc1 = true;   // every descriptor does
  bool has_store = false;  // some descriptor gives a full-state store
  bool can_colnorm_out = true;  // scores and the hand-over rows in one pass
};

namespace {

DevMat plan_mat(const zf_matrix& x) {
  DevMat d = base_mat(x.grad, x.n, x.m, x.ld_grad, x.layout, &x.sel, x.k);
  d.P = x.master;
  d.M = x.exp_avg;
  d.V = x.exp_avg_sq;
  d.ld_state = x.ld_state;
  d.weight = x.weight;
  d.ld_weight = x.ld_weight;
  d.acc = x.acc;
  d.ld_acc = x.ld_acc;
  d.norms = x.norms_sq;
  d.out = x.unpacked;
  d.ld_out = x.ld_unpacked;
  d.sel_sq = x.sel_sq;
  d.acc_sq = x.acc_sq;
  d.wcols = x.weight_cols;
  d.ld_wcols = x.ld_weight_cols;
  d.acc1 = x.acc_first;
  d.ld_acc1 = x.ld_acc_first;
  apply_source(d, &x.src);
  return d;
}

// Validates what a descriptor provides; records which stages it can run.
zf_status check_plan_matrix(const zf_matrix& x, zf_plan& p) {
  const int64_t n = x.n, m = x.m, k = x.k;
  const int32_t L = x.layout;
  if (!layout_ok(L) || L != p.layout || !shape_ok(n, m, k)) return ZF_EINVAL;
  const int64_t words = ceil_div(m, 64);
  const Ext eg = ext(L, n, m), ea = ext(L, n, m - k);
  const Span g = span(x.grad, eg, x.ld_grad, 2);
  const bool have_grad = mat_ok(x.grad, eg, x.ld_grad, 2);
  const bool have_mask = vector_ok(x.sel.sel_mask, words, 8) && vector_ok(x.sel.sel_prefix, words, 4);
  const bool have_idx = vector_ok(x.sel.sel_idx, k, 4) && vector_ok(x.sel.unsel_idx, m - k, 4);
  const bool have_norms = vector_ok(x.norms_sq, m, 4);
  p.can_colnorm = p.can_colnorm && have_grad && have_norms &&
                  !overlaps(g, span_of(x.norms_sq, 1, m, m, 4));
  p.can_topk = p.can_topk && have_norms && have_mask && have_idx;

  DevMat d = plan_mat(x);
  p.can_adam = p.can_adam && have_grad && have_mask && have_idx &&
               (n * k == 0 || adam_args_ok(d, zf::kInplace, g));
  p.can_remap = p.can_remap && p.can_adam && (n * k == 0 || adam_args_ok(d, zf::kRemap, g)) &&
                !store_overlaps(d, span(x.acc, ea, x.ld_acc, 4));
  p.can_pack = p.can_pack && have_grad && have_mask && have_idx && pack_args_ok(d, 1, 1, g);
  p.can_unpack = p.can_unpack && have_mask && mat_ok(x.acc, ea, x.ld_acc, 4) &&
                 mat_ok(x.unpacked, eg, x.ld_unpacked, 4) &&
                 !overlaps(span(x.acc, ea, x.ld_acc, 4), span(x.unpacked, eg, x.ld_unpacked, 4));
  {
    // fused hand-over: the unpacked buffer must be disjoint from everything the update touches
    const Span o = span(x.unpacked, eg, x.ld_unpacked, 4);
    const Ext es = ext(L, n, k);
    p.can_handover = p.can_handover && mat_ok(x.unpacked, eg, x.ld_unpacked, 4) &&
                     (n * m == 0 || x.unpacked != nullptr) && !overlaps(o, g) &&
                     !overlaps(o, span(x.acc, ea, x.ld_acc, 4)) &&
                     !overlaps(o, span(x.master, es, x.ld_state, 4)) &&
                     !overlaps(o, span(x.exp_avg, es, x.ld_state, 4)) &&
                     !overlaps(o, span(x.exp_avg_sq, es, x.ld_state, 4)) &&
                     !overlaps(o, span(x.weight, eg, x.ld_weight, 2)) && !store_overlaps(d, o);
  }
  p.can_scatter = p.can_scatter && have_mask && mat_ok(x.weight_cols, ea, x.ld_weight_cols, 2) &&
                  (n * (m - k) == 0 || device_accessible(x.weight_cols)) &&
                  mat_ok(x.weight, eg, x.ld_weight, 2) &&
                  !overlaps(span(x.weight_cols, ea, x.ld_weight_cols, 2),
                            span(x.weight, eg, x.ld_weight, 2));
  p.can_scatter_skip = p.can_scatter_skip && p.can_scatter && vector_ok(x.src.prev_mask, words, 8);
  p.can_colnorm_out = p.can_colnorm_out && p.can_colnorm && p.can_handover &&
                      !overlaps(span_of(x.norms_sq, 1, m, m, 4),
                                span(x.unpacked, eg, x.ld_unpacked, 4));
  // refresh with the owed deferred update: the store, and the previous
  // interval's sums, read only, disjoint from everything the update writes
  {
    const Span pa = span(x.src.pend_acc, ea, x.src.ld_pend, 4);
    const Ext es = ext(L, n, k);
    p.can_pending = p.can_pending && x.src.store_master != nullptr &&
                    mat_ok(x.src.pend_acc, ea, x.src.ld_pend, 4) &&
                    (n * (m - k) == 0 || device_accessible(x.src.pend_acc)) &&
                    !overlaps(pa, span(x.acc, ea, x.ld_acc, 4)) &&
                    !overlaps(pa, span(x.master, es, x.ld_state, 4)) &&
                    !overlaps(pa, span(x.exp_avg, es, x.ld_state, 4)) &&
                    !overlaps(pa, span(x.exp_avg_sq, es, x.ld_state, 4)) &&
                    !overlaps(pa, span(x.weight, eg, x.ld_weight, 2)) && !store_overlaps(d, pa);
  }
  // Zen-auto statistics: [k] and [m-k] fp32 outputs that overlap neither
  // each other nor any buffer the fused update touches.
  {
    const Span zsel = span_of(x.sel_sq, 1, k, k, 4), zacc = span_of(x.acc_sq, 1, m - k, m - k, 4);
    const Span others[6] = {g, span(x.acc, ea, x.ld_acc, 4),
                            span(x.master, ext(L, n, k), x.ld_state, 4),
                            span(x.exp_avg, ext(L, n, k), x.ld_state, 4),
                            span(x.exp_avg_sq, ext(L, n, k), x.ld_state, 4),
                            span(x.weight, eg, x.ld_weight, 2)};
    bool ok = vector_ok(x.sel_sq, k, 4) && vector_ok(x.acc_sq, m - k, 4) &&
              !overlaps(zsel, zacc);
    for (int a = 0; ok && a < 6; ++a) ok = !overlaps(zsel, others[a]) && !overlaps(zacc, others[a]);
    p.can_zen = p.can_zen && ok;
  }
  // The bf16 first-step stage (the gradient's shape: channel-major one row
  // per channel, row-major [n][ld >= m] with 16-byte rows): disjoint from
  // everything the update reads or writes.
  if (x.acc_first != nullptr) {
    if (!mat_ok(x.acc_first, eg, x.ld_acc_first, 2)) return ZF_EINVAL;
    // (16-byte rows; a single row never uses its stride)
    if (L == zf::kRowMajor && (!aligned(x.acc_first, 16) || (n > 1 && x.ld_acc_first % 8 != 0)))
      return ZF_EINVAL;
    const Span st = span(x.acc_first, eg, x.ld_acc_first, 2);
    const Ext es = ext(L, n, k);
    if (overlaps(st, g) || overlaps(st, span(x.acc, ea, x.ld_acc, 4)) ||
        overlaps(st, span(x.weight, eg, x.ld_weight, 2)) ||
        overlaps(st, span(x.master, es, x.ld_state, 4)) ||
        overlaps(st, span(x.exp_avg, es, x.ld_state, 4)) ||
        overlaps(st, span(x.exp_avg_sq, es, x.ld_state, 4)) ||
        overlaps(st, span(x.unpacked, eg, x.ld_unpacked, 4)) || store_overlaps(d, st))
      return ZF_EINVAL;
    p.has_acc1 = true;
  } else {
    p.all_acc1 = false;
  }
  // Strides must be valid whenever the buffer is given.
  if (x.weight && !mat_ok(x.weight, eg, x.ld_weight, 2)) return ZF_EINVAL;
  if (x.acc && !mat_ok(x.acc, ea, x.ld_acc, 4)) return ZF_EINVAL;
  if (x.unpacked && !mat_ok(x.unpacked, eg, x.ld_unpacked, 4)) return ZF_EINVAL;
  if (x.grad && !have_grad) return ZF_EINVAL;
  return ZF_OK;
}

// Validates the descriptors and computes everything a plan holds on the
// host: geometry, grids, the host image of its device tables and the size
// of its workspaces.  No device work.
zf_status build_plan_impl(const zf_matrix* mats, int32_t nmats, zf_plan* p) {
  if (mats == nullptr || nmats < 1) return ZF_EINVAL;
  p->nmats = nmats;
  p->layout = mats[0].layout;
  std::vector<std::pair<int64_t, int64_t>> shapes;
  for (int32_t q = 0; q < nmats; ++q) {
    const zf_status st = check_plan_matrix(mats[q], *p);
    if (st != ZF_OK) return st;
    shapes.emplace_back(mats[q].n, mats[q].m);
  }
  const int cn_rows = pick_colnorm_rows(shapes);
  const int up_rows = pick_update_rows(shapes);
  // a row-major plan with the Zen-auto statistics runs the 16-byte update in
  // blocks of the column-score row blocks, so that its fused statistics are
  // the statistics pass's partials (same row blocks, same order)
  const int rv_rows = (p->layout == zf::kRowMajor && p->can_zen) ? cn_rows : pick_rv_rows(shapes);
  // the row-major 16-byte update serves the plan if every matrix qualifies
  bool all_rv = p->layout == zf::kRowMajor;
  for (int32_t q = 0; q < nmats && all_rv; ++q) {
    DevMat d = plan_mat(mats[q]);
    finish_geometry(d, cn_rows, up_rows, p->can_zen);
    all_rv = rv_ok(d) && strides_fit(d, rv_rows);
  }
  std::vector<int64_t> off_cn(nmats + 1), off_fin(nmats + 1), off_top(nmats + 1),
      off_up(nmats + 1), off_unp(nmats + 1), off_zen(nmats + 1), off_zp(nmats + 1),
      off_upv(nmats + 1), off_sel(nmats + 1);
  int64_t ws_doubles = 0, zs_doubles = 0;
  const bool cm = p->layout == zf::kChannelMajor;
  p->mats.resize(nmats);
  for (int32_t q = 0; q < nmats; ++q) {
    DevMat d = plan_mat(mats[q]);
    finish_geometry(d, cn_rows, up_rows, p->can_zen);
    set_rv(d, rv_rows, all_rv);
    if (!cm && !rm_strides_ok(d)) return ZF_EINVAL;
    d.cn_ws = ws_doubles;
    if (!cm) ws_doubles += static_cast<int64_t>(d.cn_rb) * d.m;
    d.zs_off = zs_doubles;
    if (p->can_zen) {
      // channel-major: per-wave partials of the fused pass; row-major: the
      // separate pass reuses the column-score workspace (cn_rb x m doubles)
      if (cm) zs_doubles += d.m * static_cast<int64_t>(d.cm_nch) * zf::kCmWaves;
      off_zen[q] = p->blk_zen;
      p->blk_zen += ceil_div(d.m, zf::kZenCols);
      off_zp[q] = p->blk_zp;
      if (!cm) p->blk_zp += ceil_div(d.m, zf::kZenCols) * static_cast<int64_t>(d.cn_rb);
    }
    p->k_total += d.k;
    p->u_total += d.m - d.k;
    off_cn[q] = p->blk_cn;
    off_fin[q] = p->blk_fin;
    off_top[q] = p->blk_top;
    off_up[q] = p->blk_up;
    off_upv[q] = p->blk_upv;
    off_sel[q] = p->blk_sel;
    off_unp[q] = p->blk_unp;
    p->blk_cn += colnorm_grid(d);
    p->blk_fin += cm ? 0 : ceil_div(d.m, zf::kFinalizeCols);
    p->blk_top += 1;
    p->blk_up += update_grid(d);
    if (d.rv) p->blk_upv += rv_grid(d);
    if (cm) p->blk_sel += d.k * static_cast<int64_t>(d.cm_snch);
    p->has_store = p->has_store || d.st_P != nullptr;
    p->blk_unp += unpack_grid(d);
    p->mats[q] = d;
  }
  off_cn[nmats] = p->blk_cn;
  off_fin[nmats] = p->blk_fin;
  off_top[nmats] = p->blk_top;
  off_up[nmats] = p->blk_up;
  off_unp[nmats] = p->blk_unp;
  off_zen[nmats] = p->blk_zen;
  off_zp[nmats] = p->blk_zp;
  off_upv[nmats] = p->blk_upv;
  off_sel[nmats] = p->blk_sel;
  // one launch holds at most 2^32 - 1 work-items in x (the dispatch
  // packet's grid size is a 32-bit count of work-items)
  const int64_t max_blocks = ((int64_t(1) << 32) - 1) / zf::kThreads;
  if (p->blk_cn > max_blocks || p->blk_up > max_blocks || p->blk_unp > max_blocks ||
      p->blk_upv > max_blocks || p->blk_sel > max_blocks ||
      p->blk_zp > max_blocks)
    return ZF_EINVAL;  // grid too large for one launch

  const size_t mats_bytes = sizeof(DevMat) * nmats;
  const size_t off_bytes = sizeof(int64_t) * (nmats + 1);
  const size_t head = (mats_bytes + 9 * off_bytes + 255) & ~size_t(255);
  p->ws_doubles = ws_doubles;
  p->zs_doubles = zs_doubles;
  p->zb_doubles = p->can_zen ? 2 * p->blk_zen : 0;
  p->head_bytes = head;
  p->dev_bytes =
      head + sizeof(double) * static_cast<size_t>(ws_doubles + zs_doubles + p->zb_doubles);
  p->image.assign(head, 0);
  char* img = p->image.data();
  std::memcpy(img, p->mats.data(), mats_bytes);
  const std::vector<int64_t>* offs[9] = {&off_cn, &off_fin, &off_top, &off_up, &off_unp,
                                         &off_zen, &off_zp, &off_upv, &off_sel};
  for (int a = 0; a < 9; ++a)
    std::memcpy(img + mats_bytes + a * off_bytes, offs[a]->data(), off_bytes);
  return ZF_OK;
}

// build_plan_impl with host allocation failures (std::bad_alloc from its
// vectors) turned into a status: no exception crosses the C ABI.
zf_status build_plan(const zf_matrix* mats, int32_t nmats, zf_plan* p) {
  try {
    return build_plan_impl(mats, nmats, p);
  } catch (...) {
    return ZF_ENOMEM;
  }
}

// Points the plan's tables and workspaces into `dev` (the table layout of
// build_plan's image).
void place_plan(zf_plan* p, void* dev) {
  const int32_t nmats = p->nmats;
  const size_t mats_bytes = sizeof(DevMat) * nmats;
  char* base = static_cast<char*>(dev);
  p->dev = dev;
  p->d_mats = reinterpret_cast<DevMat*>(base);
  p->d_off_cn = reinterpret_cast<int64_t*>(base + mats_bytes);
  p->d_off_fin = p->d_off_cn + (nmats + 1);
  p->d_off_top = p->d_off_fin + (nmats + 1);
  p->d_off_up = p->d_off_top + (nmats + 1);
  p->d_off_unp = p->d_off_up + (nmats + 1);
  p->d_off_zen = p->d_off_unp + (nmats + 1);
  p->d_off_zp = p->d_off_zen + (nmats + 1);
  p->d_off_upv = p->d_off_zp + (nmats + 1);
  p->d_off_sel = p->d_off_upv + (nmats + 1);
  p->d_ws = reinterpret_cast<double*>(base + p->head_bytes);
  p->d_zs = p->d_ws + p->ws_doubles;
  p->d_zb = p->d_zs + p->zs_doubles;
}

}  // namespace

extern "C" {

zf_status zf_plan_query(const zf_matrix* mats, int32_t nmats, size_t* device_bytes) {
  if (device_bytes == nullptr) return ZF_EINVAL;
  zf_plan* p = new (std::nothrow) zf_plan();
  if (p == nullptr) return ZF_ENOMEM;
  const zf_status st = build_plan(mats, nmats, p);
  if (st == ZF_OK) *device_bytes = p->dev_bytes;
  delete p;
  return st;
}

zf_status zf_plan_create(const zf_matrix* mats, int32_t nmats, void* device_mem,
                         size_t device_bytes, zf_stream stream, zf_plan** out) {
  if (out == nullptr || device_mem == nullptr || !aligned(device_mem, 256)) return ZF_EINVAL;
  zf_plan* p = new (std::nothrow) zf_plan();
  if (p == nullptr) return ZF_ENOMEM;
  zf_status st = build_plan(mats, nmats, p);
  if (st == ZF_OK && device_bytes < p->dev_bytes) st = ZF_EWORKSPACE;
  if (st != ZF_OK) {
    delete p;
    return st;
  }
  place_plan(p, device_mem);
  // stream-ordered upload of the tables; the host image stays with the plan
  const hipError_t e = hipMemcpyAsync(p->dev, p->image.data(), p->head_bytes,
                                      hipMemcpyHostToDevice, as_stream(stream));
  if (e != hipSuccess) {
    g_last_hip_error = static_cast<int>(e);
    delete p;
    return ZF_EHIP;
  }
  *out = p;
  return ZF_OK;
}

void zf_plan_destroy(zf_plan* plan) { delete plan; }

size_t zf_plan_device_bytes(const zf_plan* plan) { return plan ? plan->dev_bytes : 0; }

zf_status zf_plan_colnorm(zf_plan* p, zf_stream stream) {
  if (p == nullptr || !p->can_colnorm) return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_cn, p->nmats};
  hipError_t e;
  if (p->layout == zf::kChannelMajor) {
    e = zf::launch_cm_colnorm(t, p->mats[0], p->blk_cn, as_stream(stream));
  } else {
    const Table tf{p->d_mats, p->d_off_fin, p->nmats};
    e = zf::launch_colnorm(t, p->mats[0], p->blk_cn, tf, p->blk_fin, p->d_ws, as_stream(stream));
  }
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_colnorm_stage(zf_plan* p, zf_stream stream) {
  if (p == nullptr || !p->can_colnorm || !p->has_acc1) return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_cn, p->nmats};
  hipError_t e;
  if (p->layout == zf::kChannelMajor) {
    e = zf::launch_cm_colnorm(t, p->mats[0], p->blk_cn, as_stream(stream), 1);
  } else {
    const Table tf{p->d_mats, p->d_off_fin, p->nmats};
    e = zf::launch_colnorm(t, p->mats[0], p->blk_cn, tf, p->blk_fin, p->d_ws, as_stream(stream),
                           true);
  }
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_colnorm_handover(zf_plan* p, float scale, zf_stream stream) {
  if (p == nullptr || !p->can_colnorm_out || p->layout != zf::kChannelMajor ||
      !std::isfinite(scale))
    return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_cn, p->nmats};
  const hipError_t e =
      zf::launch_cm_colnorm(t, p->mats[0], p->blk_cn, as_stream(stream), 2, scale);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_topk_select(zf_plan* p, zf_stream stream) {
  if (p == nullptr || !p->can_topk) return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_top, p->nmats};
  const hipError_t e = zf::launch_topk(t, p->mats[0], p->blk_top, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

}  // extern "C"

namespace {

// The pack phase passed to the update kernels: 1 on an interval's first
// step, 2 on its second when the plan keeps a bf16 first-step stage, else
// 0.
int32_t pack_phase(const zf_plan* p, int64_t step_in_interval) {
  if (step_in_interval == 1) return 1;
  return (step_in_interval == 2 && p->has_acc1) ? 2 : 0;
}

// The plan's update launch: the row-major 16-byte kernel where it applies
// (its own block table); channel-major Adam alone without a store over the
// selected channels only (its own block table); else the plan's update
// kernel.
hipError_t plan_update_launch(const zf_plan* p, const AdamK& c, int32_t mode, int32_t first,
                              bool adam, bool pack, bool handover, float scale, hipStream_t s) {
  if (p->layout == zf::kChannelMajor && adam && !pack && !handover && !p->has_store) {
    const Table ts{p->d_mats, p->d_off_sel, p->nmats};
    return zf::launch_cm_adam_selected_grid(ts, p->mats[0], p->blk_sel, c, mode, s);
  }
  const bool rv = use_rv(p->mats[0], mode, adam);
  const Table t{p->d_mats, rv ? p->d_off_upv : p->d_off_up, p->nmats};
  return launch_update_any(t, p->mats[0], rv ? p->blk_upv : p->blk_up, c, adam ? mode : 0, first,
                           adam, pack, p->layout, s, handover, scale, rv);
}

}  // namespace

extern "C" {

zf_status zf_plan_update(zf_plan* p, const zf_adam_hparams* hp, int64_t step, int32_t mode,
                         int64_t step_in_interval, int64_t accum_interval, int32_t do_adam,
                         int32_t do_pack, zf_stream stream) {
  if (p == nullptr || (!do_adam && !do_pack)) return ZF_EINVAL;
  AdamK c{};
  if (do_adam) {
    if (!p->can_adam || !hparams_ok(hp) || step < 1) return ZF_EINVAL;
    if (mode != zf::kInplace && mode != zf::kRemap && mode != zf::kInit) return ZF_EINVAL;
    if (mode == zf::kRemap && !p->can_remap) return ZF_EINVAL;
    c = adam_consts(*hp, step);
  }
  if (do_pack) {
    if (!p->can_pack || accum_interval < 1 || step_in_interval < 1 ||
        step_in_interval > accum_interval)
      return ZF_EINVAL;
  }
  const hipError_t e = plan_update_launch(p, c, mode, do_pack ? pack_phase(p, step_in_interval) : 0,
                                          do_adam != 0, do_pack != 0, false, 1.0f,
                                          as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_update_adam_handover(zf_plan* p, const zf_adam_hparams* hp, int64_t step,
                                       int32_t mode, zf_stream stream) {
  if (p == nullptr || !p->can_adam || !p->can_handover || p->layout != zf::kChannelMajor ||
      p->has_store)
    return ZF_EINVAL;
  if (!hparams_ok(hp) || step < 1) return ZF_EINVAL;
  if (mode != zf::kInplace && mode != zf::kRemap && mode != zf::kInit) return ZF_EINVAL;
  if (mode == zf::kRemap && !p->can_remap) return ZF_EINVAL;
  const Table ts{p->d_mats, p->d_off_sel, p->nmats};
  const hipError_t e = zf::launch_cm_adam_selected_grid(ts, p->mats[0], p->blk_sel,
                                                        adam_consts(*hp, step), mode,
                                                        as_stream(stream), true);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_unpack_first(zf_plan* p, float scale, zf_stream stream) {
  if (p == nullptr || !p->can_unpack || !p->all_acc1 || p->layout != zf::kChannelMajor)
    return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_unp, p->nmats};
  const hipError_t e =
      zf::launch_cm_unpack(t, p->mats[0], p->blk_unp, scale, as_stream(stream), true);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_unpack(zf_plan* p, float scale, zf_stream stream) {
  if (p == nullptr || !p->can_unpack) return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_unp, p->nmats};
  const hipError_t e =
      launch_unpack_any(t, p->mats[0], p->blk_unp, scale, p->layout, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_update_handover(zf_plan* p, const zf_adam_hparams* hp, int64_t step,
                                  int32_t mode, int64_t step_in_interval, int64_t accum_interval,
                                  float scale, zf_stream stream) {
  // (an interval's first step hands over scale * G: the packed buffer is
  // neither read nor written, so a plan without one may run it)
  if (p == nullptr || !p->can_adam || !p->can_handover) return ZF_EINVAL;
  if (!p->can_pack && step_in_interval != 1) return ZF_EINVAL;
  if (!hparams_ok(hp) || step < 1) return ZF_EINVAL;
  if (mode != zf::kInplace && mode != zf::kRemap && mode != zf::kInit) return ZF_EINVAL;
  if (mode == zf::kRemap && !p->can_remap) return ZF_EINVAL;
  if (accum_interval < 1 || step_in_interval < 1 || step_in_interval > accum_interval)
    return ZF_EINVAL;
  const AdamK c = adam_consts(*hp, step);
  const hipError_t e = plan_update_launch(p, c, mode, pack_phase(p, step_in_interval), true, true,
                                          true, scale, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

}  // extern "C"

namespace {

// The earlier steps' plans of a call with deferred packing (oldest first):
// the same matrices as p (count, shapes, k; channel-major: access path and
// geometry), each with its gradient, read only and disjoint from every
// buffer the step writes.  rv (row-major): cleared when an earlier gradient
// does not fit the 16-byte kernel's addressing.
zf_status gather_earlier(const zf_plan* p, const zf_plan* const* earlier, int32_t n_earlier,
                         zf::HistTable& h, bool& rv) {
  if (n_earlier < 0 || n_earlier > zf::kMaxDeferred || (n_earlier > 0 && earlier == nullptr))
    return ZF_EINVAL;
  const int32_t L = p->layout;
  const bool cm = L == zf::kChannelMajor;
  h.n = n_earlier;
  for (int32_t s = 0; s < n_earlier; ++s) {
    const zf_plan* e = earlier[s];
    if (e == nullptr || e->nmats != p->nmats || e->layout != L) return ZF_EINVAL;
    for (int32_t q = 0; q < p->nmats; ++q) {
      const DevMat& a = e->mats[q];
      const DevMat& b = p->mats[q];
      if (a.n != b.n || a.m != b.m || a.k != b.k) return ZF_EINVAL;
      if (cm && (a.vec != b.vec || a.cm_qpt != b.cm_qpt || a.cm_nch != b.cm_nch ||
                 a.cm_snch != b.cm_snch || a.cm_unch != b.cm_unch))
        return ZF_EINVAL;
      if (b.n * (b.m - b.k) > 0 && a.grad == nullptr) return ZF_EINVAL;
      if (!cm) {
        // the row blocks of this plan's kernels address the earlier rows
        // through the same 32-bit offsets
        const int64_t lim = int64_t(1) << 31;
        if (b.n > 1 && a.ld_grad * 2 >= lim / std::max<int64_t>(b.up_rows, 1)) return ZF_EINVAL;
        if (rv && !(aligned(a.grad, 16) && (b.n <= 1 || (a.ld_grad % 8 == 0 &&
                                                          a.ld_grad * 2 < lim / b.rv_rows))))
          rv = false;
      }
      // an earlier gradient is only read: disjoint from everything the step writes
      const Span g = span(a.grad, ext(L, a.n, a.m), a.ld_grad, 2);
      const Ext es = ext(L, b.n, b.k);
      if (overlaps(g, span(b.out, ext(L, b.n, b.m), b.ld_out, 4)) ||
          overlaps(g, span(b.P, es, b.ld_state, 4)) || overlaps(g, span(b.M, es, b.ld_state, 4)) ||
          overlaps(g, span(b.V, es, b.ld_state, 4)) ||
          overlaps(g, span(b.weight, ext(L, b.n, b.m), b.ld_weight, 2)))
        return ZF_EINVAL;
    }
    h.mats[s] = e->d_mats;
  }
  return ZF_OK;
}

}  // namespace

extern "C" {

zf_status zf_plan_update_handover_deferred(zf_plan* p, const zf_adam_hparams* hp, int64_t step,
                                           const zf_plan* const* earlier, int32_t n_earlier,
                                           float scale, zf_stream stream) {
  if (p == nullptr || !p->can_adam || !p->can_handover || p->has_store) return ZF_EINVAL;
  if (!hparams_ok(hp) || step < 1 || !std::isfinite(scale)) return ZF_EINVAL;
  if (earlier == nullptr || n_earlier < 1) return ZF_EINVAL;
  const bool cm = p->layout == zf::kChannelMajor;
  // row-major: the 16-byte kernel reads the earlier gradients as it reads
  // this step's (16-byte rows, strides within its 32-bit row offsets)
  bool rv = !cm && p->mats[0].rv;
  zf::HistTable h{};
  const zf_status st = gather_earlier(p, earlier, n_earlier, h, rv);
  if (st != ZF_OK) return st;
  const AdamK c = adam_consts(*hp, step);
  const hipStream_t stm = as_stream(stream);
  hipError_t e;
  if (cm) {
    e = zf::launch_cm_handover_deferred(Table{p->d_mats, p->d_off_up, p->nmats}, p->mats[0],
                                        p->blk_up, c, scale, h, stm);
  } else if (rv) {
    e = zf::launch_rv_handover_deferred(Table{p->d_mats, p->d_off_upv, p->nmats}, p->mats[0],
                                        p->blk_upv, c, scale, h, stm);
  } else {
    e = zf::launch_update(Table{p->d_mats, p->d_off_up, p->nmats}, p->mats[0], p->blk_up, c,
                          zf::kInplace, 0, true, false, false, 1.0f, stm);
    if (e == hipSuccess)
      e = zf::launch_rm_handover_deferred(Table{p->d_mats, p->d_off_unp, p->nmats}, p->blk_unp,
                                          scale, h, stm);
  }
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_scatter_weights(zf_plan* p, zf_stream stream) {
  if (p == nullptr || !p->can_scatter) return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_unp, p->nmats};
  const hipError_t e = zf::launch_scatter(t, p->mats[0], p->blk_unp, p->layout, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_update_pending(zf_plan* p, const zf_adam_hparams* hp, int64_t step,
                                 int64_t accum_interval, int64_t pend_step, float pend_scale,
                                 zf_stream stream) {
  if (p == nullptr || !p->can_remap || !p->can_pack || !p->can_pending || p->has_acc1)
    return ZF_EINVAL;
  if (!hparams_ok(hp) || step < 1 || pend_step < 1 || !std::isfinite(pend_scale) ||
      accum_interval < 1)
    return ZF_EINVAL;
  const AdamK c = adam_consts(*hp, step);
  const zf::Pending pd{adam_consts(*hp, pend_step), pend_scale};
  const hipStream_t s = as_stream(stream);
  const Table t{p->d_mats, p->d_off_up, p->nmats};
  const hipError_t e =
      p->layout == zf::kChannelMajor
          ? zf::launch_cm_update(t, p->mats[0], p->blk_up, c, zf::kRemap, 1, true, true, nullptr,
                                 false, 1.0f, s, &pd)
          : zf::launch_update(t, p->mats[0], p->blk_up, c, zf::kRemap, 1, true, true, false, 1.0f,
                              s, &pd);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_scatter_weights_skip_prev(zf_plan* p, zf_stream stream) {
  if (p == nullptr || !p->can_scatter_skip) return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_unp, p->nmats};
  const hipError_t e =
      zf::launch_scatter(t, p->mats[0], p->blk_unp, p->layout, as_stream(stream), true);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

}  // extern "C"

namespace {

// Zen-auto step over a plan; pd != nullptr: the refresh with the owed
// deferred update (kRemap, first step of an interval).
zf_status plan_update_zen(zf_plan* p, const AdamK& c, int32_t mode, int32_t first, double tau,
                          zf_zen_totals* totals, hipStream_t s, const zf::Pending* pd,
                          zf::ZenState* zst = nullptr, int32_t S_max = 1, int32_t force_end = 0) {
  const Table t{p->d_mats, p->d_off_up, p->nmats};
  const Table tz{p->d_mats, p->d_off_zen, p->nmats};
  hipError_t e;
  // force_end 2: the interval ends here and the update writes the hand-over
  // where it can (channel-major; row-major steps in place on the 16-byte
  // update); elsewhere a plain end, the hand-over left to the gated pass
  const bool rv = p->layout == zf::kRowMajor && pd == nullptr && use_rv(p->mats[0], mode, true);
  const bool fuse = force_end == 2 && p->can_handover && zst != nullptr &&
                    (p->layout == zf::kChannelMajor || rv);
  if (force_end == 2 && !fuse) force_end = 1;
  if (p->layout == zf::kChannelMajor) {
    e = zf::launch_cm_update(t, p->mats[0], p->blk_up, c, mode, first, true, true, p->d_zs,
                             fuse, 1.0f, s, pd, zst);
    if (e != hipSuccess) return hip_fail(e);
    e = zf::launch_zen_finalize(tz, p->mats[0], p->blk_zen, p->d_zs, p->d_zb, s);
  } else if (rv) {
    // 16-byte update with the statistics fused: only the finalize remains
    const Table tv{p->d_mats, p->d_off_upv, p->nmats};
    e = zf::launch_rv_update(tv, p->mats[0], p->blk_upv, c, mode, first, true, true, fuse, 1.0f,
                             s, p->d_ws, zst);
    if (e != hipSuccess) return hip_fail(e);
    const Table tp{p->d_mats, p->d_off_zp, p->nmats};
    e = zf::launch_rm_zen(tp, 0, tz, p->blk_zen, p->mats[0], p->d_ws, p->d_zb, s);
  } else {
    // the per-column update (with zst the kernel derives the phase: 1 on a
    // refresh or after an ended interval, else the interval's length + 1)
    e = zf::launch_update(t, p->mats[0], p->blk_up, c, mode, first, true, true, false, 1.0f, s,
                          pd, zst);
    if (e != hipSuccess) return hip_fail(e);
    const Table tp{p->d_mats, p->d_off_zp, p->nmats};
    e = zf::launch_rm_zen(tp, p->blk_zp, tz, p->blk_zen, p->mats[0], p->d_ws, p->d_zb, s);
  }
  if (e != hipSuccess) return hip_fail(e);
  e = zf::launch_zen_total(p->d_zb, p->blk_zen, p->k_total, p->u_total, tau,
                           reinterpret_cast<zf::ZenTotals*>(totals), s, zst,
                           mode != zf::kInplace ? 1 : 0, S_max, force_end);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

bool zen_args_ok(const zf_plan* p, const zf_adam_hparams* hp, int64_t step, double tau,
                 const zf_zen_totals* totals) {
  static_assert(sizeof(zf_zen_totals) == sizeof(zf::ZenTotals), "zen totals layout");
  // (row-major Zen-auto statistics of refresh steps read the packed buffer
  // in a separate pass: no stage there)
  return p != nullptr && p->can_zen && p->can_adam && p->can_pack && hparams_ok(hp) &&
         !(p->has_acc1 && p->layout == zf::kRowMajor) &&
         step >= 1 && tau >= 0.0 && totals != nullptr && aligned(totals, 8);
}

}  // namespace

extern "C" {

zf_status zf_plan_update_zen(zf_plan* p, const zf_adam_hparams* hp, int64_t step, int32_t mode,
                             int64_t step_in_interval, int64_t accum_interval, double tau,
                             zf_zen_totals* totals, zf_stream stream) {
  if (!zen_args_ok(p, hp, step, tau, totals)) return ZF_EINVAL;
  if (mode != zf::kInplace && mode != zf::kRemap && mode != zf::kInit) return ZF_EINVAL;
  if (mode == zf::kRemap && !p->can_remap) return ZF_EINVAL;
  if (accum_interval < 1 || step_in_interval < 1 || step_in_interval > accum_interval)
    return ZF_EINVAL;
  return plan_update_zen(p, adam_consts(*hp, step), mode, pack_phase(p, step_in_interval), tau,
                         totals, as_stream(stream), nullptr);
}

zf_status zf_plan_update_zen_device(zf_plan* p, const zf_adam_hparams* hp, int64_t step,
                                    int32_t mode, int64_t accum_interval, int32_t force_end,
                                    double tau, zf_zen_totals* totals, zf_zen_state* state,
                                    zf_stream stream) {
  static_assert(sizeof(zf_zen_state) == sizeof(zf::ZenState), "zen state layout");
  if (!zen_args_ok(p, hp, step, tau, totals) || p->has_store) return ZF_EINVAL;
  // (row-major: the phase comes from the state, so the bf16 stage, which
  // the row-major kernels select on the host, is not supported)
  if (p->layout == zf::kRowMajor && p->has_acc1) return ZF_EINVAL;
  if (mode != zf::kInplace && mode != zf::kRemap && mode != zf::kInit) return ZF_EINVAL;
  if (mode == zf::kRemap && !p->can_remap) return ZF_EINVAL;
  if (accum_interval < 1 || accum_interval > INT32_MAX || state == nullptr ||
      !aligned(state, 4))
    return ZF_EINVAL;
  // 2: end here with the hand-over fused into the update where the plan can
  if (force_end < 0 || force_end > 2) return ZF_EINVAL;
  return plan_update_zen(p, adam_consts(*hp, step), mode, 0, tau, totals, as_stream(stream),
                         nullptr, reinterpret_cast<zf::ZenState*>(state),
                         static_cast<int32_t>(accum_interval), force_end);
}

zf_status zf_plan_handover_zen(zf_plan* p, const zf_zen_state* state, zf_stream stream) {
  if (p == nullptr || !p->can_unpack || state == nullptr || !aligned(state, 4) ||
      (p->has_acc1 && (!p->all_acc1 || p->layout == zf::kRowMajor)))
    return ZF_EINVAL;
  const Table t{p->d_mats, p->d_off_unp, p->nmats};
  const auto* zst = reinterpret_cast<const zf::ZenState*>(state);
  const hipError_t e =
      p->layout == zf::kChannelMajor
          ? zf::launch_cm_unpack_zen(t, p->mats[0], p->blk_unp, zst, p->all_acc1,
                                     as_stream(stream))
          : zf::launch_unpack_zen(t, p->blk_unp, zst, as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_update_zen_deferred(zf_plan* p, const zf_adam_hparams* hp, int64_t step,
                                      int32_t mode, int64_t accum_interval,
                                      const zf_plan* const* earlier, int32_t n_earlier,
                                      int32_t force_end, double tau, zf_zen_totals* totals,
                                      zf_zen_state* state, zf_stream stream) {
  if (p == nullptr || p->layout != zf::kChannelMajor || !p->can_zen || !p->can_adam ||
      !p->can_handover || p->has_store || !hparams_ok(hp) || step < 1 || !(tau >= 0.0) ||
      totals == nullptr || !aligned(totals, 8))
    return ZF_EINVAL;
  if (mode != zf::kInplace && mode != zf::kRemap && mode != zf::kInit) return ZF_EINVAL;
  if (mode == zf::kRemap && !p->can_remap) return ZF_EINVAL;
  if (accum_interval < 1 || accum_interval > INT32_MAX || state == nullptr ||
      !aligned(state, 4) || force_end < 0 || force_end > 2)
    return ZF_EINVAL;
  zf::HistTable h{};
  bool rv = false;
  const zf_status st = gather_earlier(p, earlier, n_earlier, h, rv);
  if (st != ZF_OK) return st;
  auto* zst = reinterpret_cast<zf::ZenState*>(state);
  const hipStream_t s = as_stream(stream);
  const Table t{p->d_mats, p->d_off_up, p->nmats};
  const Table tz{p->d_mats, p->d_off_zen, p->nmats};
  hipError_t e = zf::launch_cm_update_zen_deferred(t, p->mats[0], p->blk_up,
                                                   adam_consts(*hp, step), mode, p->d_zs,
                                                   force_end == 2, h, zst, s);
  if (e == hipSuccess) e = zf::launch_zen_finalize(tz, p->mats[0], p->blk_zen, p->d_zs, p->d_zb, s);
  if (e == hipSuccess)
    e = zf::launch_zen_total(p->d_zb, p->blk_zen, p->k_total, p->u_total, tau,
                             reinterpret_cast<zf::ZenTotals*>(totals), s, zst,
                             mode != zf::kInplace ? 1 : 0, static_cast<int32_t>(accum_interval),
                             force_end);
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_handover_zen_deferred(zf_plan* p, const zf_plan* const* earlier,
                                        int32_t n_earlier, const zf_zen_state* state,
                                        zf_stream stream) {
  // (the gradient, the selection mask and `unpacked`, as the update it follows)
  if (p == nullptr || p->layout != zf::kChannelMajor || !p->can_adam || !p->can_handover ||
      state == nullptr || !aligned(state, 4))
    return ZF_EINVAL;
  zf::HistTable h{};
  bool rv = false;
  const zf_status st = gather_earlier(p, earlier, n_earlier, h, rv);
  if (st != ZF_OK) return st;
  const hipError_t e = zf::launch_cm_unpack_zen_deferred(
      Table{p->d_mats, p->d_off_unp, p->nmats}, p->blk_unp, h,
      reinterpret_cast<const zf::ZenState*>(state), as_stream(stream));
  return e == hipSuccess ? ZF_OK : hip_fail(e);
}

zf_status zf_plan_update_zen_pending(zf_plan* p, const zf_adam_hparams* hp, int64_t step,
                                     int64_t accum_interval, int64_t pend_step, float pend_scale,
                                     double tau, zf_zen_totals* totals, zf_stream stream) {
  if (!zen_args_ok(p, hp, step, tau, totals) || !p->can_remap || !p->can_pending || p->has_acc1)
    return ZF_EINVAL;
  if (pend_step < 1 || !std::isfinite(pend_scale) || accum_interval < 1) return ZF_EINVAL;
  const zf::Pending pd{adam_consts(*hp, pend_step), pend_scale};
  return plan_update_zen(p, adam_consts(*hp, step), zf::kRemap, 1, tau, totals,
                         as_stream(stream), &pd);
}

}  // extern "C"
