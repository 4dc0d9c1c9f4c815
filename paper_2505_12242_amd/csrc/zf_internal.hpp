// Internal types shared by the host entry points and the gfx950 kernels of
// libzf.  Nothing here is part of the public C ABI (include/zf.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zf.h"

namespace zf {

// Tile shapes.  A colnorm block covers 512 columns (64 lanes x 8 bf16 = one
// 16-byte load per lane per row) and cn_rpb rows split over 4 waves.  An
// update / unpack block covers 256 columns (4 waves x 64 lanes, one column
// and one selection-mask word per wave) and up_rows rows.
constexpr int kThreads = 256;
constexpr int kColnormCols = 512;
constexpr int kUpdateCols = 256;
constexpr int kFinalizeCols = 256;
constexpr int kTopkThreads = 1024;

// Row-major update with 16-byte accesses: a block covers rv_w <= kRvMaxCols
// columns (equal-width tiles per matrix, multiples of 8) and rv_rows rows.
constexpr int kRvMaxCols = 1000;

// Channel-major layout: an update block covers one channel and
// cm_qpt * kThreads * 4 of its rows (cm_qpt quads of 4 elements per thread,
// kCmQpt / 2 or kCmQpt, chosen per matrix to fill the lanes); a block of the
// Adam grid over the selected channels alone one channel and kThreads * 4
// rows (one quad per thread; cm_snch chunks per channel); an unpack block one
// channel and kCmUnpackChunk rows; a colnorm block covers kThreads / 64
// channels, one per wave.  Measured on MI355X: the Adam-only pass is fastest
// with one quad per thread, the passes that pack or sum the unselected
// channels (two or three streams of 8 or 16 bytes per quad) need two to four
// quads per thread in flight.
#ifndef ZF_CM_QPT
#define ZF_CM_QPT 4
#endif
#ifndef ZF_CM_UNPACK_QPT
#define ZF_CM_UNPACK_QPT 2
#endif
constexpr int kCmQpt = ZF_CM_QPT;
static_assert(kCmQpt >= 2 && kCmQpt % 2 == 0, "two quad counts per thread: kCmQpt / 2 and kCmQpt");
constexpr int kCmUnpackQpt = ZF_CM_UNPACK_QPT;
constexpr int kCmUnpackChunk = kThreads * 4 * kCmUnpackQpt;
constexpr int kCmSelChunk = kThreads * 4;  // rows per block of the selected-only Adam grid
constexpr int kCmColnormCols = kThreads / 64;
constexpr int kCmWaves = kThreads / 64;  // waves per update block (one statistics partial each)

// Zen-auto: channels per finalize block; threads of the one-block total.
constexpr int kZenCols = 256;
constexpr int kZenTotalThreads = 256;

enum StateMode : int32_t { kInplace = 0, kRemap = 1, kInit = 2 };
enum Layout : int32_t { kRowMajor = 0, kChannelMajor = 1 };

// One matrix as the kernels see it.  Host-computed geometry is appended.
struct DevMat {
  int64_t n, m, k;
  const uint16_t* grad;
  int64_t ld_grad;
  uint16_t* weight;
  int64_t ld_weight;
  float* P;
  float* M;
  float* V;
  int64_t ld_state;
  float* acc;
  int64_t ld_acc;
  float* norms;
  int32_t* sel_idx;
  int32_t* unsel_idx;
  uint64_t* mask;
  int32_t* prefix;
  float* out;
  int64_t ld_out;
  const uint64_t* prev_mask;
  const int32_t* prev_prefix;
  const float* prev_P;
  const float* prev_M;
  const float* prev_V;
  int64_t ld_prev;
  const float* init_P;
  int64_t ld_init;
  float* st_P;       // full-state store (swap in / out), n x m in the layout
  float* st_M;
  float* st_V;
  int64_t ld_store;
  const uint16_t* wcols;  // deferred update: bf16 weights of the unselected columns (slot order)
  int64_t ld_wcols;
  const float* pend_acc;  // owed deferred update: packed sums under the previous selection
  int64_t ld_pend;
  uint16_t* acc1;    // bf16 first-step stage of the packed buffer, in the gradient's shape
                     // (channel-major row j = channel j; row-major [n][ld >= m]) (optional)
  int64_t ld_acc1;
  float* sel_sq;     // Zen-auto: [k] squared norms of the selected channels' gradient
  float* acc_sq;     // Zen-auto: [m-k] squared norms of the accumulated channels
  // geometry
  int64_t zs_off;    // offset (in doubles) of this matrix's Zen-auto partials
  int64_t cn_ws;     // offset (in doubles) of this matrix's colnorm partials
  int32_t cn_rpb;    // rows per colnorm block
  int32_t cn_rb;     // colnorm row blocks (0 when n == 0)
  int32_t cn_cb;     // colnorm column blocks
  int32_t up_rows;   // rows per update / unpack block
  int32_t up_rb;     // update row blocks
  int32_t up_cb;     // update column blocks
  int32_t vec;       // 16-byte vector path allowed (alignment, strides, sizes)
  int32_t layout;    // Layout
  int32_t cm_nch;    // channel-major: row chunks per channel (update)
  int32_t cm_unch;   // channel-major: row chunks per channel (unpack)
  int32_t cm_qpt;    // channel-major: quads (4 elements) per thread in the update (kCmQpt / 2 or kCmQpt)
  int32_t cm_snch;   // channel-major: row chunks per channel of the selected-only Adam grid
  int32_t scat_vec;  // channel-major: 16-byte path of the weight scatter
  int32_t rv;        // row-major: the 16-byte update kernel is used (else per-column)
  int32_t rv_w;      // row-major 16-byte update: tile width (columns)
  int32_t rv_cb;     // row-major 16-byte update: column tiles
  int32_t rv_rows;   // row-major 16-byte update: rows per block
};

// Per-kernel view of a batch: a device array of matrices and the first
// block of each matrix in this kernel's grid (off[nmats] = grid size).
// mats == nullptr means a single matrix passed by value.
struct Table {
  const DevMat* mats;
  const int64_t* off;
  int32_t nmats;
};

// Adam constants for one step, fp32 (computed in double on the host).
struct AdamK {
  float b1, b2, c1, c2, lr, eps, wd, ib1, ib2;
};

// The deferred update that the full-state store still owes the columns
// entering the selection at a refresh: each first takes gradient
// scale * (its packed sum under the previous selection) with constants c.
struct Pending {
  AdamK c;
  float scale;
};

// Deferred packing: the device tables of the plans of an interval's earlier
// steps (the same matrices; their descriptors' grad = that step's gradient).
constexpr int kMaxDeferred = 15;
struct HistTable {
  const DevMat* mats[kMaxDeferred];
  int32_t n;
};

// Zen-auto's interval state when the device drives the interval
// (zf_zen_state): steps of the current interval so far, and whether the
// last step ended it.
struct ZenState {
  int32_t length;
  int32_t ended;
};

// Hyperparameter validation and the constants of a 1-based step
// (zf_api.hip): B1 = beta1, C1 = 1 - beta1, B2 = beta2, C2 = 1 - beta2,
// LR = lr, EPS = eps, WD = lr * weight_decay, IB1 = 1 / (1 - beta1^t),
// IB2 = 1 / (1 - beta2^t), each computed in double and rounded once.
bool hparams_ok(const zf_adam_hparams* hp);
AdamK adam_consts(const zf_adam_hparams& hp, int64_t step);

// Kernel launchers (zf_kernels.hip).  `blocks` is the grid size.
// stage: also copy every element read to the same place of acc1 (the
// bf16 first-step stage; row-major plans that have one).
hipError_t launch_colnorm(const Table& t, const DevMat& one, int64_t blocks,
                          const Table& tf, int64_t fin_blocks, double* ws, hipStream_t s,
                          bool stage = false);
hipError_t launch_topk(const Table& t, const DevMat& one, int64_t blocks, hipStream_t s);
// pend != nullptr: fused Adam + pack in kRemap against the store, with the
// owed deferred update applied to the entering columns first.
// zst (Zen-auto with the interval driven on the device; packing passes
// only): an in-place step takes its phase from the interval state
hipError_t launch_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                         int32_t mode, int32_t first, bool adam, bool pack, bool handover,
                         float scale, hipStream_t s, const Pending* pend = nullptr,
                         const ZenState* zst = nullptr);
hipError_t launch_unpack(const Table& t, const DevMat& one, int64_t blocks, float scale,
                         hipStream_t s);
// The hand-over of an interval Zen-auto ended on the device (row-major):
// nothing unless zst->ended; `units` = the table's unpack blocks.
hipError_t launch_unpack_zen(const Table& t, int64_t units, const ZenState* zst, hipStream_t s);

// Row-major update with 16-byte accesses (zf_kernels_rv.hip); same contract
// as launch_update, geometry rv_w / rv_cb / rv_rows.  zs != nullptr (fused
// update only, rv_rows == cn_rpb): also the Zen-auto partials of the
// row-major statistics pass, into zs at each matrix's cn_ws.
hipError_t launch_rv_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                            int32_t mode, int32_t first, bool adam, bool pack, bool handover,
                            float scale, hipStream_t s, double* zs = nullptr,
                            const ZenState* zst = nullptr);
// Deferred packing, row-major, the interval's last step (states in place):
// Adam on the selected columns and the hand-over of the unselected ones,
// g_1 + ... + g_t summed in step order from h's plans (the earlier steps)
// and this plan (step t), times scale.  The 16-byte kernel over the plan's
// 16-byte update grid, as two passes (Adam-only, then the hand-over) ...
hipError_t launch_rv_handover_deferred(const Table& t, const DevMat& one, int64_t blocks,
                                       const AdamK& c, float scale, const HistTable& h,
                                       hipStream_t s);
// ... or, off the 16-byte path, the hand-over alone over the unpack grid
// (Adam then runs as the per-column update's Adam-only pass).
hipError_t launch_rm_handover_deferred(const Table& t, int64_t blocks, float scale,
                                       const HistTable& h, hipStream_t s);

// Channel-major kernels (zf_kernels_cm.hip).
// out == 1: also copy every channel's gradient row to its row of acc1 (the
// bf16 first-step stage), for matrices that have one; out == 2: also write
// scale * every channel's widened gradient row to its row of `out` (the
// hand-over of a one-step interval).
hipError_t launch_cm_colnorm(const Table& t, const DevMat& one, int64_t blocks, hipStream_t s,
                             int32_t out = 0, float scale = 1.0f);
// zs != nullptr: fused Adam + pack that also writes the Zen-auto partials.
// handover: the last step of an interval with the hand-over fused in (the
// `out` buffer receives scale * the final sums, +0.0 for selected columns;
// the packed buffer is not written).
// pend: as in launch_update (also with zs).
hipError_t launch_cm_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                            int32_t mode, int32_t first, bool adam, bool pack, double* zs,
                            bool handover, float scale, hipStream_t s,
                            const Pending* pend = nullptr, const ZenState* zst = nullptr);
// The hand-over of an interval that Zen-auto ended on the device: when
// zst->ended, every matrix's `out` receives scale * its sums with scale =
// fp32(1 / zst->length) (from the stage when stage and the interval was one
// step), +0.0 for selected channels; else nothing.  A grid of at most
// `grid` blocks loops over the `units` unpack blocks of the table.
hipError_t launch_cm_unpack_zen(const Table& t, const DevMat& one, int64_t units,
                                const ZenState* zst, bool stage, hipStream_t s);
// The last step of an interval with deferred packing (batched plans only):
// Adam on the selected channels (states in place) and +0.0 in their rows of
// `out`; at the unselected channels out = scale * (((g_1 + g_2) + ...) + g),
// g_s the channel's row of the gradient of earlier step s (h.mats[s - 1]),
// g this step's.
hipError_t launch_cm_handover_deferred(const Table& t, const DevMat& one, int64_t blocks,
                                       const AdamK& c, float scale, const HistTable& h,
                                       hipStream_t s);
// Zen-auto on the device with deferred packing (channel-major): the update
// with the statistics of the interval's running sum taken from the kept
// gradients (the last position - 1 entries of h); handover: an end the
// caller forces, scale times that sum written to the hand-over.
hipError_t launch_cm_update_zen_deferred(const Table& t, const DevMat& one, int64_t blocks,
                                         const AdamK& c, int32_t mode, double* zs, bool handover,
                                         const HistTable& h, const ZenState* zst, hipStream_t s);
// Its gated hand-over (ended == 1): the interval's sums from the kept
// gradients and the plan's own (unpack table and units).
hipError_t launch_cm_unpack_zen_deferred(const Table& t, int64_t units, const HistTable& h,
                                         const ZenState* zst, hipStream_t s);
// from_stage: the source is the bf16 first-step stage (a one-step interval;
// every matrix of the table has one).
hipError_t launch_cm_unpack(const Table& t, const DevMat& one, int64_t blocks, float scale,
                            hipStream_t s, bool from_stage = false);
// Adam only over a grid of the selected channels alone (cm_snch blocks per
// selected channel; table offsets over sum(k * cm_snch)); for plans without
// a full-state store (nothing to do for the unselected channels).
// zero_out: also +0.0 into the selected channels' rows of `out` (after the
// score pass wrote the hand-over of a one-step interval).
hipError_t launch_cm_adam_selected_grid(const Table& t, const DevMat& one, int64_t blocks,
                                        const AdamK& c, int32_t mode, hipStream_t s,
                                        bool zero_out = false);

// Deferred update write-back (zf_kernels_offload.hip): W[:, unsel[u]] =
// wcols[:, u] in either layout (grid: unpack geometry); skip_prev: columns
// set in prev_mask are left untouched.
hipError_t launch_scatter(const Table& t, const DevMat& one, int64_t blocks, int32_t layout,
                          hipStream_t s, bool skip_prev = false);

// Zen-auto reductions (zf_kernels_zen.hip).  Totals as written to device
// memory; the layout equals the public zf_zen_totals.
struct ZenTotals {
  double sum_sel;
  double sum_acc;
  int64_t k_total;
  int64_t u_total;
  int32_t trigger;
  int32_t pad_;
};

// Per-channel statistics from the partials zs, and two fp64 partial sums
// (selected, accumulated) per finalize block into zb[2 * blocks].
hipError_t launch_zen_finalize(const Table& t, const DevMat& one, int64_t blocks,
                               const double* zs, double* zb, hipStream_t s);
// Row-major statistics pass (after the update; batched tables only):
// per-column partials over the column-score row blocks into zs (the plan's
// column-score workspace), then the row-major finalize into zb.
hipError_t launch_rm_zen(const Table& tp, int64_t partial_blocks, const Table& tf,
                         int64_t finalize_blocks, const DevMat& one, double* zs, double* zb,
                         hipStream_t s);
// One block: sums zb in a fixed order and evaluates the trigger.
// Streaming reference passes (zf_measure.h): kind 0 read, 1 copy, 2
// read-modify-write in place.
int64_t stream_probe_blocks(int64_t bytes);
hipError_t launch_stream_probe(int32_t kind, const void* src, void* dst, int64_t bytes,
                               uint32_t key, hipStream_t s);

// zst != nullptr (the interval driven on the device): the step's position
// is 1 after a refresh or an ended interval, else zst->length + 1; the
// kernel stores it in zst->length and ends the interval when the trigger
// fires, the position reaches S_max, or force_end.
hipError_t launch_zen_total(const double* zb, int64_t blocks, int64_t k_total, int64_t u_total,
                            double tau, ZenTotals* out, hipStream_t s, ZenState* zst = nullptr,
                            int32_t refresh = 0, int32_t S_max = 1, int32_t force_end = 0);

}  // namespace zf
