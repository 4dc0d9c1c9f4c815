// Internal types shared by the host entry points and the gfx950 kernels of
// libzf.  Nothing here is part of the public C ABI (include/zf.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

// Channel-major layout: an update block covers one channel and
// cm_vpt * kThreads * 8 of its rows (cm_vpt 16-byte groups per thread, at
// most kCmVpt, chosen per matrix to fill the lanes), an unpack block one
// channel and kCmUnpackChunk rows; a colnorm block covers kThreads / 64
// channels, one per wave.
#ifndef ZF_CM_VPT
#define ZF_CM_VPT 2
#endif
#ifndef ZF_CM_UNPACK_VPT
#define ZF_CM_UNPACK_VPT 1
#endif
constexpr int kCmVpt = ZF_CM_VPT;
constexpr int kCmUnpackVpt = ZF_CM_UNPACK_VPT;
constexpr int kCmUnpackChunk = kThreads * 8 * kCmUnpackVpt;
constexpr int kCmColnormCols = kThreads / 64;

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
  // geometry
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
  int32_t cm_vpt;    // channel-major: 16-byte groups per thread in the update (1 or 2)
  int32_t pad_;
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

// Kernel launchers (zf_kernels.hip).  `blocks` is the grid size.
hipError_t launch_colnorm(const Table& t, const DevMat& one, int64_t blocks,
                          const Table& tf, int64_t fin_blocks, double* ws, hipStream_t s);
hipError_t launch_topk(const Table& t, const DevMat& one, int64_t blocks, hipStream_t s);
hipError_t launch_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                         int32_t mode, int32_t first, bool adam, bool pack, hipStream_t s);
hipError_t launch_unpack(const Table& t, const DevMat& one, int64_t blocks, float scale,
                         hipStream_t s);

// Channel-major kernels (zf_kernels_cm.hip).
hipError_t launch_cm_colnorm(const Table& t, const DevMat& one, int64_t blocks, hipStream_t s);
hipError_t launch_cm_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                            int32_t mode, int32_t first, bool adam, bool pack, hipStream_t s);
hipError_t launch_cm_unpack(const Table& t, const DevMat& one, int64_t blocks, float scale,
                            hipStream_t s);

}  // namespace zf
