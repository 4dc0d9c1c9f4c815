// gfx950 reductions of Zen-auto, the adaptive accumulation interval (paper,
// Zero-stall Pipeline, "Hyperparameter Auto-tuning"): the unimportant part's
// mean accumulated channel norm is compared with the important part's mean
// channel norm, and the deferred update is triggered once the first becomes
// comparable to the second.
//
// The fused update pass (channel-major, STATS) leaves one fp64 partial sum of
// squares per wave: kCmWaves partials per chunk of a channel's rows.  Here
//   finalize: per channel, the partials are added in (chunk, wave) order and
//             rounded once to fp32 -- the channel's squared norm, written in
//             slot order to sel_sq (selected) or acc_sq (accumulated); the
//             fp64 square roots of those fp32 values are summed per block in
//             a fixed tree, separately for the two parts;
//   total:    one block adds the block sums in a fixed order and evaluates
//             sum_acc * k >= (tau * sum_sel) * u in fp64 (the pooled means
//             sum_acc / u and sum_sel / k compared without a division).
// Every order is fixed, so results are deterministic.
//
// Row-major layout: the update's tiles (256 columns x a few rows) leave no
// per-column partial without atomics, so the statistics come from a
// separate pass after the update: virtual column c < k is the selected
// gradient column sel_idx[c], c >= k the packed column u = c - k of the
// accumulated buffer; a block sums the squares of 256 virtual columns over
// one row block (the column-score row blocks) in fp64 and stores one
// partial per column and row block in the plan's column-score workspace;
// the row-major finalize adds them in row-block order.
#include "zf_device.hpp"

namespace zf {
namespace {

template <bool BATCHED>
__global__ __launch_bounds__(kZenCols) void zen_finalize_kernel(const DevMat* __restrict__ mats,
                                                               const int64_t* __restrict__ off,
                                                               int32_t nmats, DevMat one,
                                                               const double* __restrict__ zs,
                                                               double* __restrict__ zb) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  const int tid = threadIdx.x;
  const int64_t j = local * kZenCols + tid;
  double root_sel = 0.0, root_acc = 0.0;
  if (j < d.m) {
    const int64_t cnt = static_cast<int64_t>(d.cm_nch) * kCmWaves;
    const double* __restrict__ p = zs + d.zs_off + j * cnt;
    double s = 0.0;
    for (int64_t i = 0; i < cnt; ++i) s += p[i];
    const float f = static_cast<float>(s);
    const double root = sqrt(static_cast<double>(f));
    const int64_t w = j >> 6;
    const uint64_t mw = d.mask[w];
    const int64_t r = static_cast<int64_t>(d.prefix[w]) +
                      __popcll(mw & ((uint64_t(1) << (j & 63)) - 1));
    if ((mw >> (j & 63)) & 1ull) {
      d.sel_sq[r] = f;
      root_sel = root;
    } else {
      d.acc_sq[j - r] = f;
      root_acc = root;
    }
  }
  __shared__ double red[2][kZenCols];
  red[0][tid] = root_sel;
  red[1][tid] = root_acc;
  __syncthreads();
#pragma unroll
  for (int h = kZenCols / 2; h >= 1; h >>= 1) {
    if (tid < h) {
      red[0][tid] += red[0][tid + h];
      red[1][tid] += red[1][tid + h];
    }
    __syncthreads();
  }
  if (tid == 0) {
    zb[2 * b] = red[0][0];
    zb[2 * b + 1] = red[1][0];
  }
}

template <bool BATCHED>
__global__ __launch_bounds__(kZenCols) void rm_zen_partial_kernel(const DevMat* __restrict__ mats,
                                                                 const int64_t* __restrict__ off,
                                                                 int32_t nmats, DevMat one,
                                                                 double* __restrict__ zs) {
  int64_t local;
  const DevMat& d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int64_t cb = (d.m + kZenCols - 1) / kZenCols;
  const int64_t rblk = local / cb;
  const int64_t c = (local % cb) * kZenCols + threadIdx.x;
  if (c >= d.m) return;
  const int64_t i0 = rblk * d.cn_rpb;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.cn_rpb), d.n);
  double s = 0.0;
  if (c < d.k) {
    const uint16_t* __restrict__ g = d.grad + d.sel_idx[c];
    for (int64_t i = i0; i < i1; ++i) {
      const double x = static_cast<double>(widen_bf16(g[i * d.ld_grad]));
      s = __builtin_fma(x, x, s);
    }
  } else {
    const float* __restrict__ a = d.acc + (c - d.k);
    for (int64_t i = i0; i < i1; ++i) {
      const double x = static_cast<double>(a[i * d.ld_acc]);
      s = __builtin_fma(x, x, s);
    }
  }
  zs[d.cn_ws + rblk * d.m + c] = s;
}

template <bool BATCHED>
__global__ __launch_bounds__(kZenCols) void rm_zen_finalize_kernel(
    const DevMat* __restrict__ mats, const int64_t* __restrict__ off, int32_t nmats, DevMat one,
    const double* __restrict__ zs, double* __restrict__ zb) {
  int64_t local;
  const DevMat& d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  const int tid = threadIdx.x;
  const int64_t c = local * kZenCols + tid;
  double root_sel = 0.0, root_acc = 0.0;
  if (c < d.m) {
    double s = 0.0;
    for (int32_t rb = 0; rb < d.cn_rb; ++rb) s += zs[d.cn_ws + static_cast<int64_t>(rb) * d.m + c];
    const float f = static_cast<float>(s);
    const double root = sqrt(static_cast<double>(f));
    if (c < d.k) {
      d.sel_sq[c] = f;
      root_sel = root;
    } else {
      d.acc_sq[c - d.k] = f;
      root_acc = root;
    }
  }
  __shared__ double red[2][kZenCols];
  red[0][tid] = root_sel;
  red[1][tid] = root_acc;
  __syncthreads();
#pragma unroll
  for (int h = kZenCols / 2; h >= 1; h >>= 1) {
    if (tid < h) {
      red[0][tid] += red[0][tid + h];
      red[1][tid] += red[1][tid + h];
    }
    __syncthreads();
  }
  if (tid == 0) {
    zb[2 * b] = red[0][0];
    zb[2 * b + 1] = red[1][0];
  }
}

__global__ __launch_bounds__(kZenTotalThreads) void zen_total_kernel(const double* __restrict__ zb,
                                                                    int64_t blocks,
                                                                    int64_t k_total,
                                                                    int64_t u_total, double tau,
                                                                    ZenTotals* __restrict__ out,
                                                                    ZenState* __restrict__ zst,
                                                                    int32_t refresh, int32_t S_max,
                                                                    int32_t force_end) {
  const int tid = threadIdx.x;
  double a = 0.0, c = 0.0;
  for (int64_t i = tid; i < blocks; i += kZenTotalThreads) {
    a += zb[2 * i];
    c += zb[2 * i + 1];
  }
  __shared__ double red[2][kZenTotalThreads];
  red[0][tid] = a;
  red[1][tid] = c;
  __syncthreads();
#pragma unroll
  for (int h = kZenTotalThreads / 2; h >= 1; h >>= 1) {
    if (tid < h) {
      red[0][tid] += red[0][tid + h];
      red[1][tid] += red[1][tid + h];
    }
    __syncthreads();
  }
  if (tid == 0) {
    const double sum_sel = red[0][0];
    const double sum_acc = red[1][0];
    const double lhs = sum_acc * static_cast<double>(k_total);
    const double rhs = (tau * sum_sel) * static_cast<double>(u_total);
    out->sum_sel = sum_sel;
    out->sum_acc = sum_acc;
    out->k_total = k_total;
    out->u_total = u_total;
    const int32_t trigger = (k_total > 0 && u_total > 0 && lhs >= rhs) ? 1 : 0;
    out->trigger = trigger;
    out->pad_ = 0;
    if (zst != nullptr) {
      // the position the update of this step took (it read the same state)
      const int32_t pos = (refresh || zst->ended) ? 1 : zst->length + 1;
      zst->length = pos;
      // 2: the update of this step already wrote the hand-over (fused);
      // 1: the interval ended and waits for the hand-over pass
      zst->ended = force_end == 2 ? 2 : (trigger || pos >= S_max || force_end) ? 1 : 0;
    }
  }
}

}  // namespace

hipError_t launch_zen_finalize(const Table& t, const DevMat& one, int64_t blocks,
                               const double* zs, double* zb, hipStream_t s) {
  (void)hipGetLastError();
  if (blocks > 0) {
    if (t.mats != nullptr)
      hipLaunchKernelGGL((zen_finalize_kernel<true>), dim3(static_cast<uint32_t>(blocks)),
                         dim3(kZenCols), 0, s, t.mats, t.off, t.nmats, one, zs, zb);
    else
      hipLaunchKernelGGL((zen_finalize_kernel<false>), dim3(static_cast<uint32_t>(blocks)),
                         dim3(kZenCols), 0, s, t.mats, t.off, t.nmats, one, zs, zb);
  }
  return hipGetLastError();
}

hipError_t launch_rm_zen(const Table& tp, int64_t partial_blocks, const Table& tf,
                         int64_t finalize_blocks, const DevMat& one, double* zs, double* zb,
                         hipStream_t s) {
  (void)hipGetLastError();
  if (partial_blocks > 0)
    hipLaunchKernelGGL((rm_zen_partial_kernel<true>), dim3(static_cast<uint32_t>(partial_blocks)),
                       dim3(kZenCols), 0, s, tp.mats, tp.off, tp.nmats, one, zs);
  if (finalize_blocks > 0)
    hipLaunchKernelGGL((rm_zen_finalize_kernel<true>),
                       dim3(static_cast<uint32_t>(finalize_blocks)), dim3(kZenCols), 0, s, tf.mats,
                       tf.off, tf.nmats, one, zs, zb);
  return hipGetLastError();
}

hipError_t launch_zen_total(const double* zb, int64_t blocks, int64_t k_total, int64_t u_total,
                            double tau, ZenTotals* out, hipStream_t s, ZenState* zst,
                            int32_t refresh, int32_t S_max, int32_t force_end) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(zen_total_kernel, dim3(1), dim3(kZenTotalThreads), 0, s, zb, blocks,
                     k_total, u_total, tau, out, zst, refresh, S_max, force_end);
  return hipGetLastError();
}

}  // namespace zf
