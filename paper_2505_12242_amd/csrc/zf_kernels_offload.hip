// gfx950 kernel of the deferred update's write-back: the bf16 weights the
// host optimizer produced for the unselected columns (slot order) are
// scattered into the weight matrix, W[i][unsel_idx[u]] = wcols[i][u];
// selected columns are not touched (the selective optimizer owns them).
// The source may be device memory or pinned host memory that the kernel
// reads in place.  Column -> slot comes from the selection mask and prefix.
// SKIP: columns set in prev_mask (the selection that replaced the one the
// weights were computed under) are left as they are.
#include "zf_device.hpp"

namespace zf {
namespace {

// Channel-major: block = one channel x kCmUnpackChunk of its rows (the
// hand-over's geometry); a selected channel's block exits at once.
template <bool BATCHED, bool SKIP>
__global__ __launch_bounds__(kThreads) void cm_scatter_kernel(const DevMat* __restrict__ mats,
                                                             const int64_t* __restrict__ off,
                                                             int32_t nmats, DevMat one) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int64_t j = local / d.cm_unch;
  const int64_t e0 = (local % d.cm_unch) * kCmUnpackChunk;
  const int64_t len = min(static_cast<int64_t>(kCmUnpackChunk), d.n - e0);
  const int64_t w = j >> 6;
  const uint64_t mw = uniform_u64(d.mask[w]);
  if ((mw >> (j & 63)) & 1ull) return;
  if (SKIP && ((uniform_u64(d.prev_mask[w]) >> (j & 63)) & 1ull)) return;
  const int64_t u = j - (static_cast<int64_t>(uniform_i32(d.prefix[w])) +
                         __popcll(mw & ((uint64_t(1) << (j & 63)) - 1)));
  const uint16_t* __restrict__ src = d.wcols + u * d.ld_wcols + e0;
  uint16_t* __restrict__ dst = d.weight + j * d.ld_weight + e0;
  if (d.scat_vec) {
    const uint4* __restrict__ s4 = reinterpret_cast<const uint4*>(src);
    uint4* __restrict__ d4 = reinterpret_cast<uint4*>(dst);
    for (int64_t g = threadIdx.x; g * 8 < len; g += kThreads) d4[g] = s4[g];
  } else {
    for (int64_t e = threadIdx.x; e < len; e += kThreads) dst[e] = src[e];
  }
}

// Row-major: block = 256 columns (one per thread) x up_rows rows.
template <bool BATCHED, bool SKIP>
__global__ __launch_bounds__(kThreads) void scatter_kernel(const DevMat* __restrict__ mats,
                                                          const int64_t* __restrict__ off,
                                                          int32_t nmats, DevMat one) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int64_t cblk = local % d.up_cb;
  const int64_t rblk = local / d.up_cb;
  const int64_t j = cblk * kUpdateCols + threadIdx.x;
  if (j >= d.m) return;
  const int64_t w = j >> 6;
  const uint64_t mw = d.mask[w];
  if ((mw >> (j & 63)) & 1ull) return;
  if (SKIP && ((d.prev_mask[w] >> (j & 63)) & 1ull)) return;
  const int64_t u = j - (static_cast<int64_t>(d.prefix[w]) +
                         __popcll(mw & ((uint64_t(1) << (j & 63)) - 1)));
  const int64_t i0 = rblk * d.up_rows;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.up_rows), d.n);
  for (int64_t i = i0; i < i1; ++i) d.weight[i * d.ld_weight + j] = d.wcols[i * d.ld_wcols + u];
}

}  // namespace

template <bool SKIP>
static void launch_scatter_t(const Table& t, const DevMat& one, dim3 grid, int32_t layout,
                             hipStream_t s) {
  if (layout == kChannelMajor) {
    if (t.mats != nullptr)
      hipLaunchKernelGGL((cm_scatter_kernel<true, SKIP>), grid, dim3(kThreads), 0, s, t.mats,
                         t.off, t.nmats, one);
    else
      hipLaunchKernelGGL((cm_scatter_kernel<false, SKIP>), grid, dim3(kThreads), 0, s, t.mats,
                         t.off, t.nmats, one);
  } else {
    if (t.mats != nullptr)
      hipLaunchKernelGGL((scatter_kernel<true, SKIP>), grid, dim3(kThreads), 0, s, t.mats, t.off,
                         t.nmats, one);
    else
      hipLaunchKernelGGL((scatter_kernel<false, SKIP>), grid, dim3(kThreads), 0, s, t.mats,
                         t.off, t.nmats, one);
  }
}

hipError_t launch_scatter(const Table& t, const DevMat& one, int64_t blocks, int32_t layout,
                          hipStream_t s, bool skip_prev) {
  (void)hipGetLastError();
  if (blocks <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (skip_prev) launch_scatter_t<true>(t, one, grid, layout, s);
  else launch_scatter_t<false>(t, one, grid, layout, s);
  return hipGetLastError();
}

}  // namespace zf
