// gfx950 kernels of the selective-update hot path.
//
// All kernels are bandwidth-bound streaming passes (no contraction, so no
// MFMA).  Every kernel reads its matrix descriptor from a batch table (one
// grid over many matrices; block -> matrix by binary search over the
// per-kernel block offsets) or from a single descriptor passed by value.
//
// Compiled with -ffp-contract=off and correctly rounded fp32 division and
// square root, so that each arithmetic line below is one IEEE operation.
#include "zf_internal.hpp"

namespace zf {
namespace {

__device__ __forceinline__ float widen_bf16(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest, ties to even; NaN stays a (quiet) NaN.
__device__ __forceinline__ uint16_t round_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Number of set bits of `mask` at lane positions below the calling lane.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

__device__ __forceinline__ DevMat get_mat(const Table& t, const DevMat& one, int64_t b,
                                          int64_t& local) {
  if (t.mats == nullptr) {
    local = b;
    return one;
  }
  int lo = 0, hi = t.nmats - 1;
  while (lo < hi) {  // largest q with off[q] <= b
    const int mid = (lo + hi + 1) >> 1;
    if (t.off[mid] <= b) lo = mid; else hi = mid - 1;
  }
  local = b - t.off[lo];
  return t.mats[lo];
}

// ---------------------------------------------------------------------------
// a1: column scores.  Stage 1: a block sums the squares of a 512-column x
// cn_rpb-row tile in fp64 (squares of bf16 values are exact), each lane
// owning 8 adjacent columns and reading them with one 16-byte load per row;
// the four waves take interleaved rows and are combined in LDS in fixed
// order.  Stage 2 adds the row-block partials of each column in order and
// rounds once to fp32.  No atomics: the result is deterministic.
// ---------------------------------------------------------------------------

__device__ __forceinline__ void accum8(double (&acc)[8], uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const double lo = static_cast<double>(__uint_as_float(w[h] << 16));
    const double hi = static_cast<double>(__uint_as_float(w[h] & 0xffff0000u));
    acc[2 * h] = __builtin_fma(lo, lo, acc[2 * h]);
    acc[2 * h + 1] = __builtin_fma(hi, hi, acc[2 * h + 1]);
  }
}

__global__ __launch_bounds__(kThreads) void colnorm_partial_kernel(Table t, DevMat one,
                                                                   double* __restrict__ ws) {
  int64_t local;
  const DevMat d = get_mat(t, one, blockIdx.x, local);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t cblk = local % d.cn_cb;
  const int64_t rblk = local / d.cn_cb;
  const int64_t c0 = cblk * kColnormCols + lane * 8;
  const int64_t r0 = rblk * d.cn_rpb;
  const int64_t r1 = min(r0 + static_cast<int64_t>(d.cn_rpb), d.n);

  double acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = 0.0;

  if (c0 < d.m) {
    const uint16_t* __restrict__ base = d.grad + c0;
    const int64_t ld = d.ld_grad;
    if (d.vec && c0 + 8 <= d.m) {
      int64_t i = r0 + wave;
      for (; i + 12 < r1; i += 16) {
        const uint4 v0 = *reinterpret_cast<const uint4*>(base + i * ld);
        const uint4 v1 = *reinterpret_cast<const uint4*>(base + (i + 4) * ld);
        const uint4 v2 = *reinterpret_cast<const uint4*>(base + (i + 8) * ld);
        const uint4 v3 = *reinterpret_cast<const uint4*>(base + (i + 12) * ld);
        accum8(acc, v0);
        accum8(acc, v1);
        accum8(acc, v2);
        accum8(acc, v3);
      }
      for (; i < r1; i += 4) accum8(acc, *reinterpret_cast<const uint4*>(base + i * ld));
    } else {
      const int64_t nc = min(static_cast<int64_t>(8), d.m - c0);
      for (int64_t i = r0 + wave; i < r1; i += 4) {
        const uint16_t* row = base + i * ld;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          if (c < nc) {
            const double x = static_cast<double>(widen_bf16(row[c]));
            acc[c] = __builtin_fma(x, x, acc[c]);
          }
        }
      }
    }
  }

  __shared__ double red[4][kColnormCols];
#pragma unroll
  for (int c = 0; c < 8; ++c) red[wave][lane * 8 + c] = acc[c];
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int col = threadIdx.x + h * kThreads;
    const int64_t j = cblk * kColnormCols + col;
    if (j < d.m) {
      const double s = ((red[0][col] + red[1][col]) + red[2][col]) + red[3][col];
      ws[d.cn_ws + rblk * d.m + j] = s;
    }
  }
}

__global__ __launch_bounds__(kFinalizeCols) void colnorm_finalize_kernel(
    Table t, DevMat one, const double* __restrict__ ws) {
  int64_t local;
  const DevMat d = get_mat(t, one, blockIdx.x, local);
  const int64_t j = local * kFinalizeCols + threadIdx.x;
  if (j >= d.m) return;
  double s = 0.0;
  const double* p = ws + d.cn_ws + j;
  for (int32_t r = 0; r < d.cn_rb; ++r) s += p[static_cast<int64_t>(r) * d.m];
  d.norms[j] = static_cast<float>(s);
}

// ---------------------------------------------------------------------------
// a2: selection.  One 1024-thread block per matrix.  Scores are mapped to
// unsigned keys that order like the float values (with -0.0 == +0.0); an
// MSB-first 8-bit radix select finds the k-th largest key T and how many
// keys equal to T are taken; a compaction pass in ascending column order
// then emits sel / unsel, the 64-bit mask words (one wave ballot each) and
// their prefix counts.  Among keys equal to T the lowest columns win.
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u << 1) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Block-wide exclusive count of `flag` over the 16 waves of a topk block.
// Returns the count before this thread; *total receives the block total,
// *wave_before the count of the waves before this one, *ballot the wave's
// ballot.  Contains two barriers.
__device__ __forceinline__ uint32_t block_excl_count(bool flag, uint32_t* sh_wave,
                                                     uint32_t* total, uint32_t* wave_before,
                                                     uint64_t* ballot) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint64_t b = __ballot(flag);
  if (lane == 0) sh_wave[wave] = static_cast<uint32_t>(__popcll(b));
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kTopkThreads / 64; ++w) {
    const uint32_t c = sh_wave[w];
    before += (w < wave) ? c : 0u;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  *wave_before = before;
  *ballot = b;
  return before + lanes_below(b);
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(Table t, DevMat one) {
  int64_t local;
  const DevMat d = get_mat(t, one, blockIdx.x, local);
  const int64_t m = d.m;
  const int64_t k = d.k;
  if (m == 0) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const float* __restrict__ s = d.norms;

  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_wave[kTopkThreads / 64];
  __shared__ uint32_t sh_digit, sh_above;

  uint32_t thr, need;
  if (k == 0) {
    thr = 0xffffffffu;
    need = 0u;
  } else if (k == m) {
    thr = 0u;
    need = static_cast<uint32_t>(m);
  } else {
    uint32_t prefix = 0u, pmask = 0u, rem = static_cast<uint32_t>(k);
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) hist[tid] = 0u;
      if (tid == 0) {
        sh_digit = 0u;
        sh_above = 0u;
      }
      __syncthreads();
      for (int64_t j = tid; j < m; j += kTopkThreads) {
        const uint32_t key = order_key(s[j]);
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (wave == 0) {
        // lane l holds bins 255-4l .. 252-4l (descending digit order)
        uint32_t h[4], tot = 0u;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          h[c] = hist[255 - 4 * lane - c];
          tot += h[c];
        }
        uint32_t incl = tot;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const uint32_t v = __shfl_up(incl, off, 64);
          if (lane >= off) incl += v;
        }
        const uint32_t excl = incl - tot;
        if (excl < rem && rem <= incl) {
          uint32_t run = excl;
          for (int c = 0; c < 4; ++c) {
            if (run + h[c] >= rem) {
              sh_digit = static_cast<uint32_t>(255 - 4 * lane - c);
              sh_above = run;
              break;
            }
            run += h[c];
          }
        }
      }
      __syncthreads();
      const uint32_t digit = sh_digit;
      rem -= sh_above;
      prefix |= digit << shift;
      pmask |= 255u << shift;
      __syncthreads();
    }
    thr = prefix;
    need = rem;
  }

  const int64_t words = (m + 63) >> 6;
  uint32_t carry_sel = 0u, carry_eq = 0u;
  for (int64_t base = 0; base < m; base += kTopkThreads) {
    const int64_t j = base + tid;
    const bool valid = j < m;
    const uint32_t key = valid ? order_key(s[j]) : 0u;
    const bool gt = valid && key > thr;
    const bool eq = valid && key == thr;
    uint32_t eq_total, eq_wave_before, sel_total, sel_wave_before;
    uint64_t eq_ballot, sel_ballot;
    const uint32_t eq_rank =
        carry_eq + block_excl_count(eq, sh_wave, &eq_total, &eq_wave_before, &eq_ballot);
    const bool take = gt || (eq && eq_rank < need);
    const uint32_t sel_rank =
        carry_sel + block_excl_count(take, sh_wave, &sel_total, &sel_wave_before, &sel_ballot);
    // The ranks are in range whenever the select above is right; the guards
    // keep a wrong count from ever writing outside the outputs.
    if (valid) {
      if (take) {
        if (sel_rank < static_cast<uint32_t>(k)) d.sel_idx[sel_rank] = static_cast<int32_t>(j);
      } else if (j - sel_rank < m - k) {
        d.unsel_idx[j - sel_rank] = static_cast<int32_t>(j);
      }
    }
    const int64_t w = (base >> 6) + wave;
    if (lane == 0 && w < words) {
      d.mask[w] = sel_ballot;
      d.prefix[w] = static_cast<int32_t>(carry_sel + sel_wave_before);
    }
    carry_sel += sel_total;
    carry_eq += eq_total;
  }
}

// ---------------------------------------------------------------------------
// a3-a5: selective Adam with bf16 write-back, and packing of the unselected
// columns, in one pass over G.  Wave w of a block owns the 64 columns of
// selection-mask word `word`; lane l owns column 64*word + l, so its slot in
// the compact states is prefix[word] + (selected lanes below l) and its slot
// in the accumulation buffer is column - that.  Consecutive lanes therefore
// touch consecutive slots: coalesced state and accumulator traffic.  Rows
// are processed four at a time to keep loads in flight.
// ---------------------------------------------------------------------------

__device__ __forceinline__ void adam_step(float g, float& p, float& m, float& v, const AdamK& c) {
  m = c.b1 * m + c.c1 * g;
  v = c.b2 * v + c.c2 * (g * g);
  const float den = sqrtf(v * c.ib2) + c.eps;
  const float u = (m * c.ib1) / den;
  if (c.wd != 0.0f) p = p - c.wd * p;
  p = p - c.lr * u;
}

constexpr int kRowBatch = 4;

template <bool ADAM, bool PACK>
__global__ __launch_bounds__(kThreads) void update_kernel(Table t, DevMat one, AdamK c,
                                                          int32_t mode, int32_t first) {
  int64_t local;
  const DevMat d = get_mat(t, one, blockIdx.x, local);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t cblk = local % d.up_cb;
  const int64_t rblk = local / d.up_cb;
  const int64_t word = cblk * (kUpdateCols / 64) + wave;
  const int64_t j = word * 64 + lane;
  if (j >= d.m) return;

  const uint64_t mw = d.mask[word];
  const bool sel = (mw >> lane) & 1ull;
  const int64_t r = static_cast<int64_t>(d.prefix[word]) + lanes_below(mw);
  const int64_t u = j - r;
  bool was = false;
  int64_t ro = 0;
  if (ADAM && mode == kRemap) {
    const uint64_t pm = d.prev_mask[word];
    was = (pm >> lane) & 1ull;
    ro = static_cast<int64_t>(d.prev_prefix[word]) + lanes_below(pm);
  }
  const bool do_adam = ADAM && sel;
  const bool do_pack = PACK && !sel;
  if (!do_adam && !do_pack) return;

  const int64_t i0 = rblk * d.up_rows;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.up_rows), d.n);
  const uint16_t* __restrict__ G = d.grad;

  for (int64_t i = i0; i < i1; i += kRowBatch) {
    float g[kRowBatch];
#pragma unroll
    for (int b = 0; b < kRowBatch; ++b)
      g[b] = (i + b < i1) ? widen_bf16(G[(i + b) * d.ld_grad + j]) : 0.0f;

    if (do_adam) {
      float p[kRowBatch], mm[kRowBatch], vv[kRowBatch];
#pragma unroll
      for (int b = 0; b < kRowBatch; ++b) {
        if (i + b >= i1) continue;
        const int64_t row = i + b;
        if (mode == kInplace) {
          const int64_t o = row * d.ld_state + r;
          p[b] = d.P[o];
          mm[b] = d.M[o];
          vv[b] = d.V[o];
        } else if (mode == kRemap && was) {
          const int64_t o = row * d.ld_prev + ro;
          p[b] = d.prev_P[o];
          mm[b] = d.prev_M[o];
          vv[b] = d.prev_V[o];
        } else {
          p[b] = d.init_P ? d.init_P[row * d.ld_init + j]
                          : widen_bf16(d.weight[row * d.ld_weight + j]);
          mm[b] = 0.0f;
          vv[b] = 0.0f;
        }
      }
#pragma unroll
      for (int b = 0; b < kRowBatch; ++b) {
        if (i + b >= i1) continue;
        const int64_t row = i + b;
        adam_step(g[b], p[b], mm[b], vv[b], c);
        const int64_t o = row * d.ld_state + r;
        d.P[o] = p[b];
        d.M[o] = mm[b];
        d.V[o] = vv[b];
        d.weight[row * d.ld_weight + j] = round_bf16(p[b]);
      }
    }
    if (do_pack) {
      float a[kRowBatch];
#pragma unroll
      for (int b = 0; b < kRowBatch; ++b) {
        if (i + b >= i1) continue;
        a[b] = first ? g[b] : d.acc[(i + b) * d.ld_acc + u] + g[b];
      }
#pragma unroll
      for (int b = 0; b < kRowBatch; ++b) {
        if (i + b >= i1) continue;
        d.acc[(i + b) * d.ld_acc + u] = a[b];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// a6: hand-over.  Same column mapping as the update pass.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kThreads) void unpack_kernel(Table t, DevMat one, float scale) {
  int64_t local;
  const DevMat d = get_mat(t, one, blockIdx.x, local);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t cblk = local % d.up_cb;
  const int64_t rblk = local / d.up_cb;
  const int64_t word = cblk * (kUpdateCols / 64) + wave;
  const int64_t j = word * 64 + lane;
  if (j >= d.m) return;
  const uint64_t mw = d.mask[word];
  const bool sel = (mw >> lane) & 1ull;
  const int64_t u = j - (static_cast<int64_t>(d.prefix[word]) + lanes_below(mw));
  const int64_t i0 = rblk * d.up_rows;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.up_rows), d.n);
  for (int64_t i = i0; i < i1; i += kRowBatch) {
    float a[kRowBatch];
#pragma unroll
    for (int b = 0; b < kRowBatch; ++b)
      a[b] = (!sel && i + b < i1) ? d.acc[(i + b) * d.ld_acc + u] * scale : 0.0f;
#pragma unroll
    for (int b = 0; b < kRowBatch; ++b)
      if (i + b < i1) d.out[(i + b) * d.ld_out + j] = a[b];
  }
}

}  // namespace

hipError_t launch_colnorm(const Table& t, const DevMat& one, int64_t blocks, const Table& tf,
                          int64_t fin_blocks, double* ws, hipStream_t s) {
  (void)hipGetLastError();
  if (blocks > 0)
    hipLaunchKernelGGL(colnorm_partial_kernel, dim3(static_cast<uint32_t>(blocks)),
                       dim3(kThreads), 0, s, t, one, ws);
  if (fin_blocks > 0)
    hipLaunchKernelGGL(colnorm_finalize_kernel, dim3(static_cast<uint32_t>(fin_blocks)),
                       dim3(kFinalizeCols), 0, s, tf, one, static_cast<const double*>(ws));
  return hipGetLastError();
}

hipError_t launch_topk(const Table& t, const DevMat& one, int64_t blocks, hipStream_t s) {
  (void)hipGetLastError();
  if (blocks > 0)
    hipLaunchKernelGGL(topk_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTopkThreads), 0,
                       s, t, one);
  return hipGetLastError();
}

hipError_t launch_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                         int32_t mode, int32_t first, bool adam, bool pack, hipStream_t s) {
  (void)hipGetLastError();
  if (blocks <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(blocks)), block(kThreads);
  if (adam && pack)
    hipLaunchKernelGGL((update_kernel<true, true>), grid, block, 0, s, t, one, c, mode, first);
  else if (adam)
    hipLaunchKernelGGL((update_kernel<true, false>), grid, block, 0, s, t, one, c, mode, first);
  else if (pack)
    hipLaunchKernelGGL((update_kernel<false, true>), grid, block, 0, s, t, one, c, mode, first);
  return hipGetLastError();
}

hipError_t launch_unpack(const Table& t, const DevMat& one, int64_t blocks, float scale,
                         hipStream_t s) {
  (void)hipGetLastError();
  if (blocks > 0)
    hipLaunchKernelGGL(unpack_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, s,
                       t, one, scale);
  return hipGetLastError();
}

}  // namespace zf
