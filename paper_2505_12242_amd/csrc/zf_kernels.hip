// gfx950 kernels of the selective-update hot path.
//
// All kernels are bandwidth-bound streaming passes (no contraction, so no
// MFMA).  Every kernel reads its matrix descriptor from a batch table (one
// grid over many matrices; block -> matrix by binary search over the
// per-kernel block offsets) or from a single descriptor passed by value.
//
// Compiled with -ffp-contract=off and correctly rounded fp32 division and
// square root, so that each arithmetic line below is one IEEE operation.
#include "zf_device.hpp"

namespace zf {
namespace {

// ---------------------------------------------------------------------------
// a1: column scores.  Stage 1: a block sums the squares of a 512-column x
// cn_rpb-row tile in fp64 (squares of bf16 values are exact), each lane
// owning 8 adjacent columns and reading them with one 16-byte load per row;
// the four waves take interleaved rows and are combined in LDS in fixed
// order.  Stage 2 adds the row-block partials of each column in order and
// rounds once to fp32.  No atomics: the result is deterministic.
// ---------------------------------------------------------------------------

constexpr int kCnBatch = 4;  // rows per wave loaded before they are added

// G is read once and the stage written once per pass: both non-temporal
__device__ __forceinline__ u32x4 cn_load(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void cn_store(uint16_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

__device__ __forceinline__ void accum8(double (&acc)[8], u32x4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const double lo = static_cast<double>(__uint_as_float(w[h] << 16));
    const double hi = static_cast<double>(__uint_as_float(w[h] & 0xffff0000u));
    acc[2 * h] = __builtin_fma(lo, lo, acc[2 * h]);
    acc[2 * h + 1] = __builtin_fma(hi, hi, acc[2 * h + 1]);
  }
}

// STAGE (a refresh step that starts an interval, plans with the bf16
// first-step stage): the pass also copies every element it reads to the
// same place of the stage (one bf16 row per gradient row), the packing of
// whichever columns the selection leaves unselected, so that the step's
// update runs the Adam part alone.
template <bool BATCHED, bool STAGE>
__global__ __launch_bounds__(kThreads) void colnorm_partial_kernel(const DevMat* __restrict__ mats, const int64_t* __restrict__ off, int32_t nmats, DevMat one,
                                                                   double* __restrict__ ws) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const bool st = STAGE && d.acc1 != nullptr;
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
    uint16_t* __restrict__ sbase = st ? d.acc1 + c0 : nullptr;
    const int64_t sld = d.ld_acc1;
    if (d.vec && c0 + 8 <= d.m) {
      int64_t i = r0 + wave;
      for (; i + 4 * (kCnBatch - 1) < r1; i += 4 * kCnBatch) {
        u32x4 v[kCnBatch];
#pragma unroll
        for (int b = 0; b < kCnBatch; ++b) v[b] = cn_load(base + (i + 4 * b) * ld);
        if (st) {
#pragma unroll
          for (int b = 0; b < kCnBatch; ++b) cn_store(sbase + (i + 4 * b) * sld, v[b]);
        }
#pragma unroll
        for (int b = 0; b < kCnBatch; ++b) accum8(acc, v[b]);
      }
      for (; i < r1; i += 4) {
        const u32x4 v = cn_load(base + i * ld);
        if (st) cn_store(sbase + i * sld, v);
        accum8(acc, v);
      }
    } else {
      const int64_t nc = min(static_cast<int64_t>(8), d.m - c0);
      for (int64_t i = r0 + wave; i < r1; i += 4) {
        const uint16_t* row = base + i * ld;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          if (c < nc) {
            if (st) sbase[i * sld + c] = row[c];
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

template <bool BATCHED>
__global__ __launch_bounds__(kFinalizeCols) void colnorm_finalize_kernel(
    const DevMat* __restrict__ mats, const int64_t* __restrict__ off, int32_t nmats, DevMat one, const double* __restrict__ ws) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
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

template <bool BATCHED>
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(const DevMat* __restrict__ mats, const int64_t* __restrict__ off, int32_t nmats, DevMat one) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
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
// columns, in one pass over G.  A block owns a 256-column tile (four mask
// words) and a range of rows.  Its columns split into cu unselected slots
// [us, us+cu) of the accumulation buffer and cs selected slots [rs, rs+cs)
// of the compact states, both contiguous; thread t < cu owns unselected
// slot us+t, thread cu <= t < cu+cs owns selected slot rs+t-cu.  Each
// thread reads its column index once and then walks the rows: consecutive
// lanes touch consecutive slots (fully coalesced A and P/M/V traffic), the
// G gathers of a wave fall in one or two cache lines, and only the one or
// two waves holding selected slots execute the Adam arithmetic.  Rows are
// processed kRowBatch at a time with all loads issued before use.
// ---------------------------------------------------------------------------


#ifndef ZF_PACK_BATCH
#define ZF_PACK_BATCH 8
#endif
#ifndef ZF_ADAM_BATCH
#define ZF_ADAM_BATCH 8
#endif
#ifndef ZF_RM_AUX_RO
#define ZF_RM_AUX_RO kCached
#endif
#ifndef ZF_RM_AUX_W
#define ZF_RM_AUX_W kCached
#endif
constexpr int kRowBatch = ZF_PACK_BATCH;   // rows in flight per pack lane (and unpack)
constexpr int kAdamBatch = ZF_ADAM_BATCH;  // rows in flight per Adam lane

// Selected and unselected slot ranges of the tile starting at column c0.
struct TileSlots {
  int64_t rs, cs, us, cu, width;
};

__device__ __forceinline__ TileSlots tile_slots(const DevMat& d, int64_t c0) {
  TileSlots ts;
  ts.width = min(static_cast<int64_t>(kUpdateCols), d.m - c0);
  const int64_t words = (d.m + 63) >> 6;
  const int64_t w1 = (c0 + ts.width + 63) >> 6;
  ts.rs = d.prefix[c0 >> 6];
  const int64_t re = (w1 < words) ? static_cast<int64_t>(d.prefix[w1]) : d.k;
  ts.cs = re - ts.rs;
  ts.cu = ts.width - ts.cs;
  ts.us = c0 - ts.rs;
  return ts;
}

// Pack lane: A[i][u] (+)= G[i][j] over the block's rows.  HAND (last step
// of an interval, fused hand-over): scale * the new sum goes to D[i][j] (rD,
// vD, sD) and A is not written.  A16 (the bf16 first-step stage, element
// (i, j) at rS/vS/sS): 1 -- the first step stores the gradient's bits there
// instead of fp32 A; 2 -- the second step reads its previous values there.
template <bool FIRST, bool HAND = false, int A16 = 0>
__device__ __forceinline__ void pack_rows(rsrc_t rG, uint32_t vG, uint32_t sG, rsrc_t rA,
                                          uint32_t vA, uint32_t sA, int32_t rows,
                                          rsrc_t rD = rsrc_t(), uint32_t vD = 0, uint32_t sD = 0,
                                          float scale = 1.0f, rsrc_t rS = rsrc_t(),
                                          uint32_t vS = 0, uint32_t sS = 0) {
  int32_t i = 0;
  for (; i + kRowBatch <= rows; i += kRowBatch) {
    uint16_t gb[kRowBatch];
    float a[kRowBatch];
#pragma unroll
    for (int b = 0; b < kRowBatch; ++b) gb[b] = buf_u16<ZF_RM_AUX_RO>(rG, vG, (i + b) * sG);
    if constexpr (!FIRST) {
#pragma unroll
      for (int b = 0; b < kRowBatch; ++b)
        a[b] = A16 == 2 ? widen_bf16(buf_u16(rS, vS, (i + b) * sS)) : buf_f32(rA, vA, (i + b) * sA);
#pragma unroll
      for (int b = 0; b < kRowBatch; ++b) a[b] = a[b] + widen_bf16(gb[b]);
    } else {
#pragma unroll
      for (int b = 0; b < kRowBatch; ++b) a[b] = widen_bf16(gb[b]);
    }
#pragma unroll
    for (int b = 0; b < kRowBatch; ++b) {
      if constexpr (HAND) buf_put_f32(a[b] * scale, rD, vD, (i + b) * sD);
      else if constexpr (FIRST && A16 == 1) buf_put_u16(gb[b], rS, vS, (i + b) * sS);
      else buf_put_f32(a[b], rA, vA, (i + b) * sA);
    }
  }
  for (; i < rows; ++i) {
    const uint16_t gb = buf_u16<ZF_RM_AUX_RO>(rG, vG, i * sG);
    const float g = widen_bf16(gb);
    float a = g;
    if constexpr (!FIRST)
      a = (A16 == 2 ? widen_bf16(buf_u16(rS, vS, i * sS)) : buf_f32(rA, vA, i * sA)) + g;
    if constexpr (HAND) buf_put_f32(a * scale, rD, vD, i * sD);
    else if constexpr (FIRST && A16 == 1) buf_put_u16(gb, rS, vS, i * sS);
    else buf_put_f32(a, rA, vA, i * sA);
  }
}

// Where an Adam lane's (p, m, v) come from; see zf_state_mode.
struct AdamSrc {
  rsrc_t rP, rM, rV, rW;        // states and weight being written
  uint32_t vS, sS, vG, sW;      // slot / column byte offsets, row strides
  rsrc_t rSP, rSM, rSV;         // previous states (remap)
  uint32_t vPrev, sPrev;
  bool was;                     // column was selected before (remap)
  rsrc_t rI;                    // fp32 init master (init from master)
  uint32_t vI, sI;
  rsrc_t rTP, rTM, rTV;         // full-state store (swap-in)
  uint32_t vT, sT;
  rsrc_t rPA;                   // owed deferred update: previous interval's sums
  uint32_t vPA, sPA;
};

enum SrcKind {
  kSrcInplace = 0, kSrcRemapW, kSrcRemapMaster, kSrcInitW, kSrcInitMaster,
  kSrcRemapStore, kSrcInitStore,  // swap-in of new columns from the full-state store
  kSrcRemapStorePend              // the same, after the owed deferred step (Pending)
};

template <int SRC>
__device__ __forceinline__ void load_state(const AdamSrc& a, int32_t i, float& p, float& m,
                                           float& v, const Pending* pd = nullptr) {
  if constexpr (SRC == kSrcInplace) {
    p = buf_f32(a.rP, a.vS, i * a.sS);
    m = buf_f32(a.rM, a.vS, i * a.sS);
    v = buf_f32(a.rV, a.vS, i * a.sS);
  } else if constexpr (SRC == kSrcRemapStore || SRC == kSrcInitStore ||
                       SRC == kSrcRemapStorePend) {
    // Only the lanes of entering columns read the store (it may be pinned
    // host memory, where every lane's 4-byte read is its own PCIe request);
    // the others read their previous compact states.
    if (SRC != kSrcInitStore && a.was) {
      p = buf_f32(a.rSP, a.vPrev, i * a.sPrev);
      m = buf_f32(a.rSM, a.vPrev, i * a.sPrev);
      v = buf_f32(a.rSV, a.vPrev, i * a.sPrev);
    } else {
      p = buf_f32(a.rTP, a.vT, i * a.sT);
      m = buf_f32(a.rTM, a.vT, i * a.sT);
      v = buf_f32(a.rTV, a.vT, i * a.sT);
      if constexpr (SRC == kSrcRemapStorePend)  // the owed deferred step first
        adam_step(buf_f32(a.rPA, a.vPA, i * a.sPA) * pd->scale, p, m, v, pd->c);
    }
  } else {
    // init value of p for a newly selected column
    float pi;
    if constexpr (SRC == kSrcRemapMaster || SRC == kSrcInitMaster)
      pi = buf_f32(a.rI, a.vI, i * a.sI);
    else
      pi = widen_bf16(buf_u16(a.rW, a.vG, i * a.sW));
    if constexpr (SRC == kSrcRemapW || SRC == kSrcRemapMaster) {
      // both sources are read; the lane keeps the one that applies
      const float pp = buf_f32(a.rSP, a.vPrev, i * a.sPrev);
      const float mp = buf_f32(a.rSM, a.vPrev, i * a.sPrev);
      const float vp = buf_f32(a.rSV, a.vPrev, i * a.sPrev);
      p = a.was ? pp : pi;
      m = a.was ? mp : 0.0f;
      v = a.was ? vp : 0.0f;
    } else {
      p = pi;
      m = 0.0f;
      v = 0.0f;
    }
  }
}

template <int SRC>
__device__ __forceinline__ void adam_rows(const AdamSrc& a, rsrc_t rG, uint32_t sG,
                                          const AdamK& c, int32_t rows,
                                          const Pending* pd = nullptr) {
  int32_t i = 0;
  for (; i + kAdamBatch <= rows; i += kAdamBatch) {
    uint16_t gb[kAdamBatch];
    float p[kAdamBatch], mm[kAdamBatch], vv[kAdamBatch];
#pragma unroll
    for (int b = 0; b < kAdamBatch; ++b) gb[b] = buf_u16<ZF_RM_AUX_RO>(rG, a.vG, (i + b) * sG);
#pragma unroll
    for (int b = 0; b < kAdamBatch; ++b) load_state<SRC>(a, i + b, p[b], mm[b], vv[b], pd);
#pragma unroll
    for (int b = 0; b < kAdamBatch; ++b) {
      adam_step(widen_bf16(gb[b]), p[b], mm[b], vv[b], c);
      const uint32_t so = (i + b) * a.sS;
      buf_put_f32(p[b], a.rP, a.vS, so);
      buf_put_f32(mm[b], a.rM, a.vS, so);
      buf_put_f32(vv[b], a.rV, a.vS, so);
      buf_put_u16<ZF_RM_AUX_W>(round_bf16(p[b]), a.rW, a.vG, (i + b) * a.sW);
    }
  }
  for (; i < rows; ++i) {
    float p, mm, vv;
    const float g = widen_bf16(buf_u16<ZF_RM_AUX_RO>(rG, a.vG, i * sG));
    load_state<SRC>(a, i, p, mm, vv, pd);
    adam_step(g, p, mm, vv, c);
    buf_put_f32(p, a.rP, a.vS, i * a.sS);
    buf_put_f32(mm, a.rM, a.vS, i * a.sS);
    buf_put_f32(vv, a.rV, a.vS, i * a.sS);
    buf_put_u16<ZF_RM_AUX_W>(round_bf16(p), a.rW, a.vG, i * a.sW);
  }
}

// PEND (fused Adam + pack in kRemap against the store only): a column that
// enters the selection takes the owed deferred step pd first, from its slot
// among the previous selection's unselected columns.
template <bool BATCHED, bool ADAM, bool PACK, bool HAND, bool PEND>
__global__ __launch_bounds__(kThreads) void update_kernel(const DevMat* __restrict__ mats,
                                                          const int64_t* __restrict__ off,
                                                          int32_t nmats, DevMat one, AdamK c,
                                                          int32_t mode, int32_t first,
                                                          float scale, Pending pd,
                                                          const ZenState* __restrict__ zst) {
  // Zen-auto with the interval driven on the device: a refresh step, or
  // any step after an ended interval, overwrites; else it accumulates
  if (zst != nullptr)
    first = (mode != kInplace || uniform_i32(zst->ended)) ? 1 : uniform_i32(zst->length) + 1;
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int64_t cblk = local % d.up_cb;
  const int64_t rblk = local / d.up_cb;
  const int64_t c0 = cblk * kUpdateCols;
  const TileSlots ts = tile_slots(d, c0);
  const int tid = threadIdx.x;
  const bool swap_out = mode == kRemap && d.st_P != nullptr;
  const bool is_unsel = (PACK || swap_out) && tid < ts.cu;
  const bool is_adam = ADAM && tid >= ts.cu && tid < ts.width;
  if (!is_unsel && !is_adam) return;

  const int64_t i0 = rblk * d.up_rows;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.up_rows), d.n);
  const int32_t rows = static_cast<int32_t>(i1 - i0);
  const rsrc_t rG = rows_rsrc(d.grad, i0, i1, d.ld_grad, d.m);
  const uint32_t sG = static_cast<uint32_t>(d.ld_grad * 2);  // bytes per G row

  if (is_unsel) {
    const uint32_t u = static_cast<uint32_t>(ts.us + tid);
    const uint32_t j = static_cast<uint32_t>(d.unsel_idx[u]);
    if (swap_out) {
      // a column that left the selection: previous compact (p, m, v) -> store
      const uint64_t pm = d.prev_mask[j >> 6];
      if ((pm >> (j & 63u)) & 1ull) {
        const int64_t ro = static_cast<int64_t>(d.prev_prefix[j >> 6]) +
                           __popcll(pm & ((uint64_t(1) << (j & 63u)) - 1));
        for (int64_t i = i0; i < i1; ++i) {
          d.st_P[i * d.ld_store + j] = d.prev_P[i * d.ld_prev + ro];
          d.st_M[i * d.ld_store + j] = d.prev_M[i * d.ld_prev + ro];
          d.st_V[i * d.ld_store + j] = d.prev_V[i * d.ld_prev + ro];
        }
      }
    }
    if constexpr (PACK) {
      const uint32_t vG = j * 2u;
      const rsrc_t rA = rows_rsrc(d.acc, i0, i1, d.ld_acc, d.m - d.k);
      const uint32_t sA = static_cast<uint32_t>(d.ld_acc * 4);
      // the bf16 first-step stage at element (i, j): first == 1 on an
      // interval's first step, 2 on its second (a matrix without a stage
      // takes 2 as any later step)
      const bool a16 = d.acc1 != nullptr;
      const rsrc_t rS = a16 ? rows_rsrc(d.acc1, i0, i1, d.ld_acc1, d.m) : rA;
      const uint32_t sS = a16 ? static_cast<uint32_t>(d.ld_acc1 * 2) : 0u;
      if constexpr (HAND) {
        const rsrc_t rD = rows_rsrc(d.out, i0, i1, d.ld_out, d.m);
        const uint32_t sD = static_cast<uint32_t>(d.ld_out * 4);
        if (first == 1)
          pack_rows<true, true>(rG, vG, sG, rA, u * 4u, sA, rows, rD, j * 4u, sD, scale);
        else if (a16 && first == 2)
          pack_rows<false, true, 2>(rG, vG, sG, rA, u * 4u, sA, rows, rD, j * 4u, sD, scale, rS,
                                    vG, sS);
        else pack_rows<false, true>(rG, vG, sG, rA, u * 4u, sA, rows, rD, j * 4u, sD, scale);
      } else {
        if (first == 1) {
          if (a16)
            pack_rows<true, false, 1>(rG, vG, sG, rA, u * 4u, sA, rows, rsrc_t(), 0, 0, 1.0f, rS,
                                      vG, sS);
          else pack_rows<true>(rG, vG, sG, rA, u * 4u, sA, rows);
        } else if (a16 && first == 2) {
          pack_rows<false, false, 2>(rG, vG, sG, rA, u * 4u, sA, rows, rsrc_t(), 0, 0, 1.0f, rS,
                                     vG, sS);
        } else {
          pack_rows<false>(rG, vG, sG, rA, u * 4u, sA, rows);
        }
      }
    }
    return;
  }

  // Adam lane: selected slot r, column j.
  AdamSrc a;
  const uint32_t r = static_cast<uint32_t>(ts.rs + (tid - ts.cu));
  const uint32_t j = static_cast<uint32_t>(d.sel_idx[r]);
  a.vS = r * 4u;
  a.vG = j * 2u;
  a.rP = rows_rsrc(d.P, i0, i1, d.ld_state, d.k);
  a.rM = rows_rsrc(d.M, i0, i1, d.ld_state, d.k);
  a.rV = rows_rsrc(d.V, i0, i1, d.ld_state, d.k);
  a.sS = static_cast<uint32_t>(d.ld_state * 4);
  a.rW = rows_rsrc(d.weight, i0, i1, d.ld_weight, d.m);
  a.sW = static_cast<uint32_t>(d.ld_weight * 2);
  a.rSP = a.rP;
  a.rSM = a.rM;
  a.rSV = a.rV;
  a.vPrev = 0;
  a.sPrev = 0;
  a.was = false;
  a.rI = a.rW;
  a.vI = 0;
  a.sI = 0;
  const bool master = d.init_P != nullptr;
  const bool store = d.st_P != nullptr;
  if (mode != kInplace && master) {
    a.rI = rows_rsrc(d.init_P, i0, i1, d.ld_init, d.m);
    a.vI = j * 4u;
    a.sI = static_cast<uint32_t>(d.ld_init * 4);
  }
  a.rTP = a.rTM = a.rTV = a.rPA = a.rP;
  a.vT = a.vPA = 0;
  a.sT = a.sPA = 0;
  if (mode != kInplace && store) {
    a.rTP = rows_rsrc(d.st_P, i0, i1, d.ld_store, d.m);
    a.rTM = rows_rsrc(d.st_M, i0, i1, d.ld_store, d.m);
    a.rTV = rows_rsrc(d.st_V, i0, i1, d.ld_store, d.m);
    a.vT = j * 4u;
    a.sT = static_cast<uint32_t>(d.ld_store * 4);
  }
  if (mode == kRemap) {
    const uint32_t w = j >> 6;
    const uint64_t pm = d.prev_mask[w];
    a.was = (pm >> (j & 63u)) & 1ull;
    const uint32_t ro = static_cast<uint32_t>(d.prev_prefix[w]) +
                        static_cast<uint32_t>(__popcll(pm & ((uint64_t(1) << (j & 63u)) - 1)));
    // a column that was not selected reads slot 0 (any valid slot), unused
    a.vPrev = (a.was ? ro : 0u) * 4u;
    a.sPrev = static_cast<uint32_t>(d.ld_prev * 4);
    a.rSP = rows_rsrc(d.prev_P, i0, i1, d.ld_prev, d.m);
    a.rSM = rows_rsrc(d.prev_M, i0, i1, d.ld_prev, d.m);
    a.rSV = rows_rsrc(d.prev_V, i0, i1, d.ld_prev, d.m);
    if constexpr (PEND) {
      // (no unselected columns: an empty resource, every read returns 0)
      a.rPA = d.m > d.k ? rows_rsrc(d.pend_acc, i0, i1, d.ld_pend, d.m - d.k)
                        : make_rsrc(d.pend_acc, 0);
      a.vPA = (a.was ? 0u : j - ro) * 4u;
      a.sPA = static_cast<uint32_t>(d.ld_pend * 4);
    }
  }
  if constexpr (HAND) {
    // the hand-over buffer is +0.0 at a selected column
    const rsrc_t rD = rows_rsrc(d.out, i0, i1, d.ld_out, d.m);
    const uint32_t sD = static_cast<uint32_t>(d.ld_out * 4);
    for (int32_t i = 0; i < rows; ++i) buf_put_f32(0.0f, rD, j * 4u, i * sD);
  }
  if (mode == kInplace) adam_rows<kSrcInplace>(a, rG, sG, c, rows);
  else if (mode == kRemap) {
    if (PEND) adam_rows<kSrcRemapStorePend>(a, rG, sG, c, rows, &pd);
    else if (store) adam_rows<kSrcRemapStore>(a, rG, sG, c, rows);
    else if (master) adam_rows<kSrcRemapMaster>(a, rG, sG, c, rows);
    else adam_rows<kSrcRemapW>(a, rG, sG, c, rows);
  } else {
    if (store) adam_rows<kSrcInitStore>(a, rG, sG, c, rows);
    else if (master) adam_rows<kSrcInitMaster>(a, rG, sG, c, rows);
    else adam_rows<kSrcInitW>(a, rG, sG, c, rows);
  }
}

// ---------------------------------------------------------------------------
// a6: hand-over.  Same column mapping as the update pass.
// ---------------------------------------------------------------------------

// One block's share of the hand-over: the block-th tile (rows x 256
// columns) of matrix d.
__device__ __forceinline__ void unpack_unit(const DevMat& d, int64_t local, float scale) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t cblk = local % d.up_cb;
  const int64_t rblk = local / d.up_cb;
  const int64_t word = cblk * (kUpdateCols / 64) + wave;
  const int64_t j = word * 64 + lane;
  if (j >= d.m) return;
  const uint64_t mw = d.mask[word];
  const bool sel = (mw >> lane) & 1ull;
  const uint32_t u =
      static_cast<uint32_t>(j - (static_cast<int64_t>(d.prefix[word]) + lanes_below(mw)));
  const int64_t i0 = rblk * d.up_rows;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.up_rows), d.n);
  const int32_t rows = static_cast<int32_t>(i1 - i0);
  const rsrc_t rA = rows_rsrc(d.acc, i0, i1, d.ld_acc, d.m - d.k);
  const rsrc_t rD = rows_rsrc(d.out, i0, i1, d.ld_out, d.m);
  const uint32_t sA = static_cast<uint32_t>(d.ld_acc * 4);
  const uint32_t sD = static_cast<uint32_t>(d.ld_out * 4);
  const uint32_t vD = static_cast<uint32_t>(j) * 4u;
  int32_t i = 0;
  if (d.m == d.k) {  // every column selected: no accumulated data to read
    for (; i < rows; ++i) buf_put_f32(0.0f, rD, vD, i * sD);
    return;
  }
  // A selected lane reads a neighbouring valid slot (same cache lines as its
  // wave) and writes +0.0, so the wave runs one uniform loop.
  const uint32_t vA = min(u, static_cast<uint32_t>(d.m - d.k - 1)) * 4u;
  for (; i + kRowBatch <= rows; i += kRowBatch) {
    float a[kRowBatch];
#pragma unroll
    for (int b = 0; b < kRowBatch; ++b) a[b] = buf_f32(rA, vA, (i + b) * sA);
#pragma unroll
    for (int b = 0; b < kRowBatch; ++b)
      buf_put_f32(sel ? 0.0f : a[b] * scale, rD, vD, (i + b) * sD);
  }
  for (; i < rows; ++i) {
    const float a = buf_f32(rA, vA, i * sA);
    buf_put_f32(sel ? 0.0f : a * scale, rD, vD, i * sD);
  }
}

template <bool BATCHED>
__global__ __launch_bounds__(kThreads) void unpack_kernel(const DevMat* __restrict__ mats,
                                                          const int64_t* __restrict__ off,
                                                          int32_t nmats, DevMat one,
                                                          float scale) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
  unpack_unit(d, local, scale);
}

// The hand-over of an interval that Zen-auto ended on the device: nothing
// unless zst->ended == 1; then scale = fp32(1 / length) (a correctly rounded
// fp32 division, the value the host passes as fp32(1.0 / length)).  A fixed
// grid walks the table's unpack tiles, so that a step that does not end its
// interval costs one short launch.
__global__ __launch_bounds__(kThreads) void unpack_zen_kernel(const DevMat* __restrict__ mats,
                                                             const int64_t* __restrict__ off,
                                                             int32_t nmats, int64_t units,
                                                             const ZenState* __restrict__ zst) {
  if (uniform_i32(zst->ended) != 1) return;  // (2: already handed over)
  const float scale = 1.0f / static_cast<float>(uniform_i32(zst->length));
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  int lo = 0;
  for (int64_t u = b; u < units; u += gridDim.x) {
    int hi = nmats - 1;
    while (lo < hi) {  // largest q with off[q] <= u (u only grows)
      const int mid = (lo + hi + 1) >> 1;
      if (off[mid] <= u) lo = mid; else hi = mid - 1;
    }
    unpack_unit(mats[lo], u - off[lo], scale);
  }
}

// a3-a6 with deferred packing, row-major buffers off the 16-byte path: the
// interval's hand-over from the gradients it kept (the earlier steps' plans,
// then this step's), summed in step order in fp32 and scaled, +0.0 at a
// selected column.  Same column mapping as the hand-over above; the Adam
// part of the step is the per-column update's.
__global__ __launch_bounds__(kThreads) void rm_handover_deferred_kernel(
    const DevMat* __restrict__ mats, const int64_t* __restrict__ off, int32_t nmats, float scale,
    HistTable hist) {
  int64_t local;
  const DevMat& d = get_mat<true>(mats, off, nmats, mats[0], local);
  const int32_t q = static_cast<int32_t>(&d - mats);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t cblk = local % d.up_cb;
  const int64_t rblk = local / d.up_cb;
  const int64_t word = cblk * (kUpdateCols / 64) + wave;
  const int64_t j = word * 64 + lane;
  if (j >= d.m) return;
  const bool sel = (d.mask[word] >> lane) & 1ull;
  const int64_t i0 = rblk * d.up_rows;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.up_rows), d.n);
  const int32_t rows = static_cast<int32_t>(i1 - i0);
  const rsrc_t rG = rows_rsrc(d.grad, i0, i1, d.ld_grad, d.m);
  const rsrc_t rD = rows_rsrc(d.out, i0, i1, d.ld_out, d.m);
  const uint32_t sG = static_cast<uint32_t>(d.ld_grad * 2);
  const uint32_t sD = static_cast<uint32_t>(d.ld_out * 4);
  const uint32_t vG = static_cast<uint32_t>(j) * 2u;
  const uint32_t vD = static_cast<uint32_t>(j) * 4u;
  for (int32_t i = 0; i < rows; ++i) {
    float a = 0.0f;
    for (int32_t st = 0; st < hist.n; ++st) {
      const auto& hd = const_table(hist.mats[st])[q];
      const rsrc_t rE = rows_rsrc(hd.grad, i0, i1, hd.ld_grad, d.m);
      const float g = widen_bf16(buf_u16<kStream>(
          rE, vG, static_cast<uint32_t>(i) * static_cast<uint32_t>(hd.ld_grad * 2)));
      a = st == 0 ? g : a + g;
    }
    const float g = widen_bf16(buf_u16<kStream>(rG, vG, static_cast<uint32_t>(i) * sG));
    a = hist.n > 0 ? a + g : g;
    buf_put_f32(sel ? 0.0f : a * scale, rD, vD, static_cast<uint32_t>(i) * sD);
  }
}

}  // namespace

#define ZF_LAUNCH(KERNEL, GRID, BLOCK, STREAM, T, ...)                                      \
  do {                                                                                     \
    if ((T).mats != nullptr)                                                               \
      hipLaunchKernelGGL((KERNEL<true>), GRID, BLOCK, 0, STREAM, (T).mats, (T).off,          \
                         (T).nmats, __VA_ARGS__);                                          \
    else                                                                                   \
      hipLaunchKernelGGL((KERNEL<false>), GRID, BLOCK, 0, STREAM, (T).mats, (T).off,         \
                         (T).nmats, __VA_ARGS__);                                          \
  } while (0)

hipError_t launch_colnorm(const Table& t, const DevMat& one, int64_t blocks, const Table& tf,
                          int64_t fin_blocks, double* ws, hipStream_t s, bool stage) {
  (void)hipGetLastError();
  if (blocks > 0) {
    const dim3 grid(static_cast<uint32_t>(blocks));
    if (stage) {
      if (t.mats != nullptr)
        hipLaunchKernelGGL((colnorm_partial_kernel<true, true>), grid, dim3(kThreads), 0, s,
                           t.mats, t.off, t.nmats, one, ws);
      else
        hipLaunchKernelGGL((colnorm_partial_kernel<false, true>), grid, dim3(kThreads), 0, s,
                           t.mats, t.off, t.nmats, one, ws);
    } else {
      if (t.mats != nullptr)
        hipLaunchKernelGGL((colnorm_partial_kernel<true, false>), grid, dim3(kThreads), 0, s,
                           t.mats, t.off, t.nmats, one, ws);
      else
        hipLaunchKernelGGL((colnorm_partial_kernel<false, false>), grid, dim3(kThreads), 0, s,
                           t.mats, t.off, t.nmats, one, ws);
    }
  }
  if (fin_blocks > 0)
    ZF_LAUNCH(colnorm_finalize_kernel, dim3(static_cast<uint32_t>(fin_blocks)),
              dim3(kFinalizeCols), s, tf, one, static_cast<const double*>(ws));
  return hipGetLastError();
}

hipError_t launch_topk(const Table& t, const DevMat& one, int64_t blocks, hipStream_t s) {
  (void)hipGetLastError();
  if (blocks > 0)
    ZF_LAUNCH(topk_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTopkThreads), s, t, one);
  return hipGetLastError();
}

template <bool ADAM, bool PACK, bool HAND, bool PEND = false>
static void launch_update_t(const Table& t, const DevMat& one, dim3 grid, const AdamK& c,
                            int32_t mode, int32_t first, float scale, hipStream_t s,
                            const Pending& pd = Pending{}, const ZenState* zst = nullptr) {
  if (t.mats != nullptr)
    hipLaunchKernelGGL((update_kernel<true, ADAM, PACK, HAND, PEND>), grid, dim3(kThreads), 0, s,
                       t.mats, t.off, t.nmats, one, c, mode, first, scale, pd, zst);
  else
    hipLaunchKernelGGL((update_kernel<false, ADAM, PACK, HAND, PEND>), grid, dim3(kThreads), 0, s,
                       t.mats, t.off, t.nmats, one, c, mode, first, scale, pd, zst);
}

hipError_t launch_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                         int32_t mode, int32_t first, bool adam, bool pack, bool handover,
                         float scale, hipStream_t s, const Pending* pend, const ZenState* zst) {
  (void)hipGetLastError();
  if (blocks <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (handover && !(adam && pack)) return hipErrorInvalidValue;
  if (zst != nullptr && (pend != nullptr || handover || !pack)) return hipErrorInvalidValue;
  if (pend != nullptr) {
    if (!(adam && pack) || handover || mode != kRemap) return hipErrorInvalidValue;
    launch_update_t<true, true, false, true>(t, one, grid, c, mode, first, 1.0f, s, *pend);
  } else if (handover) launch_update_t<true, true, true>(t, one, grid, c, mode, first, scale, s);
  else if (adam && pack)
    launch_update_t<true, true, false>(t, one, grid, c, mode, first, 1.0f, s, Pending{}, zst);
  else if (adam) launch_update_t<true, false, false>(t, one, grid, c, mode, first, 1.0f, s);
  else if (pack)
    launch_update_t<false, true, false>(t, one, grid, c, mode, first, 1.0f, s, Pending{}, zst);
  return hipGetLastError();
}

hipError_t launch_unpack(const Table& t, const DevMat& one, int64_t blocks, float scale,
                         hipStream_t s) {
  (void)hipGetLastError();
  if (blocks > 0)
    ZF_LAUNCH(unpack_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), s, t, one,
              scale);
  return hipGetLastError();
}

// 256 blocks per CU: a step that does not end its interval exits in a
// short launch, one that does keeps enough tiles in flight (4096 and a full
// grid measured slower)
constexpr int64_t kUnpackZenGrid = 65536;

hipError_t launch_unpack_zen(const Table& t, int64_t units, const ZenState* zst, hipStream_t s) {
  (void)hipGetLastError();
  if (units <= 0 || t.mats == nullptr) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(units < kUnpackZenGrid ? units : kUnpackZenGrid));
  hipLaunchKernelGGL(unpack_zen_kernel, grid, dim3(kThreads), 0, s, t.mats, t.off, t.nmats, units,
                     zst);
  return hipGetLastError();
}

hipError_t launch_rm_handover_deferred(const Table& t, int64_t blocks, float scale,
                                       const HistTable& h, hipStream_t s) {
  (void)hipGetLastError();
  if (blocks <= 0 || t.mats == nullptr) return hipSuccess;
  hipLaunchKernelGGL(rm_handover_deferred_kernel, dim3(static_cast<uint32_t>(blocks)),
                     dim3(kThreads), 0, s, t.mats, t.off, t.nmats, scale, h);
  return hipGetLastError();
}

}  // namespace zf
