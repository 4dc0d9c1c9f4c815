// gfx950 row-major fused update with 16-byte accesses: selective Adam with
// bf16 write-back, packing of the unselected columns, and the fused
// hand-over (a3-a6 in the row-major layout).
//
// A lane that owns one column and walks the rows moves 2- and 4-byte
// elements; on this chip such per-lane narrow accesses stream at about two
// thirds of the rate of 16-byte ones.  Here a block owns a tile of up to
// kRvMaxCols columns (equal-width tiles per matrix, multiples of 8) and
// rv_rows rows, and works in two index spaces:
//   column space: G is loaded with one 16-byte load per lane (8 columns,
//     two rows per block-wide load) and staged in LDS; the fused
//     hand-over's output rows are assembled in LDS and stored with 16-byte
//     stores;
//   slot space: the tile's unselected slots [us, us+cu) of the accumulation
//     buffer and its selected slots [rs, rs+cs) of the compact states are
//     contiguous ranges.  Lanes take one of three roles:
//       pack quad:  the aligned quads of 4 slots inside [us, us+cu), one per
//                   lane, A moved with one 16-byte access per row;
//       pack edge:  the at most 6 slots of the range outside whole quads
//                   (3 at each end), one per lane, 4-byte accesses;
//       Adam:       the remaining lanes take the selected slots in turn
//                   (slot rs + a + j * lanes, j < 4), so consecutive lanes
//                   hold consecutive slots: the compact states and the bf16
//                   write-back of W coalesce as well as the layout allows.
//     Every lane reads its slots' column indices once per block and gets
//     G from LDS.  With tiles of at most 1000 columns the pack roles use at
//     most 254 lanes and an Adam lane holds at most 4 slots (checked for
//     every tile width, slot alignment and selected count).
// Rows are staged kRvBatch at a time, every load of a batch issued before
// the first wait.  The kernel serves steps with the compact states in place
// (and pack-only calls); a refresh step, whose entering and leaving columns
// read and write their sources element by element, runs the per-column
// kernel.
//
// The bf16 first-step stage (acc1, optional; one bf16 row per gradient row):
// on an interval's first step (first == 1) the block stores the G rows it
// loads into the stage as they are (every column, 16 bytes per lane) and
// the pack lanes write nothing; on its second (first == 2) the stage rows
// are loaded and staged in LDS like G, and the pack lanes take their
// previous values from there instead of from A.
//
// STATS (Zen-auto, blocks of cn_rpb rows; with HAND on an end the caller
// forces, the sums before the scale): each lane also sums, in fp64 and
// in row order, the squares of its selected columns' gradient and of its
// unselected slots' new accumulated values over the block's rows, and
// writes one partial per virtual column (selected slot r, then unselected
// slot k + u) and row block into the column-score workspace -- the partials
// of the row-major statistics pass, in the same order, for its finalize.
//
// DEF (deferred packing, the hand-over of the interval's last step; no
// Adam, no packed buffer): the column-space lanes load, for their 8 columns
// of each row, that row of every earlier gradient of the interval (the same
// matrix in the earlier steps' plans) and of this step's, add them in step
// order in fp32 with this step's last, and store the hand-over -- +0.0 at a
// selected column, else the sum times `scale` -- with two 16-byte
// non-temporal stores per lane, after lane shuffles that make each store of
// a wave cover 1 KiB of the row (whole lines).  The step's Adam runs before it as the Adam-only instantiation over the
// same tiles.  (Fused into one pass with the Adam lanes the kernel needs
// registers for both and ran slower than the two passes.)
//
// The arithmetic per element is that of the per-column kernel (same fp32
// operations in the same order), so both paths give identical bits.
#include "zf_device.hpp"

namespace zf {
namespace {

#ifndef ZF_RV_BATCH
#define ZF_RV_BATCH 4
#endif
constexpr int kRvBatch = ZF_RV_BATCH;  // rows staged together (two per G load)
static_assert(kRvBatch % 2 == 0 && kRvBatch >= 2, "rows are loaded in pairs");
static_assert(kRvMaxCols % 8 == 0 && kRvMaxCols <= 1000, "lane budget of the roles");

// Number of selected columns below column j (0 <= j <= m); j is the same
// for every lane.
__device__ __forceinline__ int64_t selected_below(const DevMat& d, int64_t j) {
  if (j >= d.m) return d.k;
  const int64_t w = j >> 6;
  const uint64_t mw = uniform_u64(d.mask[w]);
  return static_cast<int64_t>(uniform_i32(d.prefix[w])) +
         __popcll(mw & ((uint64_t(1) << (j & 63)) - 1));
}

// The 8 bf16 of a 16-byte group, widened (element x in half x & 1 of word
// x >> 1).
__device__ __forceinline__ void widen_group(u32x4 v, float (&f)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int x = 0; x < 8; ++x)
    f[x] = widen_bf16(static_cast<uint16_t>(w[x >> 1] >> (16 * (x & 1))));
}

// Row b of a batch, 8 columns at byte offset vo: one 16-byte load, or the
// ragged tail of a tile element by element (zeros past the tile).
template <int AUX>
__device__ __forceinline__ u32x4 load_group(rsrc_t r, uint32_t vo, uint32_t so, int32_t cols) {
  if (cols >= 8) return buf_b128<AUX>(r, vo, so);
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  for (int x = 0; x < cols; ++x)
    w[x >> 1] |= static_cast<uint32_t>(buf_u16<AUX>(r, vo + 2 * x, so)) << (16 * (x & 1));
  return u32x4{w[0], w[1], w[2], w[3]};
}

// earlier steps whose rows are loaded before they are added (2, 3 and 4
// measured alike)
constexpr int kDefBatch = 2;

__device__ __forceinline__ float4 as_f4(u32x4 v) {
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                     __uint_as_float(v.w));
}
__device__ __forceinline__ u32x4 as_u4(float a, float b, float c, float d) {
  return u32x4{__float_as_uint(a), __float_as_uint(b), __float_as_uint(c), __float_as_uint(d)};
}

template <bool BATCHED, bool ADAM, bool PACK, bool HAND, bool STATS, bool A16, bool DEF>
__global__ __launch_bounds__(kThreads) void rv_update_kernel(const DevMat* __restrict__ mats,
                                                             const int64_t* __restrict__ off,
                                                             int32_t nmats, DevMat one, AdamK c,
                                                             int32_t first, float scale,
                                                             double* __restrict__ zs,
                                                             HistTable hist,
                                                             const ZenState* __restrict__ zst) {
  static_assert(!STATS || (ADAM && PACK), "statistics of the fused update");
  static_assert(!DEF || (BATCHED && !ADAM && !PACK && !HAND && !STATS && !A16),
                "the deferred hand-over pass");
  // Zen-auto with the interval driven on the device (steps in place):
  // overwrite after an ended interval, else accumulate; HAND (an end the
  // caller forces) hands over with scale = fp32(1 / length)
  if (zst != nullptr) {
    first = uniform_i32(zst->ended) ? 1 : uniform_i32(zst->length) + 1;
    if constexpr (HAND) scale = 1.0f / static_cast<float>(first);
  }
  __shared__ __attribute__((aligned(16))) uint16_t sg[kRvBatch][kRvMaxCols];
  __shared__ __attribute__((aligned(16))) uint16_t sa[A16 ? kRvBatch : 1][A16 ? kRvMaxCols : 8];
  __shared__ __attribute__((aligned(16))) float sd[HAND ? kRvBatch : 1][HAND ? kRvMaxCols : 4];

  int64_t local;
  const DevMat& d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int32_t q = BATCHED ? static_cast<int32_t>(&d - mats) : 0;
  const int64_t cblk = local % d.rv_cb;
  const int64_t rblk = local / d.rv_cb;
  const int64_t c0 = cblk * d.rv_w;
  const int32_t width = static_cast<int32_t>(min(static_cast<int64_t>(d.rv_w), d.m - c0));
  const int64_t rs = selected_below(d, c0);
  const int32_t cs = static_cast<int32_t>(selected_below(d, c0 + width) - rs);
  const int64_t us = c0 - rs;
  const int32_t cu = width - cs;
  const bool do_u = PACK && cu > 0;

  // Lane roles (see above).  nqf whole quads [qf0, qf0 + nqf) of the
  // unselected range, then ne edge slots (head then tail), then Adam lanes.
  int64_t qf0 = 0;
  int32_t nqf = 0, nh = 0, ne = 0;
  if (do_u) {
    qf0 = (us + 3) >> 2;
    const int64_t qf1 = (us + cu) >> 2;
    if (qf1 > qf0) {
      nqf = static_cast<int32_t>(qf1 - qf0);
      nh = static_cast<int32_t>(4 * qf0 - us);
      ne = nh + static_cast<int32_t>(us + cu - 4 * qf1);
    } else {
      nh = cu;
      ne = cu;
    }
  }
  const int32_t nA = kThreads - nqf - ne;  // >= 1 whenever cs > 0
  const int tid = threadIdx.x;
  const bool is_q = tid < nqf;
  const bool is_e = !is_q && tid < nqf + ne;
  const bool is_s = ADAM && tid >= nqf + ne && cs > 0;

  // The lane's elements: slot s[e] (byte offset vs[e] in its buffer's
  // row), column offset cj[e] in the tile, valid bit e.
  int64_t Q = 0;
  uint32_t valid = 0;
  int32_t cj[4] = {0, 0, 0, 0};
  uint32_t vs[4] = {0u, 0u, 0u, 0u};
  if (is_q) {
    Q = qf0 + tid;
    valid = 0xFu;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      cj[e] = d.unsel_idx[4 * Q + e] - static_cast<int32_t>(c0);
      vs[e] = static_cast<uint32_t>((4 * Q + e) * 4);
    }
  } else if (is_e) {
    const int32_t x = tid - nqf;
    const int64_t sl = x < nh ? us + x : us + cu - (ne - x);
    valid = 1u;
    cj[0] = d.unsel_idx[sl] - static_cast<int32_t>(c0);
    vs[0] = static_cast<uint32_t>(sl * 4);
  } else if (is_s) {
    const int32_t a = tid - nqf - ne;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int32_t r = a + e * nA;
      if (r < cs) {
        valid |= 1u << e;
        cj[e] = d.sel_idx[rs + r] - static_cast<int32_t>(c0);
        vs[e] = static_cast<uint32_t>((rs + r) * 4);
      }
    }
  }
  // Indices come from the caller's selection; keep LDS accesses inside the
  // tile whatever they hold.
#pragma unroll
  for (int e = 0; e < 4; ++e) cj[e] = min(max(cj[e], 0), width - 1);

  const int64_t i0 = rblk * d.rv_rows;
  const int64_t i1 = min(i0 + static_cast<int64_t>(d.rv_rows), d.n);
  const int32_t rows = static_cast<int32_t>(i1 - i0);
  const rsrc_t rG = rows_rsrc(d.grad, i0, i1, d.ld_grad, d.m);
  const uint32_t sG = static_cast<uint32_t>(d.ld_grad * 2);
  rsrc_t rA = rsrc_t(), rP = rsrc_t(), rM = rsrc_t(), rV = rsrc_t(), rW = rsrc_t(), rD = rsrc_t();
  uint32_t sA = 0, sS = 0, sW = 0, sD = 0;
  rsrc_t rT = rsrc_t();
  uint32_t sT = 0;
  const bool a16 = A16 && PACK && d.acc1 != nullptr;
  const bool put16 = a16 && first == 1 && !HAND;  // store G rows to the stage
  const bool get16 = a16 && first == 2;           // read the stage rows
  if constexpr (PACK) {
    rA = rows_rsrc(d.acc, i0, i1, d.ld_acc, d.m - d.k);
    sA = static_cast<uint32_t>(d.ld_acc * 4);
    if (a16) {
      rT = rows_rsrc(d.acc1, i0, i1, d.ld_acc1, d.m);
      sT = static_cast<uint32_t>(d.ld_acc1 * 2);
    }
  }
  if constexpr (ADAM) {
    rP = rows_rsrc(d.P, i0, i1, d.ld_state, d.k);
    rM = rows_rsrc(d.M, i0, i1, d.ld_state, d.k);
    rV = rows_rsrc(d.V, i0, i1, d.ld_state, d.k);
    sS = static_cast<uint32_t>(d.ld_state * 4);
    rW = rows_rsrc(d.weight, i0, i1, d.ld_weight, d.m);
    sW = static_cast<uint32_t>(d.ld_weight * 2);
  }
  if constexpr (HAND || DEF) {
    rD = rows_rsrc(d.out, i0, i1, d.ld_out, d.m);
    sD = static_cast<uint32_t>(d.ld_out * 4);
  }
  // DEF: which of the lane's 8 columns are selected (c0 and g8 are
  // multiples of 8, so the 8 bits sit in one mask word)
  uint32_t sel8 = 0;

  // Column-space lane roles: G loads (row pair half h, 8-column group g8),
  // hand-over stores (4-column group).
  const int h = uniform_i32(tid >> 7);  // the same for the 64 lanes of a wave
  const int32_t g8 = (tid & 127) * 8;
  if constexpr (DEF) {
    if (g8 < width) {
      const int64_t cg = c0 + g8;
      sel8 = static_cast<uint32_t>(d.mask[cg >> 6] >> (cg & 63)) & 0xFFu;
    }
  }
  const uint32_t vQ = static_cast<uint32_t>(Q * 16);  // quad byte offset (fp32 slots)
  double zq[4] = {0.0, 0.0, 0.0, 0.0};  // STATS: sums of squares per element

  for (int32_t i = 0; i < rows; i += kRvBatch) {
    const int32_t nb = min(kRvBatch, rows - i);
    // the previous batch is done with the LDS rows (the hand-over pass uses none)
    if (i > 0 && (ADAM || PACK)) __syncthreads();

    // 1. G rows of the batch (16-byte loads of 8 columns; ragged tail of
    //    the last tile element by element).
    u32x4 gv[kRvBatch / 2], av[kRvBatch / 2];
#pragma unroll
    for (int p = 0; p < kRvBatch / 2; ++p) {
      const int b = 2 * p + h;
      gv[p] = u32x4{0u, 0u, 0u, 0u};
      av[p] = u32x4{0u, 0u, 0u, 0u};
      if (b < nb && g8 < width) {
        const uint32_t so = static_cast<uint32_t>(i + b) * sG;
        const uint32_t vo = static_cast<uint32_t>((c0 + g8) * 2);
        const uint32_t to = static_cast<uint32_t>(i + b) * sT;
        if (g8 + 8 <= width) {
          gv[p] = buf_b128<kStream>(rG, vo, so);
          if (get16) av[p] = buf_b128<kStream>(rT, vo, to);
        } else {
          uint32_t w[4] = {0u, 0u, 0u, 0u}, x4[4] = {0u, 0u, 0u, 0u};
          for (int x = 0; g8 + x < width; ++x) {
            w[x >> 1] |= static_cast<uint32_t>(buf_u16<kStream>(rG, vo + 2 * x, so))
                         << (16 * (x & 1));
            if (get16)
              x4[x >> 1] |= static_cast<uint32_t>(buf_u16<kStream>(rT, vo + 2 * x, to))
                            << (16 * (x & 1));
          }
          gv[p] = u32x4{w[0], w[1], w[2], w[3]};
          av[p] = u32x4{x4[0], x4[1], x4[2], x4[3]};
        }
      }
    }
    if (put16) {
      // the first step's packed values: the gradient rows themselves
#pragma unroll
      for (int p = 0; p < kRvBatch / 2; ++p) {
        const int b = 2 * p + h;
        if (b < nb && g8 < width) {
          const uint32_t to = static_cast<uint32_t>(i + b) * sT;
          const uint32_t vo = static_cast<uint32_t>((c0 + g8) * 2);
          if (g8 + 8 <= width) {
            buf_put_b128<kStream>(gv[p], rT, vo, to);
          } else {
            const uint32_t w[4] = {gv[p].x, gv[p].y, gv[p].z, gv[p].w};
            for (int x = 0; g8 + x < width; ++x)
              buf_put_u16<kStream>(static_cast<uint16_t>(w[x >> 1] >> (16 * (x & 1))), rT,
                                   vo + 2 * x, to);
          }
        }
      }
    }

    if constexpr (DEF) {
      // the hand-over of the lane's 8 columns in rows 2p + h of the batch
      const int32_t cols = width - g8;
      const uint32_t vo = static_cast<uint32_t>((c0 + g8) * 2);
      float a[kRvBatch / 2][8];
      for (int32_t s0 = 0; s0 < hist.n; s0 += kDefBatch) {
        u32x4 ev[kDefBatch][kRvBatch / 2];
#pragma unroll
        for (int e = 0; e < kDefBatch; ++e) {
          const int32_t st = s0 + e;
          if (st < hist.n) {
            const auto& hd = const_table(hist.mats[st])[q];
            const rsrc_t rE = rows_rsrc(hd.grad, i0, i1, hd.ld_grad, d.m);
            const uint32_t sE = static_cast<uint32_t>(hd.ld_grad * 2);
#pragma unroll
            for (int p = 0; p < kRvBatch / 2; ++p) {
              const int b = 2 * p + h;
              ev[e][p] = u32x4{0u, 0u, 0u, 0u};
              if (b < nb && cols > 0)
                ev[e][p] = load_group<kStream>(rE, vo, static_cast<uint32_t>(i + b) * sE, cols);
            }
          }
        }
#pragma unroll
        for (int e = 0; e < kDefBatch; ++e) {
          const int32_t st = s0 + e;
          if (st < hist.n) {
#pragma unroll
            for (int p = 0; p < kRvBatch / 2; ++p) {
              float g[8];
              widen_group(ev[e][p], g);
#pragma unroll
              for (int x = 0; x < 8; ++x) a[p][x] = st == 0 ? g[x] : a[p][x] + g[x];
            }
          }
        }
      }
      // The stores in whole lines: lane l of a wave holds the wave's columns
      // 8l .. 8l+7 and stores columns 4l .. 4l+3 and 256+4l .. 256+4l+3,
      // held by lanes l/2 and 32 + l/2 (their values 4(l&1) .. 4(l&1)+3),
      // so that each 16-byte store of the wave fills 1 KiB of the row.  wc:
      // the tile's columns from the wave's first (the same for the wave).
      const int lane = tid & 63;
      const int32_t wc = width - (g8 - 8 * lane);
      const uint32_t vw = static_cast<uint32_t>((c0 + g8 - 8 * lane) * 4);
#pragma unroll
      for (int p = 0; p < kRvBatch / 2; ++p) {
        const int b = 2 * p + h;
        if (b < nb && wc > 0) {
          float g[8];
          widen_group(gv[p], g);
#pragma unroll
          for (int x = 0; x < 8; ++x) {
            const float sum = hist.n > 0 ? a[p][x] + g[x] : g[x];
            a[p][x] = ((sel8 >> x) & 1u) ? 0.0f : sum * scale;
          }
          float lo[8], hi[8];
#pragma unroll
          for (int x = 0; x < 8; ++x) {
            lo[x] = __shfl(a[p][x], lane >> 1, 64);
            hi[x] = __shfl(a[p][x], 32 + (lane >> 1), 64);
          }
          const bool odd = lane & 1;
          const uint32_t so = static_cast<uint32_t>(i + b) * sD;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            float v[4];
#pragma unroll
            for (int x = 0; x < 4; ++x)
              v[x] = half == 0 ? (odd ? lo[4 + x] : lo[x]) : (odd ? hi[4 + x] : hi[x]);
            const int32_t cq = half * 256 + 4 * lane;  // the quad's first column in the wave
            if (cq + 4 <= wc) {
              buf_put_b128<kStream>(as_u4(v[0], v[1], v[2], v[3]), rD, vw + 4 * cq, so);
            } else {
#pragma unroll
              for (int x = 0; x < 4; ++x)
                if (cq + x < wc) buf_put_f32<kStream>(v[x], rD, vw + 4 * (cq + x), so);
            }
          }
        }
      }
    }

    // 2. Slot data of the batch: A (pack roles, after the first step of an
    //    interval) or the Adam states.
    float x0[kRvBatch][4], x1[kRvBatch][4], x2[kRvBatch][4];
#pragma unroll
    for (int b = 0; b < kRvBatch; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) x0[b][e] = x1[b][e] = x2[b][e] = 0.0f;
    if (PACK && first != 1 && !get16) {
      if (is_q) {
#pragma unroll
        for (int b = 0; b < kRvBatch; ++b) {
          if (b < nb) {
            const float4 v = as_f4(buf_b128(rA, vQ, static_cast<uint32_t>(i + b) * sA));
            x0[b][0] = v.x;
            x0[b][1] = v.y;
            x0[b][2] = v.z;
            x0[b][3] = v.w;
          }
        }
      } else if (is_e) {
#pragma unroll
        for (int b = 0; b < kRvBatch; ++b)
          if (b < nb) x0[b][0] = buf_f32(rA, vs[0], static_cast<uint32_t>(i + b) * sA);
      }
    }
    if (ADAM && is_s) {
#pragma unroll
      for (int b = 0; b < kRvBatch; ++b) {
        if (b < nb) {
          const uint32_t so = static_cast<uint32_t>(i + b) * sS;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if ((valid >> e) & 1u) {
              x0[b][e] = buf_f32(rP, vs[e], so);
              x1[b][e] = buf_f32(rM, vs[e], so);
              x2[b][e] = buf_f32(rV, vs[e], so);
            }
          }
        }
      }
    }

    if constexpr (!ADAM && !PACK) continue;  // the hand-over alone

    // 3. Stage G in LDS.
#pragma unroll
    for (int p = 0; p < kRvBatch / 2; ++p) {
      const int b = 2 * p + h;
      if (b < nb && g8 < width) {
        *reinterpret_cast<u32x4*>(&sg[b][g8]) = gv[p];
        if (get16) *reinterpret_cast<u32x4*>(&sa[b][g8]) = av[p];
      }
    }
    __syncthreads();

    // 4. Slot-space arithmetic and stores.
    if (is_q || is_e) {
      if constexpr (PACK) {
#pragma unroll
        for (int b = 0; b < kRvBatch; ++b) {
          if (b < nb) {
            float a[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float g = widen_bf16(sg[b][cj[e]]);
              const float prev = get16 ? widen_bf16(sa[b][cj[e]]) : x0[b][e];
              a[e] = first == 1 ? g : prev + g;
              if constexpr (STATS) {
                const double x = static_cast<double>(a[e]);
                zq[e] = __builtin_fma(x, x, zq[e]);
              }
            }
            if constexpr (HAND) {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if ((valid >> e) & 1u) sd[b][cj[e]] = a[e] * scale;
            } else if (!put16) {
              const uint32_t so = static_cast<uint32_t>(i + b) * sA;
              if (is_q) buf_put_b128(as_u4(a[0], a[1], a[2], a[3]), rA, vQ, so);
              else buf_put_f32(a[0], rA, vs[0], so);
            }
          }
        }
      }
    } else if (ADAM && is_s) {
#pragma unroll
      for (int b = 0; b < kRvBatch; ++b) {
        if (b < nb) {
          const uint32_t so = static_cast<uint32_t>(i + b) * sS;
          const uint32_t sw = static_cast<uint32_t>(i + b) * sW;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if ((valid >> e) & 1u) {
              const float g = widen_bf16(sg[b][cj[e]]);
              if constexpr (STATS) {
                const double x = static_cast<double>(g);
                zq[e] = __builtin_fma(x, x, zq[e]);
              }
              adam_step(g, x0[b][e], x1[b][e], x2[b][e], c);
              buf_put_f32(x0[b][e], rP, vs[e], so);
              buf_put_f32(x1[b][e], rM, vs[e], so);
              buf_put_f32(x2[b][e], rV, vs[e], so);
              buf_put_u16<kStream>(round_bf16(x0[b][e]), rW,
                                   static_cast<uint32_t>(c0 + cj[e]) * 2u, sw);
              if constexpr (HAND) sd[b][cj[e]] = 0.0f;  // hand-over: +0 at a selected column
            }
          }
        }
      }
    }

    // 5. Fused hand-over: the assembled output rows, 16 bytes per lane.
    if constexpr (HAND) {
      __syncthreads();
      const int32_t c4 = tid * 4;
      if (c4 < width) {
        const uint32_t vo = static_cast<uint32_t>((c0 + c4) * 4);
#pragma unroll
        for (int b = 0; b < kRvBatch; ++b) {
          if (b < nb) {
            const uint32_t so = static_cast<uint32_t>(i + b) * sD;
            if (c4 + 4 <= width) {
              buf_put_b128(*reinterpret_cast<const u32x4*>(&sd[b][c4]), rD, vo, so);
            } else {
              for (int x = 0; c4 + x < width; ++x) buf_put_f32(sd[b][c4 + x], rD, vo + 4 * x, so);
            }
          }
        }
      }
    }
  }

  if constexpr (STATS) {
    // one partial per virtual column of this row block (rv_rows = cn_rpb)
    double* __restrict__ out = zs + d.cn_ws + rblk * d.m;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if ((valid >> e) & 1u) {
        if (is_s) out[vs[e] >> 2] = zq[e];                      // selected slot r
        else if (is_q || is_e) out[d.k + (vs[e] >> 2)] = zq[e];  // k + unselected slot u
      }
    }
  }
}

template <bool ADAM, bool PACK, bool HAND, bool STATS, bool A16>
void launch_rv_a(const Table& t, const DevMat& one, dim3 grid, const AdamK& c, int32_t first,
                 float scale, hipStream_t s, double* zs, const ZenState* zst = nullptr) {
  const HistTable none{};
  if (t.mats != nullptr)
    hipLaunchKernelGGL((rv_update_kernel<true, ADAM, PACK, HAND, STATS, A16, false>), grid,
                       dim3(kThreads), 0, s, t.mats, t.off, t.nmats, one, c, first, scale, zs,
                       none, zst);
  else
    hipLaunchKernelGGL((rv_update_kernel<false, ADAM, PACK, HAND, STATS, A16, false>), grid,
                       dim3(kThreads), 0, s, t.mats, t.off, t.nmats, one, c, first, scale, zs,
                       none, zst);
}

// The stage's code (and its registers and LDS) only in the launches of the
// phases that use it: an interval's first step without the hand-over, and
// its second step.  (Zen-auto statistics never run with a row-major stage.)
template <bool ADAM, bool PACK, bool HAND, bool STATS = false>
void launch_rv_t(const Table& t, const DevMat& one, dim3 grid, const AdamK& c, int32_t first,
                 float scale, hipStream_t s, double* zs = nullptr, const ZenState* zst = nullptr) {
  if constexpr (PACK && !STATS) {
    if (zst == nullptr && (first == 2 || (first == 1 && !HAND))) {
      launch_rv_a<ADAM, PACK, HAND, STATS, true>(t, one, grid, c, first, scale, s, zs);
      return;
    }
  }
  launch_rv_a<ADAM, PACK, HAND, STATS, false>(t, one, grid, c, first, scale, s, zs, zst);
}

}  // namespace

hipError_t launch_rv_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                            int32_t mode, int32_t first, bool adam, bool pack, bool handover,
                            float scale, hipStream_t s, double* zs, const ZenState* zst) {
  (void)hipGetLastError();
  if (blocks <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (handover && !(adam && pack)) return hipErrorInvalidValue;
  if (adam && mode != kInplace) return hipErrorInvalidValue;  // refresh: per-column kernel
  if (zst != nullptr && zs == nullptr) return hipErrorInvalidValue;  // Zen-auto steps only
  if (zs != nullptr) {
    if (!(adam && pack) || (handover && zst == nullptr)) return hipErrorInvalidValue;
    if (handover) launch_rv_t<true, true, true, true>(t, one, grid, c, first, 1.0f, s, zs, zst);
    else launch_rv_t<true, true, false, true>(t, one, grid, c, first, 1.0f, s, zs, zst);
  } else if (handover) launch_rv_t<true, true, true>(t, one, grid, c, first, scale, s);
  else if (adam && pack) launch_rv_t<true, true, false>(t, one, grid, c, first, 1.0f, s);
  else if (adam) launch_rv_t<true, false, false>(t, one, grid, c, first, 1.0f, s);
  else if (pack) launch_rv_t<false, true, false>(t, one, grid, c, first, 1.0f, s);
  return hipGetLastError();
}

hipError_t launch_rv_handover_deferred(const Table& t, const DevMat& one, int64_t blocks,
                                       const AdamK& c, float scale, const HistTable& h,
                                       hipStream_t s) {
  (void)hipGetLastError();
  if (blocks <= 0 || t.mats == nullptr) return hipSuccess;
  launch_rv_a<true, false, false, false, false>(t, one, dim3(static_cast<uint32_t>(blocks)), c, 0,
                                                1.0f, s, nullptr);
  hipLaunchKernelGGL((rv_update_kernel<true, false, false, false, false, false, true>),
                     dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, s, t.mats, t.off,
                     t.nmats, one, c, 0, scale, nullptr, h, nullptr);
  return hipGetLastError();
}

}  // namespace zf
