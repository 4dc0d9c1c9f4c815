// gfx950 kernels for the channel-major layout.
//
// The paper stores gradients column-major so that an input channel can be
// accessed as one unit (Implementation, "Fully Segmented Gradient
// Selection").  Here a logical n x m weight (n outputs, m input channels) is
// held as its transpose, [m][ld >= n]: channel j is one contiguous row of n
// values.  The compact states are [k][ld_state >= n] (slot r = channel
// sel_idx[r]), the packed buffer [m-k][ld_acc >= n] (slot u = channel
// unsel_idx[u]) and the hand-over buffer [m][ld_out >= n].  Every access of
// the hot path is then a contiguous stream, and the bf16 write-back writes
// whole cache lines.
//
// Work unit of update / unpack: one channel x one chunk of its rows.
// Whether the channel is selected, and its slot, are uniform per block, so
// a block is either an Adam block or a pack block.  A block's buffer
// resources cover exactly its chunk, so quads past the end of a channel (the
// last chunk) read zeros and their stores are dropped by the hardware range
// check; the loops carry no per-quad conditions.  The vector path requires
// n % 8 == 0 and 16-byte aligned rows (DevMat::vec); other shapes take an
// element-wise path.
#include "zf_device.hpp"

namespace zf {
namespace {

constexpr int kGroup = 8;  // bf16 elements in 16 bytes

// Cache policy per stream, chosen by measurement on MI355X (7B and 13B
// sets, alternating runs per variant): streams read once by a pass -- G in
// every pass, the init sources --, streams only written by a pass (the
// hand-over output, the packed buffer on an interval's first step) and the
// bf16 weight write-back are non-temporal; read-modify-write streams keep
// the default policy (non-temporal there made the Adam pass 10-17% slower).
// Default-policy loads of the read-only streams cost 1-2% per step;
// non-temporal stores of the write-only ones gain about 1%.
#ifndef ZF_AUX_SCORE
#define ZF_AUX_SCORE kStream
#endif
#ifndef ZF_AUX_RO
#define ZF_AUX_RO kStream
#endif
#ifndef ZF_AUX_WO
#define ZF_AUX_WO kStream
#endif
#ifndef ZF_AUX_RMW
#define ZF_AUX_RMW kCached
#endif
constexpr int kAuxScore = ZF_AUX_SCORE;  // G in the column-score pass
constexpr int kAuxRO = ZF_AUX_RO;        // streams only read by a pass
constexpr int kAuxWO = ZF_AUX_WO;        // streams only written by a pass
#ifndef ZF_AUX_W
#define ZF_AUX_W kStream
#endif
#ifndef ZF_AUX_AFIRST
#define ZF_AUX_AFIRST ZF_AUX_WO
#endif
constexpr int kAuxW = ZF_AUX_W;            // the bf16 weight write-back
constexpr int kAuxAFirst = ZF_AUX_AFIRST;  // the packed buffer on an interval's first step
constexpr int kAuxRMW = ZF_AUX_RMW;      // streams read and written back

// bf16 x 8 (four dwords) -> fp32 x 8
__device__ __forceinline__ void widen8(u32x4 v, float (&f)[kGroup]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    f[2 * h] = __uint_as_float(w[h] << 16);
    f[2 * h + 1] = __uint_as_float(w[h] & 0xffff0000u);
  }
}

// The vector paths of the update, the deferred hand-over and the unpack
// work in quads: 4 consecutive elements per lane access (8 bytes of bf16,
// 16 of fp32), quad q of thread tid at elements (q * kThreads + tid) * 4 of
// the block's chunk.  The 64 lanes of a wave then touch 256 consecutive
// elements with every load and store, whole cache lines of each stream.  (A
// lane holding 8 consecutive fp32 values splits them over two accesses that
// each fill half of every line they touch; the quads measured 5-10% faster
// on MI355X, together with chunks of one quad per lane.)
constexpr int kQuad = 4;

__device__ __forceinline__ uint32_t quad_elem(int q, int tid) {
  return static_cast<uint32_t>((q * kThreads + tid) * kQuad);
}

// bf16 x 4 (two dwords) -> fp32 x 4
__device__ __forceinline__ void widen4(u32x2 v, float (&f)[kQuad]) {
  f[0] = __uint_as_float(v.x << 16);
  f[1] = __uint_as_float(v.x & 0xffff0000u);
  f[2] = __uint_as_float(v.y << 16);
  f[3] = __uint_as_float(v.y & 0xffff0000u);
}

__device__ __forceinline__ u32x2 narrow4(const float (&f)[kQuad]) {
  u32x2 v;
  v.x = static_cast<uint32_t>(round_bf16(f[0])) | (static_cast<uint32_t>(round_bf16(f[1])) << 16);
  v.y = static_cast<uint32_t>(round_bf16(f[2])) | (static_cast<uint32_t>(round_bf16(f[3])) << 16);
  return v;
}

template <int AUX>
__device__ __forceinline__ void f32x4_load(rsrc_t r, uint32_t byte_off, float (&f)[kQuad]) {
  const u32x4 a = buf_b128<AUX>(r, byte_off, 0);
  f[0] = __uint_as_float(a.x); f[1] = __uint_as_float(a.y);
  f[2] = __uint_as_float(a.z); f[3] = __uint_as_float(a.w);
}

template <int AUX>
__device__ __forceinline__ void f32x4_store(rsrc_t r, uint32_t byte_off, const float (&f)[kQuad]) {
  u32x4 a;
  a.x = __float_as_uint(f[0]); a.y = __float_as_uint(f[1]);
  a.z = __float_as_uint(f[2]); a.w = __float_as_uint(f[3]);
  buf_put_b128<AUX>(a, r, byte_off, 0);
}

// ss += x^2 over fp32 values, in fp64 (squares of fp32 values are exact in
// fp64).
template <int N>
__device__ __forceinline__ void sum_squares(const float (&f)[N], double& ss) {
#pragma unroll
  for (int i = 0; i < N; ++i)
    ss = __builtin_fma(static_cast<double>(f[i]), static_cast<double>(f[i]), ss);
}

// ---------------------------------------------------------------------------
// a1: column scores.  One wave per channel: lanes stride through the row
// with 16-byte loads and sum squares in fp64 (exact squares), then a fixed
// xor-butterfly across the wave.  Deterministic, no workspace.
// ---------------------------------------------------------------------------

// The same pass may also do the refresh step's packing, before the
// selection is known, for whichever channels it leaves unselected (the
// step's update then runs the Adam part alone):
//   OUT == 1 (an interval starts): every channel's gradient row is copied
//     to its row of the bf16 first-step stage;
//   OUT == 2 (a one-step interval, handed over at once): scale times every
//     channel's widened gradient goes to its row of the hand-over buffer
//     (the selected rows are set to +0.0 by the update).
template <bool BATCHED, int OUT>
__global__ __launch_bounds__(kThreads) void cm_colnorm_kernel(const DevMat* __restrict__ mats,
                                                             const int64_t* __restrict__ off,
                                                             int32_t nmats, DevMat one,
                                                             float scale) {
  int64_t local;
  const DevMat d = get_mat<BATCHED>(mats, off, nmats, one, local);
  const int lane = threadIdx.x & 63;
  // the wave's channel, moved to scalar registers (it is wave-uniform, which
  // the compiler cannot tell from threadIdx.x; without this every buffer
  // access of the wave sits in a per-lane loop)
  const int64_t j = local * (kThreads / 64) + uniform_i32(threadIdx.x >> 6);
  if (j >= d.m) return;
  const int64_t n = d.n;
  const rsrc_t r = make_rsrc(d.grad + j * d.ld_grad, n * 2);
  const bool st = OUT == 1 && d.acc1 != nullptr;
  const rsrc_t rS = st ? make_rsrc(d.acc1 + j * d.ld_acc1, n * 2) : r;
  const rsrc_t rO = OUT == 2 ? make_rsrc(d.out + j * d.ld_out, n * 4) : r;
  double a0 = 0.0, a1 = 0.0;
  if (d.vec) {
    // A pass covers 4 loads of kStride rows; its base is wave-uniform, so
    // the loop is too.  Groups past n read zeros (resource range), add +0.0
    // to the sums and their stores are dropped: each lane adds its groups in
    // row order, as a loop over its own groups would.
    constexpr int kStride = 64 * kGroup;  // elements per wave per load
    const int64_t lo = static_cast<int64_t>(lane) * kGroup;
    for (int64_t e0 = 0; e0 < n; e0 += 4 * kStride) {
      u32x4 v[4];
#pragma unroll
      for (int b = 0; b < 4; ++b)
        v[b] = buf_b128<kAuxScore>(r, static_cast<uint32_t>((e0 + b * kStride + lo) * 2), 0);
      if (st) {
#pragma unroll
        for (int b = 0; b < 4; ++b)
          buf_put_b128<kAuxAFirst>(v[b], rS, static_cast<uint32_t>((e0 + b * kStride + lo) * 2), 0);
      }
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        float f[kGroup];
        widen8(v[b], f);
#pragma unroll
        for (int c = 0; c < kGroup; c += 2) {
          a0 = __builtin_fma(static_cast<double>(f[c]), static_cast<double>(f[c]), a0);
          a1 = __builtin_fma(static_cast<double>(f[c + 1]), static_cast<double>(f[c + 1]), a1);
        }
        if constexpr (OUT == 2) {
          // The hand-over in whole lines.  Lane l holds elements 8l .. 8l+7
          // of this load's 512; it stores elements 4l .. 4l+3 and 256+4l ..
          // 256+4l+3, held by lanes l/2 and 32 + l/2 (their words 2(l&1)
          // and 2(l&1)+1), so that each store of the wave fills 1 KiB.  (A
          // lane storing its own 8 values fills half of every line with each
          // of two stores: non-temporal, each half reached HBM on its own.)
          const uint32_t w[4] = {v[b].x, v[b].y, v[b].z, v[b].w};
          uint32_t x[4], y[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            x[k] = static_cast<uint32_t>(__shfl(static_cast<int>(w[k]), lane >> 1, 64));
            y[k] = static_cast<uint32_t>(__shfl(static_cast<int>(w[k]), 32 + (lane >> 1), 64));
          }
          const bool odd = lane & 1;
          u32x2 qa, qb;
          qa.x = odd ? x[2] : x[0];
          qa.y = odd ? x[3] : x[1];
          qb.x = odd ? y[2] : y[0];
          qb.y = odd ? y[3] : y[1];
          float fa[kQuad], fb[kQuad];
          widen4(qa, fa);
          widen4(qb, fb);
#pragma unroll
          for (int c = 0; c < kQuad; ++c) {
            fa[c] = fa[c] * scale;
            fb[c] = fb[c] * scale;
          }
          const int64_t seg = e0 + b * kStride + kQuad * lane;
          f32x4_store<kAuxWO>(rO, static_cast<uint32_t>(seg * 4), fa);
          f32x4_store<kAuxWO>(rO, static_cast<uint32_t>((seg + kStride / 2) * 4), fb);
        }
      }
    }
  } else {
    for (int64_t e = lane; e < n; e += 64) {
      const uint16_t gb = buf_u16<kAuxScore>(r, static_cast<uint32_t>(e * 2), 0);
      if (st) buf_put_u16<kAuxAFirst>(gb, rS, static_cast<uint32_t>(e * 2), 0);
      const float g = widen_bf16(gb);
      if constexpr (OUT == 2) buf_put_f32<kAuxWO>(g * scale, rO, static_cast<uint32_t>(e * 4), 0);
      const double x = static_cast<double>(g);
      a0 = __builtin_fma(x, x, a0);
    }
  }
  double s = a0 + a1;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) d.norms[j] = static_cast<float>(s);
}

// ---------------------------------------------------------------------------
// a3-a5: fused Adam (selected channels) and pack (unselected channels).
// ---------------------------------------------------------------------------

// kCmPend: read from the store like kCmPrev, then the owed deferred step
// with gradient pd.scale * (row rPA of the previous interval's sums).
enum CmSrc { kCmInplace = 0, kCmPrev, kCmInitW, kCmInitMaster, kCmPend };

// Adam over one chunk of channel j (slot r), vector path (QPT quads per
// lane).  SRC picks where (p, m, v) come from; rS* are the source rows (the
// slot's own rows in place).
template <int SRC, int QPT, bool STATS>
__device__ __forceinline__ void cm_adam_vec(rsrc_t rG, rsrc_t rP, rsrc_t rM, rsrc_t rV,
                                            rsrc_t rW, rsrc_t rSP, rsrc_t rSM, rsrc_t rSV,
                                            rsrc_t rI, const AdamK& c, double& ss,
                                            rsrc_t rPA = rsrc_t(), const Pending* pd = nullptr) {
  const int tid = threadIdx.x;
  float g[QPT][kQuad], p[QPT][kQuad], m[QPT][kQuad], v[QPT][kQuad];
  u32x2 gv[QPT];
#pragma unroll
  for (int q = 0; q < QPT; ++q) gv[q] = buf_b64<kAuxRO>(rG, quad_elem(q, tid) * 2, 0);
#pragma unroll
  for (int q = 0; q < QPT; ++q) {
    const uint32_t e = quad_elem(q, tid);
    if constexpr (SRC == kCmInplace || SRC == kCmPrev || SRC == kCmPend) {
      f32x4_load<kAuxRMW>(rSP, e * 4, p[q]);
      f32x4_load<kAuxRMW>(rSM, e * 4, m[q]);
      f32x4_load<kAuxRMW>(rSV, e * 4, v[q]);
      if constexpr (SRC == kCmPend) {
        f32x4_load<kAuxRO>(rPA, e * 4, g[q]);
#pragma unroll
        for (int i = 0; i < kQuad; ++i) adam_step(g[q][i] * pd->scale, p[q][i], m[q][i], v[q][i], pd->c);
      }
    } else {
      if constexpr (SRC == kCmInitMaster) f32x4_load<kAuxRO>(rI, e * 4, p[q]);
      else widen4(buf_b64<kAuxRO>(rI, e * 2, 0), p[q]);
#pragma unroll
      for (int i = 0; i < kQuad; ++i) m[q][i] = v[q][i] = 0.0f;
    }
  }
#pragma unroll
  for (int q = 0; q < QPT; ++q) {
    widen4(gv[q], g[q]);
    if constexpr (STATS) sum_squares(g[q], ss);
#pragma unroll
    for (int i = 0; i < kQuad; ++i) adam_step(g[q][i], p[q][i], m[q][i], v[q][i], c);
    const uint32_t e = quad_elem(q, tid);
    f32x4_store<kAuxRMW>(rP, e * 4, p[q]);
    f32x4_store<kAuxRMW>(rM, e * 4, m[q]);
    f32x4_store<kAuxRMW>(rV, e * 4, v[q]);
    buf_put_b64<kAuxW>(narrow4(p[q]), rW, e * 2, 0);
  }
}

// Element-wise fallback of the same update (any n, any alignment).
template <int SRC, bool STATS>
__device__ __forceinline__ void cm_adam_elem(rsrc_t rG, rsrc_t rP, rsrc_t rM, rsrc_t rV,
                                             rsrc_t rW, rsrc_t rSP, rsrc_t rSM, rsrc_t rSV,
                                             rsrc_t rI, const AdamK& c, int64_t len, double& ss,
                                             rsrc_t rPA = rsrc_t(), const Pending* pd = nullptr) {
  for (int64_t e = threadIdx.x; e < len; e += kThreads) {
    const uint32_t o = static_cast<uint32_t>(e);
    const float g = widen_bf16(buf_u16<kAuxRO>(rG, o * 2, 0));
    if constexpr (STATS) ss = __builtin_fma(static_cast<double>(g), static_cast<double>(g), ss);
    float p, m, v;
    if constexpr (SRC == kCmInplace || SRC == kCmPrev || SRC == kCmPend) {
      p = buf_f32<kAuxRMW>(rSP, o * 4, 0);
      m = buf_f32<kAuxRMW>(rSM, o * 4, 0);
      v = buf_f32<kAuxRMW>(rSV, o * 4, 0);
      if constexpr (SRC == kCmPend)
        adam_step(buf_f32<kAuxRO>(rPA, o * 4, 0) * pd->scale, p, m, v, pd->c);
    } else {
      p = (SRC == kCmInitMaster) ? buf_f32<kAuxRO>(rI, o * 4, 0) : widen_bf16(buf_u16<kAuxRO>(rI, o * 2, 0));
      m = v = 0.0f;
    }
    adam_step(g, p, m, v, c);
    buf_put_f32<kAuxRMW>(p, rP, o * 4, 0);
    buf_put_f32<kAuxRMW>(m, rM, o * 4, 0);
    buf_put_f32<kAuxRMW>(v, rV, o * 4, 0);
    buf_put_u16<kAuxW>(round_bf16(p), rW, o * 2, 0);
  }
}

// HAND (the last step of an interval, fused hand-over): the new sums are not
// stored back; scale * sum goes to the channel's row of the hand-over
// buffer (rOut) instead -- the same two fp32 operations as accumulating and
// then unpacking.
//
// A16 (the packed buffer's bf16 first-step stage, rA16): 1 -- the first step
// stores its values, the widened gradient itself and so exactly a bf16, as
// the gradient's own bits into the stage instead of fp32 into A; 2 -- the
// second step reads the previous values from the stage (widened, the same
// fp32 values) instead of from A.
template <bool FIRST, int QPT, bool STATS, bool HAND = false, int A16 = 0>
__device__ __forceinline__ void cm_pack_vec(rsrc_t rG, rsrc_t rA, double& ss,
                                            rsrc_t rOut = rsrc_t(), float scale = 1.0f,
                                            rsrc_t rA16 = rsrc_t()) {
  const int tid = threadIdx.x;
  u32x2 gv[QPT];
  float a[QPT][kQuad];
#pragma unroll
  for (int q = 0; q < QPT; ++q) gv[q] = buf_b64<kAuxRO>(rG, quad_elem(q, tid) * 2, 0);
  if constexpr (!FIRST) {
    if constexpr (A16 == 2) {
#pragma unroll
      for (int q = 0; q < QPT; ++q) widen4(buf_b64<kAuxRO>(rA16, quad_elem(q, tid) * 2, 0), a[q]);
    } else {
#pragma unroll
      for (int q = 0; q < QPT; ++q) f32x4_load<kAuxRMW>(rA, quad_elem(q, tid) * 4, a[q]);
    }
  }
#pragma unroll
  for (int q = 0; q < QPT; ++q) {
    float g[kQuad];
    widen4(gv[q], g);
#pragma unroll
    for (int i = 0; i < kQuad; ++i) a[q][i] = FIRST ? g[i] : a[q][i] + g[i];
    if constexpr (STATS) sum_squares(a[q], ss);
    if constexpr (HAND) {
#pragma unroll
      for (int i = 0; i < kQuad; ++i) a[q][i] = a[q][i] * scale;
      f32x4_store<kAuxWO>(rOut, quad_elem(q, tid) * 4, a[q]);
    } else if constexpr (FIRST && A16 == 1) {
      buf_put_b64<kAuxAFirst>(gv[q], rA16, quad_elem(q, tid) * 2, 0);
    } else {
      f32x4_store<FIRST ? kAuxAFirst : kAuxRMW>(rA, quad_elem(q, tid) * 4, a[q]);
    }
  }
}

template <bool FIRST, bool STATS, bool HAND = false, int A16 = 0>
__device__ __forceinline__ void cm_pack_elem(rsrc_t rG, rsrc_t rA, int64_t len, double& ss,
                                             rsrc_t rOut = rsrc_t(), float scale = 1.0f,
                                             rsrc_t rA16 = rsrc_t()) {
  for (int64_t e = threadIdx.x; e < len; e += kThreads) {
    const uint32_t o = static_cast<uint32_t>(e);
    const uint16_t gb = buf_u16<kAuxRO>(rG, o * 2, 0);
    const float g = widen_bf16(gb);
    float a = g;
    if constexpr (!FIRST) {
      if constexpr (A16 == 2) a = widen_bf16(buf_u16<kAuxRO>(rA16, o * 2, 0)) + g;
      else a = buf_f32<kAuxRMW>(rA, o * 4, 0) + g;
    }
    if constexpr (STATS) ss = __builtin_fma(static_cast<double>(a), static_cast<double>(a), ss);
    if constexpr (HAND) buf_put_f32<kAuxWO>(a * scale, rOut, o * 4, 0);
    else if constexpr (FIRST && A16 == 1) buf_put_u16<kAuxAFirst>(gb, rA16, o * 2, 0);
    else buf_put_f32<FIRST ? kAuxAFirst : kAuxRMW>(a, rA, o * 4, 0);
  }
}

// The vector paths at a matrix's quads per lane: cm_qpt (kCmQpt / 2 or
// kCmQpt) in the full-grid passes; ONE: one quad (the selected-only Adam
// grid).
template <int SRC, bool STATS, bool ONE = false>
__device__ __forceinline__ void cm_adam_vec_any(int qpt, rsrc_t rG, rsrc_t rP, rsrc_t rM,
                                                rsrc_t rV, rsrc_t rW, rsrc_t rSP, rsrc_t rSM,
                                                rsrc_t rSV, rsrc_t rI, const AdamK& c,
                                                double& ss, rsrc_t rPA = rsrc_t(),
                                                const Pending* pd = nullptr) {
  if constexpr (ONE)
    cm_adam_vec<SRC, 1, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss, rPA, pd);
  else if (qpt >= kCmQpt)
    cm_adam_vec<SRC, kCmQpt, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss, rPA, pd);
  else
    cm_adam_vec<SRC, kCmQpt / 2, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss, rPA, pd);
}

template <bool FIRST, bool STATS, bool HAND = false, int A16 = 0>
__device__ __forceinline__ void cm_pack_vec_any(int qpt, rsrc_t rG, rsrc_t rA, double& ss,
                                                rsrc_t rOut = rsrc_t(), float scale = 1.0f,
                                                rsrc_t rA16 = rsrc_t()) {
  if (qpt >= kCmQpt)
    cm_pack_vec<FIRST, kCmQpt, STATS, HAND, A16>(rG, rA, ss, rOut, scale, rA16);
  else
    cm_pack_vec<FIRST, kCmQpt / 2, STATS, HAND, A16>(rG, rA, ss, rOut, scale, rA16);
}

// HAND: a selected channel's row of the hand-over buffer is +0.0.
__device__ __forceinline__ void cm_zero_rows(const DevMat& d, rsrc_t rOut, int64_t len) {
  if (d.vec) {
    const float z[kQuad] = {0.f, 0.f, 0.f, 0.f};
    for (int64_t g = threadIdx.x; g * kQuad < len; g += kThreads)
      f32x4_store<kAuxWO>(rOut, static_cast<uint32_t>(g * kQuad * 4), z);
  } else {
    for (int64_t e = threadIdx.x; e < len; e += kThreads)
      buf_put_f32<kAuxWO>(0.0f, rOut, static_cast<uint32_t>(e) * 4, 0);
  }
}

// Swap-out of one chunk of a channel that left the selection: its previous
// compact (p, m, v) rows are copied to its rows of the full-state store.
__device__ __forceinline__ void cm_swap_out(const DevMat& d, int64_t j, int64_t w, int64_t e0,
                                            int64_t len) {
  const uint64_t pm = uniform_u64(d.prev_mask[w]);
  if (!((pm >> (j & 63)) & 1ull)) return;
  const int64_t ro = static_cast<int64_t>(uniform_i32(d.prev_prefix[w])) +
                     __popcll(pm & ((uint64_t(1) << (j & 63)) - 1));
  const rsrc_t src[3] = {make_rsrc(d.prev_P + ro * d.ld_prev + e0, len * 4),
                         make_rsrc(d.prev_M + ro * d.ld_prev + e0, len * 4),
                         make_rsrc(d.prev_V + ro * d.ld_prev + e0, len * 4)};
  const rsrc_t dst[3] = {make_rsrc(d.st_P + j * d.ld_store + e0, len * 4),
                         make_rsrc(d.st_M + j * d.ld_store + e0, len * 4),
                         make_rsrc(d.st_V + j * d.ld_store + e0, len * 4)};
  if (d.vec) {
    for (int64_t g = threadIdx.x; g * kQuad < len; g += kThreads) {
      const uint32_t o = static_cast<uint32_t>(g * kQuad * 4);
#pragma unroll
      for (int a = 0; a < 3; ++a) {
        float f[kQuad];
        f32x4_load<kAuxRO>(src[a], o, f);
        f32x4_store<kAuxWO>(dst[a], o, f);
      }
    }
  } else {
    for (int64_t e = threadIdx.x; e < len; e += kThreads) {
      const uint32_t o = static_cast<uint32_t>(e) * 4;
#pragma unroll
      for (int a = 0; a < 3; ++a) buf_put_f32<kAuxWO>(buf_f32<kAuxRO>(src[a], o, 0), dst[a], o, 0);
    }
  }
}

// The sum over steps of an interval whose unselected gradients stayed in
// their slots: rows [e0, e0 + len) of channel j of the kept gradients of
// entries s_first .. h.n - 1 of h (oldest first), then of this step's (rG),
// added in step order in fp32 (the accumulation's own sequence, so the
// same bits as packing every step).  STATS: ss += the squares of the sums,
// in fp64; WRITE: scale times the sums to rOut.
template <int QPT, bool STATS, bool WRITE>
__device__ __forceinline__ void cm_interval_sum_vec(const HistTable& h, int32_t s_first, int32_t q,
                                                    int64_t j, int64_t e0, int64_t len,
                                                    rsrc_t rG, rsrc_t rOut, float scale,
                                                    double& ss) {
  const int tid = threadIdx.x;
  constexpr int kBatch = 4;  // steps whose rows are loaded before they are added
  float a[QPT][kQuad];
  const int32_t steps = h.n - s_first + 1;  // the kept steps, then this one
  for (int32_t s0 = 0; s0 < steps; s0 += kBatch) {
    u32x2 gv[kBatch][QPT];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int32_t s = s0 + b;
      if (s < steps) {
        rsrc_t r = rG;
        if (s < steps - 1) {
          const auto& hd = const_table(h.mats[s_first + s])[q];
          r = make_rsrc(hd.grad + j * hd.ld_grad + e0, len * 2);
        }
#pragma unroll
        for (int p = 0; p < QPT; ++p) gv[b][p] = buf_b64<kAuxRO>(r, quad_elem(p, tid) * 2, 0);
      }
    }
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int32_t s = s0 + b;
      if (s < steps) {
#pragma unroll
        for (int p = 0; p < QPT; ++p) {
          float g[kQuad];
          widen4(gv[b][p], g);
#pragma unroll
          for (int i = 0; i < kQuad; ++i) a[p][i] = s == 0 ? g[i] : a[p][i] + g[i];
        }
      }
    }
  }
#pragma unroll
  for (int p = 0; p < QPT; ++p) {
    if constexpr (STATS) sum_squares(a[p], ss);
    if constexpr (WRITE) {
#pragma unroll
      for (int i = 0; i < kQuad; ++i) a[p][i] = a[p][i] * scale;
      f32x4_store<kAuxWO>(rOut, quad_elem(p, tid) * 4, a[p]);
    }
  }
}

template <bool STATS, bool WRITE>
__device__ __forceinline__ void cm_interval_sum_elem(const HistTable& h, int32_t s_first,
                                                     int32_t q, int64_t j, int64_t e0,
                                                     int64_t len, rsrc_t rG, rsrc_t rOut,
                                                     float scale, double& ss) {
  const int32_t steps = h.n - s_first + 1;
  for (int64_t e = threadIdx.x; e < len; e += kThreads) {
    const uint32_t o = static_cast<uint32_t>(e);
    float a = 0.0f;
    for (int32_t s = 0; s < steps; ++s) {
      rsrc_t r = rG;
      if (s < steps - 1) {
        const auto& hd = const_table(h.mats[s_first + s])[q];
        r = make_rsrc(hd.grad + j * hd.ld_grad + e0, len * 2);
      }
      const float g = widen_bf16(buf_u16<kAuxRO>(r, o * 2, 0));
      a = s == 0 ? g : a + g;
    }
    if constexpr (STATS) ss = __builtin_fma(static_cast<double>(a), static_cast<double>(a), ss);
    if constexpr (WRITE) buf_put_f32<kAuxWO>(a * scale, rOut, o * 4, 0);
  }
}

// STATS (fused Adam + pack only): every wave also sums, in fp64, the squares
// of the values its lanes handled -- the gradient of a selected channel, the
// new accumulated value of an unselected one -- after a fixed xor butterfly,
// and writes that partial to zs[zs_off + (j * cm_nch + chunk) * 4 + wave].
// The partials of a channel are combined in a fixed order by the Zen-auto
// finalize kernel; no barriers, no atomics.
//
// HAND (fused Adam + pack only, the last step of an interval): the hand-over
// is written instead of the packed sums -- out row j = scale * (A + g) for an
// unselected channel, +0.0 for a selected one -- and the packed buffer is
// left as it was (it is overwritten when the next interval starts).  With
// STATS (Zen-auto, an interval the caller ends at this step) the statistics
// are those of the new sums, before the scale.
//
// PEND (fused Adam + pack in kRemap against the store, with or without
// STATS): a channel that
// enters the selection takes the owed deferred step pd first (its row of
// pend_acc is its slot among the previous selection's unselected channels:
// j minus the previously selected channels below j).
//
// SELG (Adam only, no store): the grid covers the selected channels only,
// block -> (selected slot r, row chunk), channel j = sel_idx[r]; the
// unselected channels would have nothing to do.
#ifdef ZF_CM_WAVES_PER_EU
#define ZF_CM_UPDATE_ATTR __attribute__((amdgpu_waves_per_eu(ZF_CM_WAVES_PER_EU)))
#else
#define ZF_CM_UPDATE_ATTR
#endif
//
// PH: the interval phase as a compile-time constant (1: an interval's first
// step, 2: its second, 3: a later step), or 0 to take it from `first`.  The
// fused launches of the fixed schedule pass it, so that each phase is a
// kernel of its own (its own code, its own name in a profile).
template <bool BATCHED, bool ADAM, bool PACK, bool STATS, bool HAND, bool PEND, bool SELG,
          int PH = 0, bool DEFP = false>
__global__ __launch_bounds__(kThreads) ZF_CM_UPDATE_ATTR void cm_update_kernel(const DevMat* __restrict__ mats,
                                                            const int64_t* __restrict__ off,
                                                            int32_t nmats, DevMat one, AdamK c,
                                                            int32_t mode, int32_t first,
                                                            double* __restrict__ zs, float scale,
                                                            Pending pd,
                                                            const ZenState* __restrict__ zst,
                                                            HistTable h) {
  static_assert(!SELG || (ADAM && !PACK && !STATS && !PEND), "selected-only grid");
  static_assert(!DEFP || (BATCHED && ADAM && PACK && STATS && !PEND && !SELG && PH == 0),
                "deferred packing under Zen-auto on the device");
  // the phase: a compile-time constant, the caller's, or (Zen-auto with the
  // interval driven on the device) 1 after a refresh or an ended interval,
  // else the interval's length so far + 1
  int32_t ph = PH != 0 ? PH : first;
  int32_t pos = ph;
  if (PH == 0 && zst != nullptr) {
    pos = (mode != kInplace || zst->ended) ? 1 : zst->length + 1;
    ph = pos < 3 ? pos : 3;
    // HAND (an interval the caller ends at this step): scale = fp32(1 /
    // length), a correctly rounded fp32 division
    if constexpr (HAND) scale = 1.0f / static_cast<float>(pos);
  }
  int64_t local;
  int32_t q;
  const DevMat& d = get_mat<BATCHED>(mats, off, nmats, one, local, q);
  // SELG: one quad per lane, cm_snch chunks per channel; else cm_qpt quads
  const int32_t qpt = SELG ? 1 : d.cm_qpt;
  const int64_t nch = SELG ? d.cm_snch : d.cm_nch;
  const int64_t chunk = static_cast<int64_t>(qpt) * kThreads * kQuad;
  int64_t j, r;
  bool sel;
  if constexpr (SELG) {
    r = local / nch;
    // the channel comes from the caller's selection: kept inside the matrix
    // whatever it holds, so that every address stays in its buffer
    j = min(max(static_cast<int64_t>(uniform_i32(d.sel_idx[r])), int64_t(0)), d.m - 1);
    sel = true;
  } else {
    j = local / nch;
    const uint64_t mj = uniform_u64(d.mask[j >> 6]);
    sel = (mj >> (j & 63)) & 1ull;
    r = static_cast<int64_t>(uniform_i32(d.prefix[j >> 6])) +
        __popcll(mj & ((uint64_t(1) << (j & 63)) - 1));
  }
  const int64_t ci = local % nch;
  const int64_t e0 = ci * chunk;
  const int64_t len = min(chunk, d.n - e0);
  const int64_t w = j >> 6;
  const rsrc_t rG = make_rsrc(d.grad + j * d.ld_grad + e0, len * 2);
  double ss = 0.0;

  if (!sel) {
    if (mode == kRemap && d.st_P != nullptr) cm_swap_out(d, j, w, e0, len);
    if constexpr (DEFP) {
      // deferred packing: the gradient stays in its slot.  The statistics
      // are taken on the interval's running sum, the sum of its kept steps
      // (the last pos - 1 entries of h) and this one's; HAND writes scale
      // times that sum to the hand-over.  Nothing else is written.
      const int32_t kept = min(max(pos - 1, 0), h.n);
      const rsrc_t rOut = HAND ? make_rsrc(d.out + j * d.ld_out + e0, len * 4) : rG;
      if (d.vec) {
        if (d.cm_qpt >= kCmQpt)
          cm_interval_sum_vec<kCmQpt, true, HAND>(h, h.n - kept, q, j, e0, len, rG, rOut, scale,
                                                   ss);
        else
          cm_interval_sum_vec<kCmQpt / 2, true, HAND>(h, h.n - kept, q, j, e0, len, rG, rOut,
                                                       scale, ss);
      } else {
        cm_interval_sum_elem<true, HAND>(h, h.n - kept, q, j, e0, len, rG, rOut, scale, ss);
      }
    } else if constexpr (PACK) {
      const int64_t u = j - r;
      const rsrc_t rA = make_rsrc(d.acc + u * d.ld_acc + e0, len * 4);
      // the bf16 first-step stage (row j, channel-indexed): ph == 1 on an
      // interval's first step, 2 on its second (a matrix without a stage
      // takes 2 as any later step)
      const bool a16 = d.acc1 != nullptr;
      const rsrc_t rA16 = a16 ? make_rsrc(d.acc1 + j * d.ld_acc1 + e0, len * 2) : rA;
      if constexpr (HAND) {
        const rsrc_t rOut = make_rsrc(d.out + j * d.ld_out + e0, len * 4);
        if (d.vec) {
          if (ph == 1) cm_pack_vec_any<true, STATS, true>(d.cm_qpt, rG, rA, ss, rOut, scale);
          else if (a16 && ph == 2)
            cm_pack_vec_any<false, STATS, true, 2>(d.cm_qpt, rG, rA, ss, rOut, scale, rA16);
          else cm_pack_vec_any<false, STATS, true>(d.cm_qpt, rG, rA, ss, rOut, scale);
        } else {
          if (ph == 1) cm_pack_elem<true, STATS, true>(rG, rA, len, ss, rOut, scale);
          else if (a16 && ph == 2)
            cm_pack_elem<false, STATS, true, 2>(rG, rA, len, ss, rOut, scale, rA16);
          else cm_pack_elem<false, STATS, true>(rG, rA, len, ss, rOut, scale);
        }
      } else if (d.vec) {
        if (ph == 1) {
          if (a16) cm_pack_vec_any<true, STATS, false, 1>(d.cm_qpt, rG, rA, ss, rsrc_t(), 1.0f, rA16);
          else cm_pack_vec_any<true, STATS>(d.cm_qpt, rG, rA, ss);
        } else if (a16 && ph == 2) {
          cm_pack_vec_any<false, STATS, false, 2>(d.cm_qpt, rG, rA, ss, rsrc_t(), 1.0f, rA16);
        } else {
          cm_pack_vec_any<false, STATS>(d.cm_qpt, rG, rA, ss);
        }
      } else {
        if (ph == 1) {
          if (a16) cm_pack_elem<true, STATS, false, 1>(rG, rA, len, ss, rsrc_t(), 1.0f, rA16);
          else cm_pack_elem<true, STATS>(rG, rA, len, ss);
        } else if (a16 && ph == 2) {
          cm_pack_elem<false, STATS, false, 2>(rG, rA, len, ss, rsrc_t(), 1.0f, rA16);
        } else {
          cm_pack_elem<false, STATS>(rG, rA, len, ss);
        }
      }
    }
  } else if constexpr (ADAM) {
    const rsrc_t rP = make_rsrc(d.P + r * d.ld_state + e0, len * 4);
    const rsrc_t rM = make_rsrc(d.M + r * d.ld_state + e0, len * 4);
    const rsrc_t rV = make_rsrc(d.V + r * d.ld_state + e0, len * 4);
    const rsrc_t rW = make_rsrc(d.weight + j * d.ld_weight + e0, len * 2);
    int src = kCmInplace;
    rsrc_t rSP = rP, rSM = rM, rSV = rV, rI = rW;
    int64_t ro = 0;  // previously selected channels below j
    if (mode == kRemap) {
      const uint64_t pm = uniform_u64(d.prev_mask[w]);
      ro = static_cast<int64_t>(uniform_i32(d.prev_prefix[w])) +
           __popcll(pm & ((uint64_t(1) << (j & 63)) - 1));
      if ((pm >> (j & 63)) & 1ull) {
        rSP = make_rsrc(d.prev_P + ro * d.ld_prev + e0, len * 4);
        rSM = make_rsrc(d.prev_M + ro * d.ld_prev + e0, len * 4);
        rSV = make_rsrc(d.prev_V + ro * d.ld_prev + e0, len * 4);
        src = kCmPrev;
      } else {
        src = d.init_P ? kCmInitMaster : kCmInitW;
      }
    } else if (mode == kInit) {
      src = d.init_P ? kCmInitMaster : kCmInitW;
    }
    if (mode != kInplace && src != kCmPrev && d.st_P != nullptr) {
      // swap-in from the full-state store: the same loads as a moved column
      rSP = make_rsrc(d.st_P + j * d.ld_store + e0, len * 4);
      rSM = make_rsrc(d.st_M + j * d.ld_store + e0, len * 4);
      rSV = make_rsrc(d.st_V + j * d.ld_store + e0, len * 4);
      src = PEND ? kCmPend : kCmPrev;
    }
    if (src == kCmInitMaster) rI = make_rsrc(d.init_P + j * d.ld_init + e0, len * 4);
    if (PEND && src == kCmPend) {
      const rsrc_t rPA = make_rsrc(d.pend_acc + (j - ro) * d.ld_pend + e0, len * 4);
      if (d.vec) cm_adam_vec_any<kCmPend, STATS, SELG>(qpt, rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss, rPA, &pd);
      else cm_adam_elem<kCmPend, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, len, ss, rPA, &pd);
    } else if (d.vec) {
      switch (src) {
        case kCmInplace: cm_adam_vec_any<kCmInplace, STATS, SELG>(qpt, rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss); break;
        case kCmPrev: cm_adam_vec_any<kCmPrev, STATS, SELG>(qpt, rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss); break;
        case kCmInitW: cm_adam_vec_any<kCmInitW, STATS, SELG>(qpt, rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss); break;
        default: cm_adam_vec_any<kCmInitMaster, STATS, SELG>(qpt, rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, ss); break;
      }
    } else {
      switch (src) {
        case kCmInplace: cm_adam_elem<kCmInplace, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, len, ss); break;
        case kCmPrev: cm_adam_elem<kCmPrev, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, len, ss); break;
        case kCmInitW: cm_adam_elem<kCmInitW, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, len, ss); break;
        default: cm_adam_elem<kCmInitMaster, STATS>(rG, rP, rM, rV, rW, rSP, rSM, rSV, rI, c, len, ss); break;
      }
    }
    if constexpr (HAND) cm_zero_rows(d, make_rsrc(d.out + j * d.ld_out + e0, len * 4), len);
  }
  if constexpr (STATS) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
    if ((threadIdx.x & 63) == 0)
      zs[d.zs_off + (j * d.cm_nch + ci) * kCmWaves + (threadIdx.x >> 6)] = ss;
  }
}

// ---------------------------------------------------------------------------
// a3-a6 with deferred packing: the interval's last step.  The unselected
// part of each step's gradient stayed where it was written; here it is
// summed, in step order and in fp32 (the accumulation's own sequence), and
// scaled into the hand-over.  A block owns one channel and one chunk of its
// rows, as in the update.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kThreads) void cm_handover_deferred_kernel(
    const DevMat* __restrict__ mats, const int64_t* __restrict__ off, int32_t nmats, AdamK c,
    float scale, HistTable h) {
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  int32_t lo = 0, hi = nmats - 1;
  while (lo < hi) {  // the matrix: largest q with off[q] <= b
    const int32_t mid = (lo + hi + 1) >> 1;
    if (off[mid] <= b) lo = mid; else hi = mid - 1;
  }
  const int32_t q = lo;
  const DevMat& d = mats[q];
  const int64_t local = b - off[q];
  const int64_t chunk = static_cast<int64_t>(d.cm_qpt) * kThreads * kQuad;
  const int64_t j = local / d.cm_nch;
  const int64_t ci = local % d.cm_nch;
  const int64_t e0 = ci * chunk;
  const int64_t len = min(chunk, d.n - e0);
  const uint64_t mj = uniform_u64(d.mask[j >> 6]);
  const bool sel = (mj >> (j & 63)) & 1ull;
  const rsrc_t rG = make_rsrc(d.grad + j * d.ld_grad + e0, len * 2);
  const rsrc_t rOut = make_rsrc(d.out + j * d.ld_out + e0, len * 4);
  double ss = 0.0;
  if (sel) {
    const int64_t r = static_cast<int64_t>(uniform_i32(d.prefix[j >> 6])) +
                      __popcll(mj & ((uint64_t(1) << (j & 63)) - 1));
    const rsrc_t rP = make_rsrc(d.P + r * d.ld_state + e0, len * 4);
    const rsrc_t rM = make_rsrc(d.M + r * d.ld_state + e0, len * 4);
    const rsrc_t rV = make_rsrc(d.V + r * d.ld_state + e0, len * 4);
    const rsrc_t rW = make_rsrc(d.weight + j * d.ld_weight + e0, len * 2);
    if (d.vec)
      cm_adam_vec_any<kCmInplace, false>(d.cm_qpt, rG, rP, rM, rV, rW, rP, rM, rV, rW, c, ss);
    else
      cm_adam_elem<kCmInplace, false>(rG, rP, rM, rV, rW, rP, rM, rV, rW, c, len, ss);
    cm_zero_rows(d, rOut, len);
  } else if (d.vec) {
    if (d.cm_qpt >= kCmQpt)
      cm_interval_sum_vec<kCmQpt, false, true>(h, 0, q, j, e0, len, rG, rOut, scale, ss);
    else
      cm_interval_sum_vec<kCmQpt / 2, false, true>(h, 0, q, j, e0, len, rG, rOut, scale, ss);
  } else {
    cm_interval_sum_elem<false, true>(h, 0, q, j, e0, len, rG, rOut, scale, ss);
  }
}

// ---------------------------------------------------------------------------
// a6: hand-over.  Channel j of the dense buffer is +0.0 when selected, else
// scale times its packed row -- or, STAGE (a one-step interval on a plan with
// the bf16 first-step stage), scale times its widened row of the stage.
// ---------------------------------------------------------------------------

// The hand-over of rows [e0, e0 + len) of channel j, len <= QPT * 256 * 4
// (QPT quads per lane on the vector path).
template <bool STAGE, int QPT>
__device__ __forceinline__ void cm_unpack_rows(const DevMat& d, int64_t j, int64_t e0,
                                               int64_t len, float scale) {
  const int64_t w = j >> 6;
  const uint64_t mw = uniform_u64(d.mask[w]);
  const bool sel = (mw >> (j & 63)) & 1ull;
  const rsrc_t rD = make_rsrc(d.out + j * d.ld_out + e0, len * 4);
  const int tid = threadIdx.x;
  if (sel) {
    const float z[kQuad] = {0.f, 0.f, 0.f, 0.f};
    if (d.vec) {
#pragma unroll
      for (int q = 0; q < QPT; ++q) f32x4_store<kAuxWO>(rD, quad_elem(q, tid) * 4, z);
    } else {
      for (int64_t e = tid; e < len; e += kThreads)
        buf_put_f32<kAuxWO>(0.0f, rD, static_cast<uint32_t>(e) * 4, 0);
    }
    return;
  }
  const int64_t u = j - (static_cast<int64_t>(uniform_i32(d.prefix[w])) +
                         __popcll(mw & ((uint64_t(1) << (j & 63)) - 1)));
  const rsrc_t rA = make_rsrc(d.acc + u * d.ld_acc + e0, len * 4);
  const rsrc_t rS = STAGE ? make_rsrc(d.acc1 + j * d.ld_acc1 + e0, len * 2) : rA;
  if (d.vec) {
    float a[QPT][kQuad];
#pragma unroll
    for (int q = 0; q < QPT; ++q) {
      if constexpr (STAGE) widen4(buf_b64<kAuxRO>(rS, quad_elem(q, tid) * 2, 0), a[q]);
      else f32x4_load<kAuxRO>(rA, quad_elem(q, tid) * 4, a[q]);
    }
#pragma unroll
    for (int q = 0; q < QPT; ++q) {
#pragma unroll
      for (int i = 0; i < kQuad; ++i) a[q][i] = a[q][i] * scale;
      f32x4_store<kAuxWO>(rD, quad_elem(q, tid) * 4, a[q]);
    }
  } else {
    for (int64_t e = tid; e < len; e += kThreads) {
      const uint32_t o = static_cast<uint32_t>(e) * 4;
      const float a = STAGE ? widen_bf16(buf_u16<kAuxRO>(rS, static_cast<uint32_t>(e) * 2, 0))
                            : buf_f32<kAuxRO>(rA, o, 0);
      buf_put_f32<kAuxWO>(a * scale, rD, o, 0);
    }
  }
}

// The same with deferred packing: rows [e0, e0 + len) of channel j of the
// hand-over are scale times the interval's sum, its kept steps (the last
// `kept` entries of h) and this plan's gradient, or +0.0 when selected.
template <int QPT>
__device__ __forceinline__ void cm_handover_rows_deferred(const DevMat& d, int32_t q, int64_t j,
                                                          int64_t e0, int64_t len, float scale,
                                                          const HistTable& h, int32_t kept) {
  const uint64_t mw = uniform_u64(d.mask[j >> 6]);
  const rsrc_t rD = make_rsrc(d.out + j * d.ld_out + e0, len * 4);
  const int tid = threadIdx.x;
  if ((mw >> (j & 63)) & 1ull) {
    const float z[kQuad] = {0.f, 0.f, 0.f, 0.f};
    if (d.vec) {
#pragma unroll
      for (int p = 0; p < QPT; ++p) f32x4_store<kAuxWO>(rD, quad_elem(p, tid) * 4, z);
    } else {
      for (int64_t e = tid; e < len; e += kThreads)
        buf_put_f32<kAuxWO>(0.0f, rD, static_cast<uint32_t>(e) * 4, 0);
    }
    return;
  }
  const rsrc_t rG = make_rsrc(d.grad + j * d.ld_grad + e0, len * 2);
  double ss = 0.0;  // (no statistics)
  if (d.vec)
    cm_interval_sum_vec<QPT, false, true>(h, h.n - kept, q, j, e0, len, rG, rD, scale, ss);
  else
    cm_interval_sum_elem<false, true>(h, h.n - kept, q, j, e0, len, rG, rD, scale, ss);
}

// One unpack block's work: channel local / cm_unch, its chunk local %
// cm_unch of kCmUnpackChunk rows.
template <bool STAGE>
__device__ __forceinline__ void cm_unpack_unit(const DevMat& d, int64_t local, float scale) {
  const int64_t j = local / d.cm_unch;
  const int64_t e0 = (local % d.cm_unch) * kCmUnpackChunk;
  const int64_t len = min(static_cast<int64_t>(kCmUnpackChunk), d.n - e0);
  cm_unpack_rows<STAGE, kCmUnpackQpt>(d, j, e0, len, scale);
}

template <bool BATCHED, bool STAGE>
__global__ __launch_bounds__(kThreads) void cm_unpack_kernel(const DevMat* __restrict__ mats,
                                                            const int64_t* __restrict__ off,
                                                            int32_t nmats, DevMat one,
                                                            float scale) {
  int64_t local;
  const DevMat& d = get_mat<BATCHED>(mats, off, nmats, one, local);
  cm_unpack_unit<STAGE>(d, local, scale);
}

// The hand-over of an interval that Zen-auto ended on the device: nothing
// unless zst->ended == 1 (ended, not yet handed over: 2 means the update
// wrote the hand-over itself); then scale = fp32(1 / length) (a correctly rounded
// fp32 division, the value the host passes as fp32(1.0 / length)), from the
// stage after a one-step interval when the plan keeps one.  A fixed grid
// loops over the table's unpack blocks, so that a step that does not end
// its interval costs one short launch.
//
// DEFP (deferred packing): the interval's sums are taken from the kept
// gradients of its earlier steps (the last length - 1 entries of h) and this
// plan's gradient, as the deferred update would have written them.
template <bool DEFP>
__global__ __launch_bounds__(kThreads) void cm_unpack_zen_kernel(const DevMat* __restrict__ mats,
                                                                const int64_t* __restrict__ off,
                                                                int32_t nmats, int64_t units,
                                                                const ZenState* __restrict__ zst,
                                                                int32_t stage, HistTable h) {
  if (zst->ended != 1) return;
  const int32_t length = zst->length;
  const float scale = 1.0f / static_cast<float>(length);
  const bool from_stage = !DEFP && stage != 0 && length == 1;
  const int32_t kept = DEFP ? min(max(length - 1, 0), h.n) : 0;
  // each block walks one contiguous run of units, the runs in the
  // XCD-aware block order (XCD x covers one contiguous range, as the
  // full-grid passes do)
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t per = (units + gridDim.x - 1) / gridDim.x;
  const int64_t u0 = b * per;
  const int64_t u1 = min(units, u0 + per);
  if (u0 >= u1) return;
  int lo = 0, hi = nmats - 1;
  while (lo < hi) {  // largest q with off[q] <= u0
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= u0) lo = mid; else hi = mid - 1;
  }
  // two consecutive chunks of one channel in one pass (twice the bytes in
  // flight per lane); a lone chunk on its own
  for (int64_t u = u0; u < u1;) {
    while (lo + 1 < nmats && off[lo + 1] <= u) ++lo;
    const DevMat& d = mats[lo];
    const int64_t local = u - off[lo];
    const int64_t j = local / d.cm_unch;
    const int64_t e0 = (local % d.cm_unch) * kCmUnpackChunk;
    const bool pair = u + 1 < u1 && (local + 1) / d.cm_unch == j;
    const int64_t len = min(static_cast<int64_t>(pair ? 2 : 1) * kCmUnpackChunk, d.n - e0);
    if (pair) {
      if constexpr (DEFP) cm_handover_rows_deferred<2 * kCmUnpackQpt>(d, lo, j, e0, len, scale, h, kept);
      else if (from_stage) cm_unpack_rows<true, 2 * kCmUnpackQpt>(d, j, e0, len, scale);
      else cm_unpack_rows<false, 2 * kCmUnpackQpt>(d, j, e0, len, scale);
      u += 2;
    } else {
      if constexpr (DEFP) cm_handover_rows_deferred<kCmUnpackQpt>(d, lo, j, e0, len, scale, h, kept);
      else if (from_stage) cm_unpack_rows<true, kCmUnpackQpt>(d, j, e0, len, scale);
      else cm_unpack_rows<false, kCmUnpackQpt>(d, j, e0, len, scale);
      u += 1;
    }
  }
}

}  // namespace

template <int OUT>
static void launch_cm_colnorm_t(const Table& t, const DevMat& one, dim3 grid, float scale,
                                hipStream_t s) {
  if (t.mats != nullptr)
    hipLaunchKernelGGL((cm_colnorm_kernel<true, OUT>), grid, dim3(kThreads), 0, s, t.mats, t.off,
                       t.nmats, one, scale);
  else
    hipLaunchKernelGGL((cm_colnorm_kernel<false, OUT>), grid, dim3(kThreads), 0, s, t.mats,
                       t.off, t.nmats, one, scale);
}

hipError_t launch_cm_colnorm(const Table& t, const DevMat& one, int64_t blocks, hipStream_t s,
                             int32_t out, float scale) {
  (void)hipGetLastError();
  if (blocks > 0) {
    const dim3 grid(static_cast<uint32_t>(blocks));
    if (out == 1) launch_cm_colnorm_t<1>(t, one, grid, scale, s);
    else if (out == 2) launch_cm_colnorm_t<2>(t, one, grid, scale, s);
    else launch_cm_colnorm_t<0>(t, one, grid, scale, s);
  }
  return hipGetLastError();
}

// LDS reserved (and unused) per update block: caps the blocks resident on a
// CU (160 KiB of LDS per CU) and so the number of concurrent HBM streams.
#ifndef ZF_CM_UPDATE_LDS
#define ZF_CM_UPDATE_LDS 0
#endif
constexpr unsigned kCmUpdateLds = ZF_CM_UPDATE_LDS;

template <bool ADAM, bool PACK, bool STATS, bool HAND, bool PEND = false, bool SELG = false,
          int PH = 0>
static void launch_cm_update_t(const Table& t, const DevMat& one, dim3 grid, const AdamK& c,
                               int32_t mode, int32_t first, double* zs, float scale,
                               hipStream_t s, const Pending& pd = Pending{},
                               const ZenState* zst = nullptr) {
  if (t.mats != nullptr)
    hipLaunchKernelGGL((cm_update_kernel<true, ADAM, PACK, STATS, HAND, PEND, SELG, PH>), grid,
                       dim3(kThreads), kCmUpdateLds, s, t.mats, t.off, t.nmats, one, c, mode,
                       first, zs, scale, pd, zst, HistTable{});
  else
    hipLaunchKernelGGL((cm_update_kernel<false, ADAM, PACK, STATS, HAND, PEND, SELG, PH>), grid,
                       dim3(kThreads), kCmUpdateLds, s, t.mats, t.off, t.nmats, one, c, mode,
                       first, zs, scale, pd, zst, HistTable{});
}

// The fused update (HAND: with the hand-over) with its interval phase as a
// compile-time constant.
template <bool HAND>
static void launch_cm_fused_phase(const Table& t, const DevMat& one, dim3 grid, const AdamK& c,
                                  int32_t mode, int32_t first, float scale, hipStream_t s) {
  if (first == 1)
    launch_cm_update_t<true, true, false, HAND, false, false, 1>(t, one, grid, c, mode, first,
                                                                 nullptr, scale, s);
  else if (first == 2)
    launch_cm_update_t<true, true, false, HAND, false, false, 2>(t, one, grid, c, mode, first,
                                                                 nullptr, scale, s);
  else
    launch_cm_update_t<true, true, false, HAND, false, false, 3>(t, one, grid, c, mode, first,
                                                                 nullptr, scale, s);
}

hipError_t launch_cm_adam_selected_grid(const Table& t, const DevMat& one, int64_t blocks,
                                        const AdamK& c, int32_t mode, hipStream_t s,
                                        bool zero_out) {
  (void)hipGetLastError();
  if (blocks <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (zero_out)
    launch_cm_update_t<true, false, false, true, false, true>(t, one, grid, c, mode, 0, nullptr,
                                                              1.0f, s);
  else
    launch_cm_update_t<true, false, false, false, false, true>(t, one, grid, c, mode, 0, nullptr,
                                                               1.0f, s);
  return hipGetLastError();
}

hipError_t launch_cm_update(const Table& t, const DevMat& one, int64_t blocks, const AdamK& c,
                            int32_t mode, int32_t first, bool adam, bool pack, double* zs,
                            bool handover, float scale, hipStream_t s, const Pending* pend,
                            const ZenState* zst) {
  (void)hipGetLastError();
  if (blocks <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if ((zs != nullptr || handover) && !(adam && pack)) return hipErrorInvalidValue;
  if (zs != nullptr && handover && zst == nullptr) return hipErrorInvalidValue;
  if (zst != nullptr && (zs == nullptr || pend != nullptr)) return hipErrorInvalidValue;
  if (pend != nullptr) {
    if (!(adam && pack) || handover || mode != kRemap) return hipErrorInvalidValue;
    if (zs != nullptr)
      launch_cm_update_t<true, true, true, false, true>(t, one, grid, c, mode, first, zs, 1.0f, s,
                                                        *pend);
    else
      launch_cm_update_t<true, true, false, false, true>(t, one, grid, c, mode, first, nullptr,
                                                         1.0f, s, *pend);
  } else if (zs != nullptr && handover) {
    // Zen-auto on the device, an interval the caller ends here: the
    // hand-over fused, its scale from the interval's length
    launch_cm_update_t<true, true, true, true>(t, one, grid, c, mode, first, zs, 1.0f, s,
                                               Pending{}, zst);
  } else if (zs != nullptr) {
    launch_cm_update_t<true, true, true, false>(t, one, grid, c, mode, first, zs, 1.0f, s,
                                                Pending{}, zst);
  } else if (handover) {
    launch_cm_fused_phase<true>(t, one, grid, c, mode, first, scale, s);
  } else if (adam && pack) {
    launch_cm_fused_phase<false>(t, one, grid, c, mode, first, 1.0f, s);
  } else if (adam) {
    launch_cm_update_t<true, false, false, false>(t, one, grid, c, mode, first, nullptr, 1.0f, s);
  } else if (pack) {
    launch_cm_update_t<false, true, false, false>(t, one, grid, c, mode, first, nullptr, 1.0f, s);
  }
  return hipGetLastError();
}

template <bool STAGE>
static void launch_cm_unpack_t(const Table& t, const DevMat& one, dim3 grid, float scale,
                               hipStream_t s) {
  if (t.mats != nullptr)
    hipLaunchKernelGGL((cm_unpack_kernel<true, STAGE>), grid, dim3(kThreads), 0, s, t.mats, t.off,
                       t.nmats, one, scale);
  else
    hipLaunchKernelGGL((cm_unpack_kernel<false, STAGE>), grid, dim3(kThreads), 0, s, t.mats,
                       t.off, t.nmats, one, scale);
}

hipError_t launch_cm_handover_deferred(const Table& t, const DevMat& one, int64_t blocks,
                                       const AdamK& c, float scale, const HistTable& h,
                                       hipStream_t s) {
  (void)hipGetLastError();
  (void)one;
  if (blocks <= 0 || t.mats == nullptr) return hipSuccess;
  hipLaunchKernelGGL(cm_handover_deferred_kernel, dim3(static_cast<uint32_t>(blocks)),
                     dim3(kThreads), 0, s, t.mats, t.off, t.nmats, c, scale, h);
  return hipGetLastError();
}

hipError_t launch_cm_update_zen_deferred(const Table& t, const DevMat& one, int64_t blocks,
                                         const AdamK& c, int32_t mode, double* zs, bool handover,
                                         const HistTable& h, const ZenState* zst,
                                         hipStream_t s) {
  (void)hipGetLastError();
  if (blocks <= 0 || t.mats == nullptr) return hipSuccess;
  if (zs == nullptr || zst == nullptr) return hipErrorInvalidValue;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (handover)
    hipLaunchKernelGGL((cm_update_kernel<true, true, true, true, true, false, false, 0, true>),
                       grid, dim3(kThreads), kCmUpdateLds, s, t.mats, t.off, t.nmats, one, c,
                       mode, 1, zs, 1.0f, Pending{}, zst, h);
  else
    hipLaunchKernelGGL((cm_update_kernel<true, true, true, true, false, false, false, 0, true>),
                       grid, dim3(kThreads), kCmUpdateLds, s, t.mats, t.off, t.nmats, one, c,
                       mode, 1, zs, 1.0f, Pending{}, zst, h);
  return hipGetLastError();
}

constexpr int64_t kCmUnpackZenGrid = 4096;  // 16 blocks per CU

hipError_t launch_cm_unpack_zen(const Table& t, const DevMat& one, int64_t units,
                                const ZenState* zst, bool stage, hipStream_t s) {
  (void)hipGetLastError();
  (void)one;
  if (units <= 0 || t.mats == nullptr) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(units < kCmUnpackZenGrid ? units : kCmUnpackZenGrid));
  hipLaunchKernelGGL(cm_unpack_zen_kernel<false>, grid, dim3(kThreads), 0, s, t.mats, t.off,
                     t.nmats, units, zst, stage ? 1 : 0, HistTable{});
  return hipGetLastError();
}

hipError_t launch_cm_unpack_zen_deferred(const Table& t, int64_t units, const HistTable& h,
                                         const ZenState* zst, hipStream_t s) {
  (void)hipGetLastError();
  if (units <= 0 || t.mats == nullptr) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(units < kCmUnpackZenGrid ? units : kCmUnpackZenGrid));
  hipLaunchKernelGGL(cm_unpack_zen_kernel<true>, grid, dim3(kThreads), 0, s, t.mats, t.off,
                     t.nmats, units, zst, 0, h);
  return hipGetLastError();
}

hipError_t launch_cm_unpack(const Table& t, const DevMat& one, int64_t blocks, float scale,
                            hipStream_t s, bool from_stage) {
  (void)hipGetLastError();
  if (blocks > 0) {
    const dim3 grid(static_cast<uint32_t>(blocks));
    if (from_stage) launch_cm_unpack_t<true>(t, one, grid, scale, s);
    else launch_cm_unpack_t<false>(t, one, grid, scale, s);
  }
  return hipGetLastError();
}

}  // namespace zf
