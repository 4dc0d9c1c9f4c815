// Device helpers shared by the gfx950 kernels of libzf (row-major and
// channel-major): bf16 conversions, wave bit counts, descriptor lookup, raw
// buffer resources and the Adam element update.
#pragma once

#include "zf_internal.hpp"

namespace zf {

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

// A value every lane of the wave holds (loaded from the same address, e.g.
// the selection word of a block's channel) moved to scalar registers.
// Buffer resources built from it are then scalar as the hardware requires,
// instead of being wrapped by the compiler in per-access lane loops.
__device__ __forceinline__ uint64_t uniform_u64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x >> 32));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ int32_t uniform_i32(int32_t x) {
  return __builtin_amdgcn_readfirstlane(x);
}

// A plan's device tables (matrix descriptors, block offsets) are written by
// the host before a launch and only read by the kernels.  Reading one
// through the constant address space lets the compiler use scalar loads:
// the values land in scalar registers without waiting for the vector loads
// in flight, and buffer resources built from them need no per-lane loop.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(4))) T* const_table(const T* p) {
  return (const __attribute__((address_space(4))) T*)(p);
}

// Number of set bits of `mask` at lane positions below the calling lane.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Workgroups are dispatched to the 8 XCDs of the chip round-robin by block
// id.  Remapping the id so that XCD x handles one contiguous range of the
// grid gives each XCD (and its L2) a contiguous address stream, which
// measured 4-5% faster for the streaming passes.  A bijection on [0, B) for
// any B (the first B mod 8 XCDs take one block more).
#ifndef ZF_XCD_REMAP
#define ZF_XCD_REMAP 1
#endif
constexpr int kXcds = 8;

__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t B) {
  if constexpr (ZF_XCD_REMAP == 0) return b;
  const int64_t q = B / kXcds, r = B % kXcds;
  const int64_t x = b % kXcds, i = b / kXcds;
  return x < r ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

// Descriptor of the matrix the (remapped) block belongs to.  BATCHED kernels
// read it from the plan's device table (scalar loads); single-matrix kernels
// take it by value.  Keeping the two apart avoids a generic pointer that
// would turn the descriptor loads into flat vector loads.
template <bool BATCHED>
__device__ __forceinline__ const DevMat& get_mat(const DevMat* __restrict__ mats,
                                                 const int64_t* __restrict__ off, int32_t nmats,
                                                 const DevMat& one, int64_t& local,
                                                 int32_t& index) {
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  if constexpr (!BATCHED) {
    local = b;
    index = 0;
    return one;
  } else {
    int lo = 0, hi = nmats - 1;
    while (lo < hi) {  // largest q with off[q] <= b
      const int mid = (lo + hi + 1) >> 1;
      if (off[mid] <= b) lo = mid; else hi = mid - 1;
    }
    local = b - off[lo];
    index = lo;
    return mats[lo];
  }
}

template <bool BATCHED>
__device__ __forceinline__ const DevMat& get_mat(const DevMat* __restrict__ mats,
                                                 const int64_t* __restrict__ off, int32_t nmats,
                                                 const DevMat& one, int64_t& local) {
  int32_t index;
  return get_mat<BATCHED>(mats, off, nmats, one, local, index);
}

// Raw buffer resources (gfx9 family word 3).  A resource is based at the
// first row a block touches; lanes pass one 32-bit byte offset that is the
// same for every row, the row part goes in the scalar offset.  num_records
// is the exact byte span of the block's rows, so an access outside them is
// dropped by the hardware rather than reaching other memory.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), kRsrcWord3);
}

// Resource over rows [i0, i1) of a row-major [.][ld] array of `width` used
// elements of T per row.
template <typename T>
__device__ __forceinline__ rsrc_t rows_rsrc(const T* base, int64_t i0, int64_t i1, int64_t ld,
                                            int64_t width) {
  const int64_t rows = i1 - i0;
  const int64_t bytes = rows > 0 ? ((rows - 1) * ld + width) * static_cast<int64_t>(sizeof(T)) : 0;
  return make_rsrc(base + i0 * ld, bytes);
}

// Cache policy of a buffer access.  Every stream of the hot path is read or
// written once per kernel, so the kernels mark their traffic non-temporal
// (kStream); kCached is the default policy.
constexpr int kCached = 0;
constexpr int kStream = 2;  // "nt"

template <int AUX = kCached>
__device__ __forceinline__ float buf_f32(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, AUX));
}
template <int AUX = kCached>
__device__ __forceinline__ uint16_t buf_u16(rsrc_t r, uint32_t voff, uint32_t soff) {
  return static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, AUX));
}
template <int AUX = kCached>
__device__ __forceinline__ void buf_put_f32(float v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, voff, soff, AUX);
}
template <int AUX = kCached>
__device__ __forceinline__ void buf_put_u16(uint16_t v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b16(v, r, voff, soff, AUX);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int AUX = kCached>
__device__ __forceinline__ u32x4 buf_b128(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX);
}
template <int AUX = kCached>
__device__ __forceinline__ void buf_put_b128(u32x4 v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, soff, AUX);
}

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

template <int AUX = kCached>
__device__ __forceinline__ u32x2 buf_b64(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, AUX);
}
template <int AUX = kCached>
__device__ __forceinline__ void buf_put_b64(u32x2 v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, voff, soff, AUX);
}

// One Adam/AdamW element update; each line is one fp32 operation (the
// library is compiled without contraction, with correctly rounded sqrt and
// division).
__device__ __forceinline__ void adam_step(float g, float& p, float& m, float& v, const AdamK& c) {
  m = c.b1 * m + c.c1 * g;
  v = c.b2 * v + c.c2 * (g * g);
  const float den = sqrtf(v * c.ib2) + c.eps;
  const float u = (m * c.ib1) / den;
  if (c.wd != 0.0f) p = p - c.wd * p;
  p = p - c.lr * u;
}

}  // namespace zf
