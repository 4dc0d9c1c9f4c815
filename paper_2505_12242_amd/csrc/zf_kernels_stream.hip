// Streaming reference kernels for measurement: the memory access pattern of
// the channel-major update pass with no arithmetic, so that what one MI355X
// reaches with it (read-only, copy, read-modify-write) can be measured in
// the same run as the hot path.  Same building blocks as the update: a
// block owns one contiguous chunk of kProbeVpt x 256 lanes x 16 bytes, raw
// buffer resources over exactly that chunk, 16-byte accesses, the XCD-aware
// block order, non-temporal loads of streams the pass only reads and the
// default policy for written and read-modify-write streams.
#include "zf_device.hpp"

namespace zf {

constexpr int kProbeVpt = 2;  // 16-byte groups per lane, as the update
constexpr int64_t kProbeChunk = int64_t(kProbeVpt) * kThreads * 16;

// KIND 0: read src; KIND 1: copy src to dst; KIND 2: dst ^= key in place.
template <int KIND>
__global__ __launch_bounds__(kThreads) void stream_probe_kernel(const uint8_t* __restrict__ src,
                                                                uint8_t* __restrict__ dst,
                                                                int64_t bytes, uint32_t key) {
  const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t off = b * kProbeChunk;
  const int64_t len = min(kProbeChunk, bytes - off);
  // KIND 0: dst is a 4-byte word (the same for every block); src is unused
  // by KIND 2
  const rsrc_t rs = KIND == 2 ? make_rsrc(dst, 0) : make_rsrc(src + off, len);
  const rsrc_t rd = KIND == 0 ? make_rsrc(dst, 4) : make_rsrc(dst + off, len);
  u32x4 v[kProbeVpt];
#pragma unroll
  for (int q = 0; q < kProbeVpt; ++q) {
    const uint32_t o = static_cast<uint32_t>((q * kThreads + threadIdx.x) * 16);
    v[q] = KIND == 2 ? buf_b128<kCached>(rd, o, 0) : buf_b128<kStream>(rs, o, 0);
  }
  if constexpr (KIND == 0) {
    // keep the loads: fold them into one word, stored (to dst's first word)
    // only if it happens to equal `key`
    uint32_t x = 0;
#pragma unroll
    for (int q = 0; q < kProbeVpt; ++q) x ^= v[q].x ^ v[q].y ^ v[q].z ^ v[q].w;
    if (x == key) __builtin_amdgcn_raw_buffer_store_b32(x, rd, 0, 0, 0);
  } else {
#pragma unroll
    for (int q = 0; q < kProbeVpt; ++q) {
      const uint32_t o = static_cast<uint32_t>((q * kThreads + threadIdx.x) * 16);
      u32x4 w = v[q];
      if constexpr (KIND == 2) {
        w.x ^= key;
        w.y ^= key;
        w.z ^= key;
        w.w ^= key;
      }
      buf_put_b128<kCached>(w, rd, o, 0);
    }
  }
}

int64_t stream_probe_blocks(int64_t bytes) { return (bytes + kProbeChunk - 1) / kProbeChunk; }

hipError_t launch_stream_probe(int32_t kind, const void* src, void* dst, int64_t bytes,
                               uint32_t key, hipStream_t s) {
  (void)hipGetLastError();
  const dim3 grid(static_cast<uint32_t>(stream_probe_blocks(bytes)));
  const auto* sp = static_cast<const uint8_t*>(src);
  auto* dp = static_cast<uint8_t*>(dst);
  if (kind == 0)
    hipLaunchKernelGGL(stream_probe_kernel<0>, grid, dim3(kThreads), 0, s, sp, dp, bytes, key);
  else if (kind == 1)
    hipLaunchKernelGGL(stream_probe_kernel<1>, grid, dim3(kThreads), 0, s, sp, dp, bytes, key);
  else
    hipLaunchKernelGGL(stream_probe_kernel<2>, grid, dim3(kThreads), 0, s, sp, dp, bytes, key);
  return hipGetLastError();
}

}  // namespace zf
