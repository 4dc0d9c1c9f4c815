// Streaming reference kernels for measurement: the memory access pattern of
// the channel-major passes with no arithmetic, so that what one MI355X
// reaches with it (read-only, copy, read-modify-write) can be measured in
// the same run as the hot path.  Same building blocks as the passes: raw
// buffer resources over exactly a block's chunk, 16-byte accesses that a
// wave issues over 1 KiB of consecutive bytes, the XCD-aware block order,
// non-temporal loads and stores of streams only read or only written and
// the default policy for read-modify-write streams.  A block owns one chunk
// of 256 lanes x 16 bytes: of the chunk sizes measured on MI355X (4, 8 and
// 16 KiB per 256-thread block) the fastest for each of the three streams
// (read 7.6, copy 6.5, read-modify-write 6.3 TB/s against 6.9, 5.9 and 5.8
// with 8 KiB).
#include "zf_device.hpp"

namespace zf {

constexpr int kProbeVpt = 1;  // 16-byte groups per lane
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
      if constexpr (KIND == 2) buf_put_b128<kCached>(w, rd, o, 0);
      else buf_put_b128<kStream>(w, rd, o, 0);
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
