/*
 * zf_measure.h -- measurement helpers of libzf (not part of the method).
 *
 * The hot path of ZenFlow's GPU side is bound by HBM bandwidth (every pass
 * streams its operands once).  To state how close each pass comes to what
 * the chip can stream with the same access pattern, the library exports
 * reference streams built from the update pass's own building blocks (one
 * contiguous 4 KiB chunk per 256-thread block, 16-byte raw buffer accesses,
 * the XCD-aware block order, the update's cache policies) with no
 * arithmetic.  Conventions (device pointers, caller-owned memory, stream
 * ordering, status codes) are those of zf.h.
 */
#ifndef ZF_MEASURE_H
#define ZF_MEASURE_H

#include <stddef.h>
#include <stdint.h>

#include "zf.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum zf_stream_probe_kind {
  ZF_PROBE_READ = 0, /* reads `bytes` of src; dst is a 4-byte word that is
                        written only if the loaded data fold to `key` */
  ZF_PROBE_COPY = 1, /* copies `bytes` from src to dst (disjoint) */
  ZF_PROBE_RMW = 2   /* dst ^= key per 32-bit word, in place (`bytes` read and
                        written back); src unused (may be NULL) */
} zf_stream_probe_kind;

/* Enqueues one streaming pass of `kind` over `bytes` on `stream`.
 * bytes: > 0, a multiple of 16, at most (2^32 - 1) / 256 blocks of 4 KiB; src and
 * dst 16-byte aligned (dst 4-byte aligned for ZF_PROBE_READ).  ZF_EINVAL
 * (nothing enqueued) otherwise, or when src and dst overlap for
 * ZF_PROBE_COPY.  Bytes moved: `bytes` for READ, 2 * `bytes` for COPY and
 * RMW. */
zf_status zf_stream_probe(int32_t kind, const void* src, void* dst, size_t bytes, uint32_t key,
                          zf_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* ZF_MEASURE_H */
