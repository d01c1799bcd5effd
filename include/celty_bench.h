/*
 * celty_bench.h -- a measurement reference exported by libcelty, not part of
 * the product: a plain streaming read of device memory.
 *
 * The product's kernels read compressed column segments (Section 3.1); this
 * call reads the same number of bytes as one contiguous stream, so that the
 * benchmark can report what the memory system delivers to a single launch of
 * that size (launch, ramp and drain included) beside the product's time.  It
 * computes nothing of the method.
 */
#ifndef CELTY_BENCH_H
#define CELTY_BENCH_H

#include <stddef.h>
#include <stdint.h>

#include "celty.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Reads `bytes` of device memory at p with 16-byte non-temporal loads in one
 * kernel launch of `blocks` workgroups of `threads` lanes, each lane keeping
 * four loads in flight, and writes one word per workgroup (an XOR of what it
 * read) to sink, so that no load is dead.
 *   p        device, 16-byte aligned; bytes a multiple of 16 (0 allowed).
 *   sink     device uint32[blocks], 4-byte aligned.
 *   blocks   1 .. 65535;  threads  64 .. 1024, a multiple of 64.
 *   stream   HIP stream (NULL = default); asynchronous.
 * Errors: EINVAL (null or misaligned pointers, sizes outside the ranges),
 * EHIP.
 */
celty_status celty_bench_stream_read(const void* p, size_t bytes, uint32_t* sink, int32_t blocks, int32_t threads,
                                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CELTY_BENCH_H */
