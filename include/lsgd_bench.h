/*
 * lsgd_bench.h - measurement utility exported by liblsgd.so. Not part of the
 * Layered SGD method: a plain streaming copy that gives the HBM bandwidth a
 * kernel of this library can reach for a simple read+write stream, and a
 * kernel of known traffic for calibrating hardware byte counters.
 */
#ifndef LSGD_BENCH_H
#define LSGD_BENCH_H

#include "lsgd.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * dst[0..bytes) = src[0..bytes): device-to-device copy with 128-bit
 * nontemporal loads and stores, one 16-byte unit per lane, workgroups in the
 * XCD-chunked order of the launch shape. Moves exactly `bytes` read and
 * `bytes` written.
 *   dst, src  device pointers, 16-byte aligned (LSGD_ERR_ALIGN), non-NULL when
 *             bytes > 0 (LSGD_ERR_NULL), non-overlapping (LSGD_ERR_ALIAS).
 *   bytes     a multiple of 16, >= 0 (LSGD_ERR_SIZE); 0 is a no-op.
 * Stream-ordered and asynchronous like every other call.
 */
LSGD_API lsgd_status lsgd_stream_copy(void* dst, const void* src, int64_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LSGD_BENCH_H */
