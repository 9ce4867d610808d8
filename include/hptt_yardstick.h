/*
 * hptt_yardstick.h -- measurement kernels that put the transposition's
 * bandwidth in context, after Section 4 and Table 2 of the HPTT paper, which
 * compare against the SAXPY (y <- alpha*x + y) and STREAM-triad bandwidth of
 * each machine.  Bandwidth is counted as in Eq. (2): bytes that must cross
 * memory divided by time.
 *
 * All calls queue one kernel on `stream` and return without waiting; pointers
 * are device pointers owned by the caller.  They return HPTT_ERROR_INVALID_ARGUMENT
 * for null or misaligned pointers or sizes, HPTT_ERROR_HIP if the launch fails.
 */
#ifndef HPTT_YARDSTICK_H
#define HPTT_YARDSTICK_H

#include <stddef.h>
#include <stdint.h>

#include "hptt.h"

#ifdef __cplusplus
extern "C" {
#endif

/* dst <- src over `bytes` bytes (reads S, writes S: the lambda = 2 yardstick).
 * src and dst 16-byte aligned, bytes a multiple of 16, ranges disjoint. */
hptt_status_t hptt_yardstick_copy(const void *src, void *dst, size_t bytes, hipStream_t stream);

/* y <- alpha*x + beta*y over n elements of dtype (reads 2S, writes S: the
 * lambda = 3 SAXPY-like yardstick of Table 2).  x and y 16-byte aligned,
 * n*elem a multiple of 16. */
hptt_status_t hptt_yardstick_axpby(hptt_dtype_t dtype, double alpha, const void *x, double beta,
                                   void *y, size_t n, hipStream_t stream);

/* Write the 32-bit pattern `value` over `bytes` bytes of buf (16-byte aligned,
 * bytes a multiple of 16).  A fill of more than the last-level cache evicts
 * the tensors between timed runs ("caches are cleared in between runs",
 * Section 4). */
hptt_status_t hptt_yardstick_fill(void *buf, size_t bytes, uint32_t value, hipStream_t stream);

/* Read `bytes` bytes of buf (16-byte aligned, a multiple of 16) and write
 * one 32-bit checksum per workgroup into sink (at least 4096 bytes).  Reading
 * more than the last-level cache leaves it holding only clean lines of buf,
 * so the next kernel starts cold and owes no write-back of earlier data. */
hptt_status_t hptt_yardstick_read(const void *buf, size_t bytes, void *sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HPTT_YARDSTICK_H */
