/*
 * tsr_measure.h -- measurement aids exported by libtsr.so.
 *
 * NOT part of the composed-prefill path and not taken from the paper.  These
 * two kernels exist only so that a benchmark can report, next to the
 * published peaks, the rates the running GPU sustains (the matrix cores hold
 * a lower clock under load than the one the published figures assume).  A
 * serving caller never needs them.
 *
 * tsr_peak_mfma: n_workgroups workgroups of 256 threads each issue
 *   iters x 8 back-to-back v_mfma_f32_32x32x16_bf16 per wave on register
 *   operands (eight independent accumulators, no memory traffic in the
 *   loop); tsr_peak_mfma_flops gives the launch's FLOP count (0 for
 *   non-positive arguments).  dev_out: device buffer of n_workgroups * 256
 *   floats (owned by the caller) that receives per-thread sums, so that the
 *   products are not optimised away.  INVALID_ARG for non-positive sizes or
 *   a NULL buffer; DEVICE if the launch fails.
 * tsr_peak_copy: dst[0, bytes) <- src[0, bytes) with 16-byte loads and
 *   stores by a grid-stride kernel.  Both pointers device memory, 16-byte
 *   aligned, not overlapping; bytes a positive multiple of 16, else
 *   INVALID_ARG.
 * Errors follow tsr.h: a status, nothing enqueued, tsr_last_error() says why.
 */
#ifndef TSR_MEASURE_H
#define TSR_MEASURE_H

#include <stddef.h>
#include <stdint.h>

#include "tsr.h"

#ifdef __cplusplus
extern "C" {
#endif

int64_t tsr_peak_mfma_flops(int32_t n_workgroups, int32_t iters);
tsr_status tsr_peak_mfma(int32_t n_workgroups, int32_t iters, float* dev_out, void* stream);
tsr_status tsr_peak_copy(void* dst, const void* src, size_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TSR_MEASURE_H */
