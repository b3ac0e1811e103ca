/*
 * dla_peak.h -- measurement kernels of libdla: the dense bfloat16 matrix-core
 * rate and the HBM read bandwidth of the device, measured rather than taken
 * from the data sheet, so that the roofline fractions the benchmark reports
 * for the DLA kernels can be stated against both.  They compute nothing of
 * the method.
 *
 * Both enqueue one kernel on `stream` (a hipStream_t as void*, NULL = the null
 * stream) and return after enqueueing; the caller times them with events.
 * `sink` is device memory of blocks * 256 floats that receives one value per
 * thread (so that the work is not optimised away); its contents mean nothing.
 * Errors: DLA_ERR_INVALID_ARG for a null pointer or a non-positive count,
 * DLA_ERR_HIP for a failed launch.
 */
#ifndef DLA_PEAK_H
#define DLA_PEAK_H

#include <stddef.h>
#include <stdint.h>

#include "dla.h"

#ifdef __cplusplus
extern "C" {
#endif

/* `blocks` workgroups of 4 waves; each wave runs 4 independent chains of
 * `iters` v_mfma_f32_32x32x16_bf16 on register operands.  Work: blocks * 16 *
 * iters * 32768 floating-point operations. */
dla_status dla_peak_mfma_bf16(int32_t blocks, int32_t iters, float* sink, void* stream);

/* `blocks` workgroups of 256 threads read `bytes` (a multiple of 4096) of the
 * device buffer `buf` once, with 16-byte non-temporal loads. */
dla_status dla_peak_hbm_read(const void* buf, size_t bytes, int32_t blocks, float* sink,
                             void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DLA_PEAK_H */
