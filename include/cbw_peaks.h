/*
 * cbw_peaks — measured machine ceilings for the roofline of the convolution
 * kernels (libcbwpeaks.so, a separate library used by the benchmark).
 *
 * These are measurement utilities, not operations of the paper: the paper
 * evaluates a simulated accelerator (Sec. V) and has no counterpart of a
 * GPU's matrix-core or HBM peak.  The convolution kernels are reported
 * against both the published MI355X peaks and these measured ones.
 *
 * Conventions: pointers are device memory owned by the caller; `stream` is a
 * hipStream_t passed as void*; each call queues one kernel and returns 0, or
 * -1 for an invalid argument (nothing launched), or -4 for a HIP launch error.
 * The caller times the launch (for example with events on `stream`).
 */
#ifndef CBW_PEAKS_H
#define CBW_PEAKS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Matrix-instruction shapes of cbw_peak_mfma (bf16 inputs, fp32 accumulation). */
#define CBW_PEAK_MFMA_16X16X32 0
#define CBW_PEAK_MFMA_32X32X16 1

/* Bytes of the operand seed cbw_peak_mfma reads (any values; 16-byte aligned). */
size_t cbw_peak_seed_bytes(void);
/* 32-bit words a sink must hold for cbw_peak_mfma with `blocks` workgroups
 * and for the stream kernels. */
size_t cbw_peak_sink_words(int blocks);
/* Floating-point operations one cbw_peak_mfma launch performs. */
double cbw_peak_mfma_flops(int shape, int blocks, int iters);

/* Matrix-core loop: `blocks` workgroups of four waves, each wave issuing
 * `iters` rounds of independent matrix instructions of `shape` on register
 * operands (no memory traffic in the loop).  With several workgroups per CU
 * the rate is the sustained matrix-core peak.  `sink` (cbw_peak_sink_words
 * words) is never written in practice. */
int cbw_peak_mfma(int shape, int blocks, int iters, const void* seed, float* sink, void* stream);

/* HBM read stream: loads every 16-byte vector of src[0, bytes) once (bytes a
 * multiple of 16, src 16-byte aligned); `sink` as above. */
int cbw_peak_hbm_read(const void* src, size_t bytes, uint32_t* sink, void* stream);

/* HBM copy stream: dst[0, bytes) = src[0, bytes), 16-byte vectors; moves
 * 2 * bytes. */
int cbw_peak_hbm_copy(const void* src, void* dst, size_t bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* CBW_PEAKS_H */
