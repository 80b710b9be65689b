/*
 * nm_micro.h -- roof micro-benchmarks for MI355X (gfx950), in libnm_micro.so,
 * separate from the product library.  They measure what the chip reaches
 * for the two roofs of the N:M SpMM path: HBM read bandwidth (the bound of
 * the short, memory-bound products) and fp32 matrix-core throughput (the
 * bound of the large ones), reported beside the published peaks, as the
 * paper reports its own measured fp32 peak (Sec. IV-E).  Timing is the
 * caller's (events on `stream`).  Return 0 on success, 1 for bad arguments,
 * 2 for a launch error.
 */
#ifndef NM_MICRO_H
#define NM_MICRO_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__)
#define NM_MICRO_API __attribute__((visibility("default")))
#else
#define NM_MICRO_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` (a multiple of 16) of DEVICE memory at `buf` (16-byte aligned)
 * once, with `blocks` workgroups of 256 threads in a grid-stride loop of
 * 16-byte loads.  sink: DEVICE memory of blocks * 256 uint32 that the kernel
 * may write (it writes only if an XOR of the data hits a fixed 32-bit
 * value). */
NM_MICRO_API int nm_micro_hbm_read(const void *buf, int64_t bytes, uint32_t *sink, int blocks,
                                   hipStream_t stream);

/* `blocks` workgroups of four waves, each wave issuing iters x 8 independent
 * v_mfma_f32_32x32x2_f32 (fp32 in, fp32 accumulate).  sink: DEVICE memory of
 * blocks * 256 floats, written. */
NM_MICRO_API int nm_micro_mfma_f32(float *sink, int iters, int blocks, hipStream_t stream);

/* Floating-point operations of one nm_micro_mfma_f32 launch. */
NM_MICRO_API double nm_micro_mfma_f32_flops(int iters, int blocks);

#ifdef __cplusplus
}
#endif
#endif /* NM_MICRO_H */
