/*
 * mure_peaks.h -- the two ceilings the measurements are reported against,
 * measured on the GPU the library runs on (libmure_peaks.so, separate from
 * libmure.so and from the mutation-testing path).
 *
 * The vendor's figures for one MI355X (HBM3E 8 TB/s, dense bf16 MFMA
 * 2.5 PFLOP/s, fp32 MFMA 157.3 TFLOP/s) are upper limits that no program
 * reaches.  A kernel's fraction of its roofline is therefore also given
 * against what a plain copy and a register-only MFMA loop sustain on the same
 * card: the copy is STREAM's "copy" kernel (every byte read once and written
 * once), the loop keeps independent accumulator chains in registers and
 * touches memory only to store one value per lane at its end.
 *
 * Both calls enqueue on `stream` (a hipStream_t, NULL for the null stream),
 * time their launches with HIP events on that stream, synchronise it and
 * return 0, or a negative hipError_t value (-(int)err) if a HIP call failed,
 * or -1 for invalid arguments (nothing is launched then).
 */
#ifndef MURE_PEAKS_H
#define MURE_PEAKS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* STREAM copy: dst[i] = src[i] for the `bytes` bytes of two device buffers
 * (16-byte aligned, `bytes` a positive multiple of 16, not overlapping),
 * in eight variants of the copy kernel (4 or 8 vectors in flight per thread,
 * plain or non-temporal stores, 8 or 32 blocks per CU), each repeated `reps`
 * times (1..1000) after one untimed launch.  *gbs receives the best launch's
 * rate, counting 2 * bytes (read and write) per launch, in GB/s (1e9 bytes
 * per second).  The caller owns both buffers. */
int mure_peak_copy(const void* src, void* dst, int64_t bytes, int reps, void* stream, double* gbs);

/* MFMA loop: `blocks` workgroups (1..65536) of 4 wavefronts, each wavefront
 * running `iters` rounds (1..10^7) of independent accumulator chains: 4 of
 * v_mfma_f32_32x32x16_bf16 (dtype 1) or 8 of v_mfma_f32_16x16x4_f32 (dtype 0),
 * repeated `reps` times (1..100) after one untimed launch.  Every lane then
 * stores the sum of its accumulators into `sink` (device, blocks * 256
 * floats, owned by the caller), so no work can be removed.  *tflops
 * receives the best launch's rate in TFLOP/s (2 flops per multiply-add). */
int mure_peak_mfma(int dtype, int blocks, int iters, int reps, float* sink, void* stream, double* tflops);

#ifdef __cplusplus
}
#endif

#endif /* MURE_PEAKS_H */
