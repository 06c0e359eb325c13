/*
 * saf_measure.h -- measurement aids of libsaf.so.  They compute nothing of
 * the layer; they give the benchmark reference readings that the layer's own
 * kernels cannot:
 *
 * - the shader clock while the layer runs (the bf16 MFMA peak scales with it:
 *   the published 2.5 PFLOP/s is quoted at 2.4 GHz), from the GPU's two
 *   hardware counters rather than a driver's DPM table;
 * - a known number of bytes read through the same load path the layer
 *   kernels use (buffer loads straight into LDS), so that a profiler's HBM
 *   byte counters can be scaled by what they read for a known size;
 * - the layer kernels' LDS operand reads one pattern at a time (which of
 *   them meet bank conflicts), and the MFMA rate of the two tile shapes.
 *
 * Conventions as in saf.h: device pointers owned by the caller, nothing
 * allocated, nothing synchronised, arguments checked before any launch.
 */
#ifndef SAF_MEASURE_H
#define SAF_MEASURE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "saf.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Shader-clock probe.  One wavefront reads the shader cycle counter
 * (s_memtime) and the constant 100 MHz reference counter (s_memrealtime),
 * then sleeps in short s_sleep steps until at least `duration_us`
 * microseconds of the reference clock have passed (the loop is also capped
 * at 2^26 iterations, so it always ends), and reads both counters again.
 *   out         : DEVICE, 2 x uint64, written: out[0] = shader cycles
 *                 elapsed, out[1] = reference ticks elapsed.  The mean shader
 *                 clock over the interval is out[0] / out[1] * 100 MHz.
 *   duration_us : 1 .. 1000000.
 * Launched on `stream`; to sample the clock while other work runs, enqueue
 * it on a second stream just before that work.  Errors: SAF_ERR_NULL,
 * SAF_ERR_SHAPE (duration out of range), SAF_ERR_ALIGNMENT (out not 8-byte
 * aligned), SAF_ERR_LAUNCH.
 */
saf_status_t saf_clock_probe(uint64_t* out, int duration_us, hipStream_t stream);

/*
 * Known-size read through the layer kernels' load path.  Workgroups of 256
 * threads copy consecutive 4 KB units of `src` into LDS with 16-byte buffer
 * loads straight to LDS (the instruction the layer kernels use for their
 * tiles), each unit read exactly once, and write one float per workgroup to
 * `sink` (so the kernel has a visible result).
 *   src   : DEVICE, `bytes` readable, 16-byte aligned; bytes a multiple of
 *           4096, 4096 .. 2^40.
 *   sink  : DEVICE float32 [ceil(bytes / 2^20)] (one per workgroup, which
 *           reads 256 units), written.
 * Errors: SAF_ERR_NULL, SAF_ERR_SHAPE, SAF_ERR_ALIGNMENT, SAF_ERR_LAUNCH.
 */
saf_status_t saf_lds_read_probe(const void* src, size_t bytes, float* sink, hipStream_t stream);

/*
 * LDS read patterns of the layer kernels, one per launch, for bank-conflict
 * counters (SQ_LDS_BANK_CONFLICT / SQ_INSTS_LDS) and timing.  256 workgroups
 * of 256 threads; each wavefront runs `iters` iterations of one pattern on a
 * 64 x 64 bf16 tile in the kernels' column-slab layout, addressed by the
 * kernels' own helpers:
 *   0  row operand of a 32 x 32 product (lane c reads row c, its 16-byte
 *      half chosen by the lane half; 4 reads per iteration)
 *   1  transposed operand of a 32 x 32 product, accumulator order (4 x 2)
 *   2  row operand of a 16 x 16 product (lanes i and i + 16 read the two
 *      halves of one row; 4)
 *   3  transposed operand of a 16 x 16 product (4 x 2)
 *   4  16-byte reads of per-row floats in the 32 x 32 accumulator order (4)
 *   5  16-byte reads of per-row floats in the 16 x 16 accumulator order (2)
 *   6  transposed operand of a 32 x 32 product, natural order (4 x 2)
 *   pattern : 0 .. 6;   iters : 1 .. 2^20;
 *   sink    : DEVICE uint32 [65536], 4-byte aligned; written only under a
 *             condition no pattern meets (it keeps the reads live).
 * Errors: SAF_ERR_NULL, SAF_ERR_SHAPE, SAF_ERR_ALIGNMENT, SAF_ERR_LAUNCH.
 */
saf_status_t saf_lds_pattern_probe(int pattern, int iters, uint32_t* sink, hipStream_t stream);

/*
 * MFMA rate of the two bf16 tile shapes the kernels use.  256 workgroups, one
 * per CU, each of 4 * waves_per_simd wavefronts; every wavefront issues
 * `iters` rounds of 131072 multiply-adds on independent accumulators:
 * 8 v_mfma_f32_32x32x16_bf16 (shape 0) or 16 v_mfma_f32_16x16x32_bf16
 * (shape 1).  FLOP per launch = 2 * 131072 * iters * 1024 * waves_per_simd.
 *   clk  : DEVICE 2 x uint64, 8-byte aligned: shader cycles and 100 MHz
 *          reference ticks of workgroup 0's run (its mean shader clock);
 *   sink : DEVICE float [256 * 64], written only under a condition the
 *          accumulators never meet.
 *   shape: 0 or 1;  waves_per_simd: 1 or 2;  iters: 1 .. 2^20.
 * Errors: SAF_ERR_NULL, SAF_ERR_SHAPE, SAF_ERR_ALIGNMENT, SAF_ERR_LAUNCH.
 */
saf_status_t saf_mfma_rate_probe(int shape, int waves_per_simd, int iters, uint64_t* clk, float* sink,
                                 hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SAF_MEASURE_H */
