/*
 * saf_measure.h -- measurement aids of libsaf.so.  They compute nothing of
 * the layer; they give the benchmark two reference readings that the layer's
 * own kernels cannot:
 *
 * - the shader clock while the layer runs (the bf16 MFMA peak scales with it:
 *   the published 2.5 PFLOP/s is quoted at 2.4 GHz), from the GPU's two
 *   hardware counters rather than a driver's DPM table;
 * - a known number of bytes read through the same load path the layer
 *   kernels use (buffer loads straight into LDS), so that a profiler's HBM
 *   byte counters can be scaled by what they read for a known size.
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

#ifdef __cplusplus
}
#endif

#endif /* SAF_MEASURE_H */
