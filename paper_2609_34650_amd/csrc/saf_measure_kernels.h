// Measurement aids (include/saf_measure.h): a shader-clock probe and a
// known-size read through the tile load path of the layer kernels.  Neither
// takes part in the layer's arithmetic.
#pragma once

#include "saf_common.h"

namespace saf {

// One wavefront: both hardware counters at the start, s_sleep steps until
// `ticks` reference ticks have passed (at most 2^26 steps), both counters
// again.  Lane 0 stores the two differences with an ordinary vector store.
__global__ __launch_bounds__(64) void clock_probe_kernel(uint64_t* out, uint64_t ticks) {
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    for (int it = 0; it < (1 << 26); ++it) {
        __builtin_amdgcn_s_sleep(1);
        if (__builtin_amdgcn_s_memrealtime() - r0 >= ticks) break;
    }
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    // Per-lane copies, so the store below is a vector store of lane 0.
    const uint64_t dt = (t1 - t0) + (uint64_t)(threadIdx.x & 0);
    const uint64_t dr = (r1 - r0) + (uint64_t)(threadIdx.x & 0);
    if (threadIdx.x == 0) {
        out[0] = dt;
        out[1] = dr;
    }
}

constexpr int PROBE_THREADS = 256;
constexpr int PROBE_UNIT = 4096;  // bytes: one 16-byte load per thread
constexpr int PROBE_UNITS_PER_WG = 256;

// Workgroup g reads units [256 g, min(256 g + 256, units)) of src into four
// rotating 4 KB LDS slots with 16-byte buffer loads straight to LDS (the
// layer kernels' tile load), then writes one LDS float to sink[g].
__global__ __launch_bounds__(PROBE_THREADS) void lds_read_probe_kernel(const char* src, unsigned long long units,
                                                                       float* sink) {
    __shared__ __attribute__((aligned(16))) float buf[4 * PROBE_UNIT / 4];
    const unsigned long long u0 = (unsigned long long)blockIdx.x * PROBE_UNITS_PER_WG;
    const unsigned long long left = units - u0;
    const int n = left < (unsigned long long)PROBE_UNITS_PER_WG ? (int)left : PROBE_UNITS_PER_WG;
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(src + u0 * PROBE_UNIT), (short)0, n * PROBE_UNIT,
                                          0x00020000);
    const int w = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    for (int k = 0; k < n; ++k) {
        lds_void* dst = (lds_void*)(reinterpret_cast<char*>(buf) + (k & 3) * PROBE_UNIT + w * 1024);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, dst, 16, k * PROBE_UNIT + w * 1024 + lane * 16, 0, 0, 0);
    }
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = buf[0];
}

}  // namespace saf
