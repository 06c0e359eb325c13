// Measurement aids (include/saf_measure.h): a shader-clock probe, a
// known-size read through the tile load path of the layer kernels, the layer
// kernels' LDS operand reads issued one pattern at a time, and an MFMA rate
// probe.  None takes part in the layer's arithmetic.
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

// LDS operand reads of the layer kernels, one pattern per kernel, through the
// library's own tile addressing (ld_row, ld_tile_t, ld_tile_t16 on one
// 64 x 64 bf16 column-slab tile, 16-byte reads of a float row array).  The
// row offset alternates between 0 and 32 through an opaque register, so every
// read stays inside the loop.  The reads are folded into one value that is
// stored (sink[blockIdx.x * 256 + threadIdx.x]) only if it equals a constant
// no pattern produces.  Every address lies inside the tile or the row array.
constexpr int LDS_PATTERN_COUNT = 7;
constexpr int LDS_PATTERN_THREADS = 256;
constexpr int LDS_PATTERN_BLOCKS = 256;

template <int P>
__global__ __launch_bounds__(LDS_PATTERN_THREADS) void lds_pattern_kernel(uint32_t* sink, int iters) {
    __shared__ __attribute__((aligned(16))) bf16 tile[tile_elems<bf16>()];
    __shared__ __attribute__((aligned(16))) float rows[2 * TILE_ROWS];
    const int t = threadIdx.x, l = t & 63, c = l & 31, hf = l >> 5, n = l & 15, g = l >> 4;
    for (int x = t; x < tile_elems<bf16>(); x += LDS_PATTERN_THREADS) tile[x] = (bf16)(float)(x & 255);
    if (t < 2 * TILE_ROWS) rows[t] = (float)t;
    __syncthreads();
    uint32_t acc = 0;
    auto fold = [&](const bf16x8& v) { acc ^= __builtin_bit_cast(uint32_t, bf16x2{v[0], v[7]}); };
    for (int it = 0; it < iters; ++it) {
        int h32 = 32 * (it & 1);
        asm volatile("" : "+v"(h32));
        h32 &= ~31;  // known to be a multiple of 32 again, so 16-byte reads stay 16-byte reads
        if constexpr (P == 0) {  // row operand of a 32 x 32 product: row c, columns 16 dc + 8 hf
#pragma unroll
            for (int dc = 0; dc < 4; ++dc) fold(ld_row<bf16>(tile, h32 + c, 16 * dc + 8 * hf));
        } else if constexpr (P == 1) {  // transposed operand of a 32 x 32 product, accumulator order
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int db = 0; db < 2; ++db) fold(ld_tile_t<true>(tile, h32 + 16 * kc, 32 * db));
        } else if constexpr (P == 2) {  // row operand of a 16 x 16 product: row 16 qt + n, columns 32 dc + 8 g
#pragma unroll
            for (int qt = 0; qt < 2; ++qt)
#pragma unroll
                for (int dc = 0; dc < 2; ++dc) fold(ld_row<bf16>(tile, h32 + 16 * qt + n, 32 * dc + 8 * g));
        } else if constexpr (P == 3) {  // transposed operand of a 16 x 16 product
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) fold(ld_tile_t16(tile, h32, 16 * dt));
        } else if constexpr (P == 4) {  // per-row floats, 32 x 32 accumulator rows: 16 bytes at 8 g + 4 hf
#pragma unroll
            for (int gg = 0; gg < 4; ++gg) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(rows + h32 + 8 * gg + 4 * hf);
                acc ^= __float_as_uint(v[0] + v[3]);
            }
        } else if constexpr (P == 5) {  // per-row floats, 16 x 16 accumulator rows: 16 bytes at 16 qt + 4 g
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(rows + h32 + 16 * qt + 4 * g);
                acc ^= __float_as_uint(v[0] + v[3]);
            }
        } else {  // transposed operand of a 32 x 32 product, natural order (fixed heads)
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int db = 0; db < 2; ++db) fold(ld_tile_t<false>(tile, h32 + 16 * kc, 32 * db));
        }
    }
    if (acc == 0x9e3779b9u) sink[blockIdx.x * LDS_PATTERN_THREADS + t] = acc;
}

// MFMA rate: one workgroup per CU (the LDS pad leaves room for no second
// one), 4 W wavefronts, each issuing `iters` rounds of 131072 bf16 MACs on
// independent accumulators: 8 v_mfma_f32_32x32x16_bf16 (SHAPE 0) or 16
// v_mfma_f32_16x16x32_bf16 (SHAPE 1).  Block 0 records the shader cycles and
// reference ticks of its run in clk[0..1] (a vector store of lane 0); the
// accumulators reach sink only under a condition they never meet.
constexpr int MFMA_PROBE_BLOCKS = 256;

template <int SHAPE>
__global__ __launch_bounds__(512) void mfma_rate_kernel(uint64_t* clk, float* sink, int iters) {
    __shared__ float pad[24 * 1024];  // 96 KB
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (bf16)(threadIdx.x * 0.001f + i);
        b[i] = (bf16)(i * 0.5f);
    }
    f32x16 c[4];
    f32x4 d[8];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int i = 0; i < 16; ++i) c[k][i] = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) d[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int it = 0; it < iters; ++it) {
        if constexpr (SHAPE == 0) {
#pragma unroll
            for (int k = 0; k < 8; ++k) mma(c[k & 3], a, b);
        } else {
#pragma unroll
            for (int k = 0; k < 16; ++k) mma16(d[k & 7], a, b);
        }
    }
    float r = pad[threadIdx.x & 63];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int i = 0; i < 16; ++i) r += c[k][i];
#pragma unroll
    for (int k = 0; k < 8; ++k) r += d[k][0] + d[k][1] + d[k][2] + d[k][3];
    if (r == 1.2345f) sink[blockIdx.x * 64 + (threadIdx.x & 63)] = r;
    __syncthreads();
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    const uint64_t dt = (t1 - t0) + (uint64_t)(threadIdx.x & 0);
    const uint64_t dr = (r1 - r0) + (uint64_t)(threadIdx.x & 0);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        clk[0] = dt;
        clk[1] = dr;
    }
}

}  // namespace saf
