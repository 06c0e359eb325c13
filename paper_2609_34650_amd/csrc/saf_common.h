// Shared device-side building blocks for the gfx950 hybrid-attention kernels.
//
// Every matrix product runs on the 32x32 MFMA tile.  With lane l of a 64-wide
// wavefront, write c = l % 32 and hf = l / 32 (the lane half).  One "k-chunk"
// of a product contracts 16 k-slots:
//   A operand (32 rows x 16 k): lane l supplies row c, k-slots 8*hf + t, t=0..7
//   B operand (16 k x 32 cols): lane l supplies col c, k-slots 8*hf + t
//   C/D accumulator (32 x 32, 16 floats per lane): register v of lane l holds
//     row 8*(v/4) + 4*hf + (v%4), col c.
// Which physical k a slot stands for is the caller's choice, as long as A and
// B agree: a product is invariant under a common permutation of its
// contraction index.  The kernels use that freedom to feed a softmax
// accumulator straight back into the next product as an operand.
//
// bf16 chunks are one v_mfma_f32_32x32x16_bf16; float32 chunks are eight
// v_mfma_f32_32x32x2_f32, instruction t taking slot 8*hf + t from each lane,
// so the register contents per lane are the same eight values in both cases.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace saf {

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(8))) float f32x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int HEAD_DIM = 64;
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
// Running-max start value: finite, so exp2(m_old - m_new) is 0 (not NaN)
// on the first visible tile.
constexpr float NEG_BIG = -1.0e30f;
// Fixed heads use the factorised exp(a - A) * exp(r - R) form only while every
// row's normaliser stays within this many natural-log units of exp(A + R);
// beyond it a workgroup falls back to exact per-element exponentials.
constexpr float FAST_GUARD = 40.0f;
// Shifted copies of a Toeplitz band in LDS: copy s starts s entries later, so
// eight consecutive entries from any start are one aligned 16-byte read.
constexpr int BAND_COPIES = 8;

template <typename T> struct Vec;
template <> struct Vec<bf16> {
    typedef bf16x8 x8;
    typedef bf16x4 x4;
    typedef bf16x2 x2;
};
template <> struct Vec<float> {
    typedef f32x8 x8;
    typedef f32x4 x4;
    typedef f32x2 x2;
};

// One k-chunk: acc += A * B.
__device__ __forceinline__ void mma(f32x16& acc, const bf16x8& a, const bf16x8& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x16& acc, const f32x8& a, const f32x8& b) {
#pragma unroll
    for (int t = 0; t < 8; ++t) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[t], b[t], acc, 0, 0, 0);
}

template <typename T>
__device__ __forceinline__ typename Vec<T>::x8 zero8() {
    typename Vec<T>::x8 z;
#pragma unroll
    for (int t = 0; t < 8; ++t) z[t] = (T)0.0f;
    return z;
}

// Eight consecutive accumulator registers (starting at v0) as an operand.
template <typename T>
__device__ __forceinline__ typename Vec<T>::x8 to_operand(const f32x16& acc, int v0) {
    typename Vec<T>::x8 o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = (T)acc[v0 + t];
    return o;
}

template <typename T>
__device__ __forceinline__ typename Vec<T>::x8 ld8(const T* p) {
    return *reinterpret_cast<const typename Vec<T>::x8*>(p);
}

template <typename T>
__device__ __forceinline__ void st8(T* p, const typename Vec<T>::x8& v) {
    *reinterpret_cast<typename Vec<T>::x8*>(p) = v;
}

template <typename T>
__device__ __forceinline__ void st4(T* p, float x0, float x1, float x2, float x3) {
    typename Vec<T>::x4 v;
    v[0] = (T)x0;
    v[1] = (T)x1;
    v[2] = (T)x2;
    v[3] = (T)x3;
    *reinterpret_cast<typename Vec<T>::x4*>(p) = v;
}

template <typename T>
__device__ __forceinline__ void st2(T* p, T x0, T x1) {
    typename Vec<T>::x2 v;
    v[0] = x0;
    v[1] = x1;
    *reinterpret_cast<typename Vec<T>::x2*>(p) = v;
}

// Position of row/key k of a 64-wide tile inside a transposed LDS tile.
// Bits 2 and 3 are swapped, so that in each 16-wide group the eight keys
// {4*hf + u, 8 + 4*hf + u : u = 0..3} -- the keys that lane half hf holds in
// an accumulator (rows 8*g + 4*hf + u) -- sit at eight consecutive positions
// 8*hf .. 8*hf + 7 and one 16-byte LDS read fetches them.
__device__ __forceinline__ int tpos(int k) {
    return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32); }

// IEEE maximum (NaN-propagating): lowers to v_maximum3_f32 chains with no
// NaN-quieting of the inputs, unlike fmaxf.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

__device__ __forceinline__ unsigned int pack_bf16(float lo, float hi) {
    const bf16x2 v = {(bf16)lo, (bf16)hi};
    return __builtin_bit_cast(unsigned int, v);
}

// Transposed store of two consecutive rows x0, x1 (eight consecutive columns
// each): dst[t * ld] = (x0[t], x1[t]) as an adjacent pair, t = 0..7.  The bf16
// version packs the halves of 32-bit words with v_perm_b32 (no per-element
// vector shuffles, which the compiler would route through scratch memory).
__device__ __forceinline__ void st_pair_t(bf16* dst, int ld, const bf16x8& x0, const bf16x8& x1) {
    const u32x4 a = __builtin_bit_cast(u32x4, x0);
    const u32x4 b = __builtin_bit_cast(u32x4, x1);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        *reinterpret_cast<unsigned int*>(dst + (2 * m) * ld) = __builtin_amdgcn_perm(b[m], a[m], 0x05040100u);
        *reinterpret_cast<unsigned int*>(dst + (2 * m + 1) * ld) = __builtin_amdgcn_perm(b[m], a[m], 0x07060302u);
    }
}
__device__ __forceinline__ void st_pair_t(float* dst, int ld, const f32x8& x0, const f32x8& x1) {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const f32x2 v = {x0[t], x1[t]};
        *reinterpret_cast<f32x2*>(dst + t * ld) = v;
    }
}

// As st_pair_t, with row x0 scaled by e0 and row x1 by e1 (rounded once).
__device__ __forceinline__ void st_pair_t_scaled(bf16* dst, int ld, const bf16x8& x0, const bf16x8& x1, float e0,
                                                 float e1) {
    const u32x4 a = __builtin_bit_cast(u32x4, x0);
    const u32x4 b = __builtin_bit_cast(u32x4, x1);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const float a_lo = __uint_as_float(a[m] << 16), a_hi = __uint_as_float(a[m] & 0xffff0000u);
        const float b_lo = __uint_as_float(b[m] << 16), b_hi = __uint_as_float(b[m] & 0xffff0000u);
        *reinterpret_cast<unsigned int*>(dst + (2 * m) * ld) = pack_bf16(a_lo * e0, b_lo * e1);
        *reinterpret_cast<unsigned int*>(dst + (2 * m + 1) * ld) = pack_bf16(a_hi * e0, b_hi * e1);
    }
}
__device__ __forceinline__ void st_pair_t_scaled(float* dst, int ld, const f32x8& x0, const f32x8& x1, float e0,
                                                 float e1) {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const f32x2 v = {x0[t] * e0, x1[t] * e1};
        *reinterpret_cast<f32x2*>(dst + t * ld) = v;
    }
}

// Sum of the eight operand values: for bf16 the rounded values that enter
// the product (four packed dot products against ones), for float32 plain adds.
__device__ __forceinline__ float sum8(const bf16x8& x, float acc) {
    const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
    for (int t = 0; t < 8; t += 2) {
        const bf16x2 pr = {x[t], x[t + 1]};
        acc = __builtin_amdgcn_fdot2_f32_bf16(pr, one, acc, false);
    }
    return acc;
}
__device__ __forceinline__ float sum8(const f32x8& x, float acc) {
#pragma unroll
    for (int t = 0; t < 8; ++t) acc += x[t];
    return acc;
}

// acc + sum_t x[t] * y[t] over eight operand values.
__device__ __forceinline__ float dot8(const bf16x8& x, const bf16x8& y, float acc) {
#pragma unroll
    for (int t = 0; t < 8; t += 2) {
        const bf16x2 px = {x[t], x[t + 1]};
        const bf16x2 py = {y[t], y[t + 1]};
        acc = __builtin_amdgcn_fdot2_f32_bf16(px, py, acc, false);
    }
    return acc;
}
__device__ __forceinline__ float dot8(const f32x8& x, const f32x8& y, float acc) {
#pragma unroll
    for (int t = 0; t < 8; ++t) acc = fmaf(x[t], y[t], acc);
    return acc;
}

// Maximum / minimum over the 256 threads of a workgroup (4 wavefronts);
// `red` is 4 floats of LDS.  Contains barriers: call from uniform code.
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}
__device__ __forceinline__ float block_max(float x, float* red) {
    x = wave_max(x);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
    __syncthreads();
    return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

}  // namespace saf
