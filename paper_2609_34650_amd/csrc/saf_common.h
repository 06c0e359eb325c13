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

}  // namespace saf
