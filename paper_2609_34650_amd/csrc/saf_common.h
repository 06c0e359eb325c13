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

#include <type_traits>

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

// 16 x 16 tiles (v_mfma_f32_16x16x32_bf16): an accumulator lane l holds
// column l % 16 and rows 4 (l / 16) .. 4 (l / 16) + 3; an operand lane holds
// row (A) or column (B) l % 16 and eight k-slots of its group l / 16.  The
// float32 form takes eight 16x16x4 steps, slot t of every group in step t.
__device__ __forceinline__ void mma16(f32x4& acc, const bf16x8& a, const bf16x8& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma16(f32x4& acc, const f32x8& a, const f32x8& b) {
#pragma unroll
    for (int t = 0; t < 8; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t], b[t], acc, 0, 0, 0);
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

// Two 16 x 16 accumulator tiles stacked along k as one operand: slots 0-3
// from lo, 4-7 from hi.
template <typename T>
__device__ __forceinline__ typename Vec<T>::x8 to_operand16(const f32x4& lo, const f32x4& hi) {
    typename Vec<T>::x8 o;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        o[t] = (T)lo[t];
        o[4 + t] = (T)hi[t];
    }
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

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// IEEE maximum (NaN-propagating): lowers to v_maximum3_f32 chains with no
// NaN-quieting of the inputs, unlike fmaxf.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Reductions over the lane pair (l, l ^ 32) with one v_permlane32_swap (a
// VALU exchange of the two wavefront halves, no LDS round trip).  Both lanes
// of a pair get the same, bitwise identical result.
__device__ __forceinline__ float pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

__device__ __forceinline__ unsigned int pack_bf16(float lo, float hi) {
    const bf16x2 v = {(bf16)lo, (bf16)hi};
    return __builtin_bit_cast(unsigned int, v);
}

// ---------------------------------------------------------------------------
// Column-slab LDS tiles.  A 64-row tile of a [rows, 64] matrix is split into
// slabs of 32 bytes of columns (16 bf16 or 8 float); each slab stores its 64
// rows 32 bytes apart, and slabs are SLAB_BYTES apart, 128 bytes more than
// 2 KB so that neighbouring slabs sit in opposite halves of the LDS banks.
// A row operand (eight consecutive columns of a row per lane) is one linear
// run, and each 16-lane group of a transposed read (four rows x 32 bytes) is
// one 128-byte run.  Measured bank conflicts (saf_lds_pattern_probe): none
// for the transposed reads and for the row operand of a 16 x 16 product
// (lanes i and i + 16 read the two halves of one row); 4 cycles per read for
// the row operand of a 32 x 32 product (lane c reads row c, so lanes i and
// i + 16, served together, read rows 16 apart at the same half, which share
// banks); a layout that swaps the halves of rows 16-31 and 48-63 removes
// those without making the kernels faster.  It is also the order in which a
// buffer load to LDS writes 64 lanes x 16 bytes.
// ---------------------------------------------------------------------------
constexpr int SLAB_BYTES = 32 * 64 + 128;
constexpr int TILE_ROWS = 64;

template <typename T> __host__ __device__ constexpr int slab_cols() { return 32 / (int)sizeof(T); }
// D: the row width (head dimension) of the matrix the tile comes from.
template <typename T, int D = HEAD_DIM> __host__ __device__ constexpr int tile_slabs() { return D / slab_cols<T>(); }
template <typename T, int D = HEAD_DIM> __host__ __device__ constexpr int tile_elems() {
    return tile_slabs<T, D>() * SLAB_BYTES / (int)sizeof(T);
}
// Element offset of (row, col) inside a tile.
template <typename T> __device__ __forceinline__ int toff(int row, int col) {
    return (col / slab_cols<T>()) * (SLAB_BYTES / (int)sizeof(T)) + row * slab_cols<T>() + (col % slab_cols<T>());
}

// The 16-byte units of a tile are split over the 4 wavefronts: unit k of lane
// `lane` in wavefront w holds row 32*(w & 1) + lane/2, slab (w >> 1) + 2*k,
// byte half lane & 1.  One wavefront's unit k covers 1 KB of LDS contiguously.
template <typename T> __device__ __forceinline__ int unit_row(int w, int lane) { return 32 * (w & 1) + (lane >> 1); }
template <typename T> __device__ __forceinline__ int unit_col(int w, int lane, int k) {
    return ((w >> 1) + 2 * k) * slab_cols<T>() + (lane & 1) * (16 / (int)sizeof(T));
}
template <typename T, int D = HEAD_DIM> __host__ __device__ constexpr int tile_units() {
    return tile_slabs<T, D>() / 2;
}

// Buffer resource over one [rows, D] slice of T; reads past `rows` return 0.
template <typename T, int D = HEAD_DIM>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t slice_rsrc(const T* base, int rows) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(base), (short)0, rows * D * (int)sizeof(T), 0x00020000);
}

typedef __attribute__((address_space(3))) void lds_void;

// Asynchronous copy of rows [row0, row0 + 64) of a slice into a tile: each
// wavefront issues tile_units() buffer loads that write LDS directly (no
// registers).  Rows past the end of the slice arrive as zeros.  The data is
// visible after the next __syncthreads().
template <typename T, int D = HEAD_DIM>
__device__ __forceinline__ void tile_load_lds(T* tile, __amdgpu_buffer_rsrc_t rsrc, int row0, int w, int lane) {
#pragma unroll
    for (int k = 0; k < tile_units<T, D>(); ++k) {
        const int s = (w >> 1) + 2 * k;
        T* dst = tile + s * (SLAB_BYTES / (int)sizeof(T)) + (w & 1) * (1024 / (int)sizeof(T));
        const int row = row0 + unit_row<T>(w, lane);
        const int voff = row * D * (int)sizeof(T) + s * 32 + (lane & 1) * 16;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)dst, 16, voff, 0, 0, 0);
    }
}

// The LDS of a workgroup: four tiles (eight in the key-block pass, which
// takes 128 queries per step), each its own __shared__ array, so that
// the compiler can tell a tile being filled by in-flight buffer loads from the
// one being read (and skips waiting for those loads before the reads); two
// small per-buffer float arrays; a few floats for reductions.  Each program
// gives the tiles its own roles.
template <typename T>
struct Tiles {
    T* t[8];
    float* aux[2];
    float* red;
};

// Double-buffered tile schedule shared by the programs.  Slots [0, P) hold
// the tiles that need masking (P even; a slot whose tile_of is -1 is
// padding), slots [P, total) the mask-free tiles.  Slot i works on buffer
// i % 2 while the copy for slot i+1 goes to the other buffer:
//   issue(buf, t)          starts copying tile t towards buffer buf (buffer
//                          loads straight to LDS, or loads into registers);
//   finish(buf)            completes a register-staged copy into LDS buffer
//                          buf, after this slot's compute (a no-op for
//                          direct loads);
//   compute(buf, t, MASK)  works on tile t in buffer buf.
// buf and MASK arrive as std::integral_constant, so every buffer access
// names a fixed LDS array and the mask-free loop holds exactly one body per
// buffer.  A __syncthreads() closes every slot; a buffer is refilled only
// after the barrier that follows its last read.
typedef std::integral_constant<int, 0> Buf0;
typedef std::integral_constant<int, 1> Buf1;

template <typename TileOf, typename Issue, typename Finish, typename Compute>
__device__ __forceinline__ void run_slots(int P, int total, TileOf tile_of, Issue issue, Finish finish,
                                          Compute compute) {
    auto pre = [&](auto buf, int i) {
        if (i < total) {
            const int t = tile_of(i);
            if (t >= 0) issue(buf, t);
        }
    };
    auto fin = [&](auto buf, int i) {
        if (i < total && tile_of(i) >= 0) finish(buf);
    };
    pre(Buf0{}, 0);
    fin(Buf0{}, 0);
    __syncthreads();
    for (int i = 0; i < P; i += 2) {
        pre(Buf1{}, i + 1);
        if (tile_of(i) >= 0) compute(Buf0{}, tile_of(i), std::true_type{});
        fin(Buf1{}, i + 1);
        __syncthreads();
        pre(Buf0{}, i + 2);
        if (tile_of(i + 1) >= 0) compute(Buf1{}, tile_of(i + 1), std::true_type{});
        fin(Buf0{}, i + 2);
        __syncthreads();
    }
    for (int i = P; i < total; i += 2) {
        pre(Buf1{}, i + 1);
        compute(Buf0{}, tile_of(i), std::false_type{});
        fin(Buf1{}, i + 1);
        __syncthreads();
        if (i + 1 >= total) break;
        pre(Buf0{}, i + 2);
        compute(Buf1{}, tile_of(i + 1), std::false_type{});
        fin(Buf0{}, i + 2);
        __syncthreads();
    }
}

// Row operand: eight consecutive columns col .. col+7 of tile row `row`.
template <typename T>
__device__ __forceinline__ typename Vec<T>::x8 ld_row(const T* tile, int row, int col) {
    return ld8<T>(tile + toff<T>(row, col));
}

// Transposed operand from a column-slab tile: the A operand whose row m is
// tile column col0 + m and whose k-slot t of lane half hf is tile row
//   row0 + 8*(t/4) + 4*hf + (t%4)   (ACC_ORDER: the order in which an MFMA
//                                     accumulator holds its rows), or
//   row0 + 8*hf + t                 (natural order).
// bf16: two ds_read_b64_tr_b16.  Within each 16-lane group that instruction
// hands lane 4a+b element b of the 8-byte chunks addressed by lanes a, a+4,
// a+8 and a+12, so lane i of a group addresses tile row (slot base + i/4) at
// column col0 + 16*(group parity) + 4*(i%4) and receives four k-slots of its
// own column.  float32: eight scalar LDS reads.
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(8))) short s16x8;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

template <bool ACC_ORDER>
__device__ __forceinline__ bf16x8 ld_tile_t(const bf16* tile, int row0, int col0) {
    const int l = threadIdx.x & 63;
    const int i = l & 15;
    const int hf = l >> 5;
    const int gp = (l >> 4) & 1;
    const int r = row0 + (ACC_ORDER ? 4 * hf : 8 * hf) + (i >> 2);
    const int col = col0 + 16 * gp + 4 * (i & 3);
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(tile + toff<bf16>(r, col)));
    const s16x4 hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(tile + toff<bf16>(r + (ACC_ORDER ? 8 : 4), col)));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}
template <bool ACC_ORDER>
__device__ __forceinline__ f32x8 ld_tile_t(const float* tile, int row0, int col0) {
    const int l = threadIdx.x & 63;
    const int c = l & 31;
    const int hf = l >> 5;
    f32x8 v;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int r = row0 + (ACC_ORDER ? 8 * (t >> 2) + 4 * hf + (t & 3) : 8 * hf + t);
        v[t] = tile[toff<float>(r, col0 + c)];
    }
    return v;
}

// Transposed operand of a 16 x 16 product from a column-slab tile: row m of
// the A operand is tile column col0 + m (m = lane % 16), and k-slot t of lane
// group g = lane / 16 is tile row row0 + 16*(t/4) + 4*g + (t%4), the order in
// which two stacked 16 x 16 accumulator tiles hold their rows.  bf16: two
// ds_read_b64_tr_b16 (lane i of a 16-lane group addresses row base + i/4 at
// column col0 + 4*(i%4) and receives four rows of column col0 + i); float32:
// eight scalar LDS reads.
__device__ __forceinline__ bf16x8 ld_tile_t16(const bf16* tile, int row0, int col0) {
    const int l = threadIdx.x & 63;
    const int i = l & 15;
    const int r = row0 + 4 * (l >> 4) + (i >> 2);
    const int col = col0 + 4 * (i & 3);
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(tile + toff<bf16>(r, col)));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(tile + toff<bf16>(r + 16, col)));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ f32x8 ld_tile_t16(const float* tile, int row0, int col0) {
    const int l = threadIdx.x & 63;
    f32x8 v;
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = tile[toff<float>(row0 + 16 * (t >> 2) + 4 * (l >> 4) + (t & 3), col0 + (l & 15))];
    return v;
}

// A 16-byte unit of a row, as it moves through registers when the kernel
// scales rows while staging them (fixed heads).
__device__ __forceinline__ u32x4 ld_unit(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
// Store a 16-byte unit scaled by e (rounded once to the element type).
__device__ __forceinline__ void st_unit_scaled(bf16* dst, const u32x4& a, float e) {
    u32x4 o;
#pragma unroll
    for (int m = 0; m < 4; ++m)
        o[m] = pack_bf16(__uint_as_float(a[m] << 16) * e, __uint_as_float(a[m] & 0xffff0000u) * e);
    *reinterpret_cast<u32x4*>(dst) = o;
}
__device__ __forceinline__ void st_unit_scaled(float* dst, const u32x4& a, float e) {
    u32x4 o;
#pragma unroll
    for (int m = 0; m < 4; ++m) o[m] = __float_as_uint(__uint_as_float(a[m]) * e);
    *reinterpret_cast<u32x4*>(dst) = o;
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

// ---------------------------------------------------------------------------
// Workgroup -> (level, batch b, query head h) for grids of n_levels x B x Hs
// x group workgroups, where a slice (b, s) of the B x Hs slices carries
// `group` query heads h = s * group + i that share its data (group = 1: one
// head per slice; grouped-query attention: the query heads of one key/value
// head).  Workgroups are dealt to the 8 XCDs in turn (workgroup i to XCD
// i mod 8), so when the slices split evenly over the XCDs:
//   * every workgroup of a slice runs on one XCD (the slice's K and V come
//     into one L2 only);
//   * slices are dealt to the XCDs in order of decreasing work, back and
//     forth (XCD 0..7, then 7..0, ...): order(k) is the k-th heaviest head
//     (or key/value head), and the slice of rank m is (b = m % B,
//     order(m / B)), so every XCD gets an equal share of ordinary and fixed
//     heads;
//   * an XCD works through its slices level by level.
// Otherwise workgroups go level by level, each level dealing the slices in
// order of decreasing work, rotated by one position per level.  Level 0 is
// dispatched first; kernels map it to their longest blocks.
// ---------------------------------------------------------------------------
struct SliceOf {
    int level, b, h;
};

template <typename Order>
__device__ __forceinline__ SliceOf slice_of(unsigned blk, int B, int Hs, int group, Order order) {
    const int n_slices = B * Hs;
    SliceOf s;
    if ((n_slices & 7) == 0) {
        const int x = (int)(blk & 7);
        const int j = (int)(blk >> 3);
        const int per_level = (n_slices >> 3) * group;  // workgroups of one level on one XCD
        s.level = j / per_level;
        const int within = j % per_level;
        const int li = within / group;  // this XCD's li-th slice
        const int m = li * 8 + ((li & 1) ? 7 - x : x);
        s.b = m % B;
        s.h = order(m / B) * group + within % group;
    } else {
        // Slices in order of decreasing work, rotated by one position per
        // level, so that every XCD sees every slice over the levels (with a
        // fixed order, a slice count such as 12 sends the same slices to the
        // same XCD at every other level).
        const int n_bh = n_slices * group;
        s.level = (int)(blk / n_bh);
        const int k = (int)((blk % n_bh + (unsigned)s.level) % n_bh);
        const int m = k / group;  // rank of the slice by work
        s.b = m % B;
        s.h = order(m / B) * group + k % group;
    }
    return s;
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
