// Backward of the hybrid causal-attention layer for the loss sum(O * dO).
//
// Split as the paper describes (Appendix "Mixed-head execution and numerical
// checks"): key-block programs accumulate dV for every head and dK for
// ordinary heads; a separate query-block pass produces dQ, for ordinary heads
// only.  Fixed heads follow dV = P^T dO (Section "Replacement schedules and
// fused execution") and get exact zeros in dQ and dK, since the pattern
// reads neither queries nor keys.
//
// Ordinary heads use the FlashAttention-2 recurrences: with P recomputed from
// the forward's LSE, dP = dO V^T, D_i = rowsum(dO * O)_i (formed by the
// query-block pass, which runs first, or by a row pre-pass), dS = P * (dP - D),
// dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d).
#pragma once

#include "saf_common.h"

namespace saf {

struct BwdArgs {
    const void* q;
    const void* k;
    const void* v;
    const void* o;
    const void* dO;
    const float* lse;
    const float* a;
    const float* r;
    void* dq;
    void* dk;
    void* dv;
    float* dsum;  // workspace: D, [B, H, N]
    uint64_t fixed_mask;
    int B, H, N, ld_prior, n_blocks;
    float scale;       // 1 / sqrt(d)
    float scale_log2;  // log2(e) / sqrt(d)
    int dq_writes_dsum;  // query-block pass: form D from O and dO and write it (no row pre-pass)
    unsigned char head_order[64];  // ordinary heads, then fixed heads (slice_of)
};

// ---------------------------------------------------------------------------
// Row pre-pass: D[b,h,i] = sum_c dO[b,h,i,c] * O[b,h,i,c] (ordinary heads).
// Eight lanes per row, 32 rows per workgroup.
// ---------------------------------------------------------------------------
constexpr int PRE_THREADS = 256;
constexpr int PRE_ROWS = PRE_THREADS / 8;

template <typename T>
__global__ __launch_bounds__(PRE_THREADS) void bwd_pre_kernel(BwdArgs p) {
    const size_t total = (size_t)p.B * p.H * p.N;
    const size_t row = (size_t)blockIdx.x * PRE_ROWS + (threadIdx.x >> 3);
    const int part = threadIdx.x & 7;
    float acc = 0.0f;
    bool live = row < total;
    if (live) {
        const int h = (int)((row / p.N) % p.H);
        live = !((p.fixed_mask >> h) & 1ull);
    }
    if (live) {
        const T* o = reinterpret_cast<const T*>(p.o) + row * HEAD_DIM + part * 8;
        const T* g = reinterpret_cast<const T*>(p.dO) + row * HEAD_DIM + part * 8;
        const typename Vec<T>::x8 ov = ld8<T>(o);
        const typename Vec<T>::x8 gv = ld8<T>(g);
#pragma unroll
        for (int t = 0; t < 8; ++t) acc += (float)ov[t] * (float)gv[t];
    }
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 4);
    if (row < total && part == 0) p.dsum[row] = acc;
}

// ---------------------------------------------------------------------------
// Key-block pass: workgroup = (b, h, 128 keys); 4 wavefronts x 32 keys,
// streaming steps of two 64-query tiles from the block's first key to N.
// KV_KB 32-key sub-blocks per wavefront: with one, a wavefront stays within
// 256 VGPRs and two of them share a SIMD.
//
// Ordinary heads: scores are formed as S (queries x keys) on 16 x 16 tiles,
// so a lane holds one key of each 16-key tile (l % 16) and eight queries of
// each 32-query half: P and dS feed directly into the B operand of
// dV^T += dO^T P and dK^T += Q^T dS, whose accumulators again hold one key
// per lane.  (With 32 x 32 tiles a lane would hold 16 queries, and read
// twice the per-row LSE and D values from LDS for the same products.)  K and
// V of the wavefront's keys stay in registers; Q and dO tiles are copied by
// buffer loads straight into column-slab LDS tiles (A operands of S and dP,
// and, through transposing reads, of the dV/dK products), double-buffered so
// the next step is in flight while this one is used.  The first step meets
// the diagonal and runs a masked body; the rest run mask-free.
//
// Fixed heads: dV[j] = sum_i P(i,j) dO[i] with P(i,j) = ea(j) er(i-j) g(i),
// ea = exp(a - A), er = exp(r - R), g(i) = exp(A + R - log Z(i)) (A: maximum
// of a over the block's keys, R: maximum of r over the offsets it meets, log Z
// from the forward's LSE).  The dO tile comes by buffer loads straight to LDS,
// unscaled; the Toeplitz band er(i-j) is kept in float32 in LDS (8 shifted
// copies, so any lane's eight consecutive offsets are aligned reads; negative
// offsets hold 0, the causal mask) beside g of the tile's rows, and the weight
// operand er(i-j) g(i) is formed in float32 per chunk and rounded once, as P
// is in the exact program; the accumulator is scaled by ea(j) at the end: no
// exponential per element.  If some row's log Z lies more than FAST_GUARD
// below A + R (g could overflow), the block runs the exact per-element
// program instead.  dK of a fixed head is written as zeros.
// ---------------------------------------------------------------------------
constexpr int KV_KB = 1;               // 32-key sub-blocks per wavefront
constexpr int KV_BN = 4 * 32 * KV_KB;  // keys per workgroup
constexpr int KV_BM = TILE_ROWS;       // queries per tile
constexpr int KV_THREADS = 256;
constexpr int KV_MASK_TILES = KV_BN / KV_BM;               // tiles that meet the diagonal
constexpr int KV_BAND = KV_BM + KV_BN - 1;                 // offsets per tile
constexpr int KV_BAND_STRIDE = (KV_BAND + 8) / 8 * 8 + 8;  // every copy 16-byte aligned
static_assert(BAND_COPIES * KV_BAND_STRIDE * 4 <= tile_elems<bf16>() * 2, "float32 band copies fit in a tile");
static_assert((KV_BM + KV_BAND + 1) * 4 <= tile_elems<bf16>() * 2, "exact-program rows fit in a tile");

struct KvLane {
    int tid, w, lane, c, hf, n, g, n0, kw, N;
};

template <typename T>
__device__ __forceinline__ void kv_store_rows(T* base, const KvLane& L, const f32x16 (&acc)[KV_KB][2],
                                              const float (&scale)[KV_KB]) {
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) {
        const int key = L.kw + 32 * kb + L.c;
        if (key >= L.N) continue;
        const float sc = scale[kb];
        T* row = base + (size_t)key * HEAD_DIM;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                st4<T>(row + 32 * db + 8 * g + 4 * L.hf, acc[kb][db][4 * g] * sc, acc[kb][db][4 * g + 1] * sc,
                       acc[kb][db][4 * g + 2] * sc, acc[kb][db][4 * g + 3] * sc);
    }
}

template <typename T>
__device__ __forceinline__ void kv_store_zero(T* base, const KvLane& L) {
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) {
        const int key = L.kw + 32 * kb + L.c;
        if (key >= L.N) continue;
        T* row = base + (size_t)key * HEAD_DIM;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g) st4<T>(row + 32 * db + 8 * g + 4 * L.hf, 0.0f, 0.0f, 0.0f, 0.0f);
    }
}

// --- ordinary heads ---------------------------------------------------------

// One query tile: q_tile / g_tile are the Q / dO tiles, rows holds
// LSE * log2(e) (first KV_BM floats) and -D (next KV_BM).  The products run on
// 16 x 16 tiles: per 32-query half, S and dP are 2 x 2 tiles (queries x the
// wavefront's 32 keys), so a lane holds eight query rows (four of each
// 16-query tile) and reads only those rows' LSE and D; the two query tiles of
// a key column, stacked, are the B operand of dV^T += dO^T P and
// dK^T += Q^T dS (k-slot t <-> query 16*(t/4) + 4*g + t%4, the order the
// transposed reads of dO and Q follow).  The row operands and row values are
// read first; the transposed operands are issued right after the S and dP
// products, so they arrive while the softmax runs.
template <typename T, bool MASK>
__device__ __forceinline__ void kv_tile(const T* q_tile, const T* g_tile, const float* rows, int mq, const KvLane& L,
                                        const typename Vec<T>::x8 (&kf)[2][2], const typename Vec<T>::x8 (&vf)[2][2],
                                        f32x4 (&dv)[4][2], f32x4 (&dk)[4][2], float scale_log2) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qs = mq + 32 * qb;
        if (MASK && (qs + 31 < L.kw || qs >= L.N)) continue;  // no query of this half sees these keys
        frag qa[2][2], ga[2][2], gta[4], qta[4];
        f32x4 l4[2], nd4[2];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
            for (int dc = 0; dc < 2; ++dc) qa[qt][dc] = ld_row<T>(q_tile, 32 * qb + 16 * qt + L.n, 32 * dc + 8 * L.g);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
            for (int dc = 0; dc < 2; ++dc) ga[qt][dc] = ld_row<T>(g_tile, 32 * qb + 16 * qt + L.n, 32 * dc + 8 * L.g);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            nd4[qt] = *reinterpret_cast<const f32x4*>(rows + KV_BM + 32 * qb + 16 * qt + 4 * L.g);
            l4[qt] = *reinterpret_cast<const f32x4*>(rows + 32 * qb + 16 * qt + 4 * L.g);
        }
        f32x4 s[2][2], dp[2][2];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
                s[qt][kt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                dp[qt][kt] = nd4[qt];  // dP - D in one go: the accumulator starts at -D of its rows
            }
#pragma unroll
        for (int dc = 0; dc < 2; ++dc)
#pragma unroll
            for (int qt = 0; qt < 2; ++qt)
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) mma16(s[qt][kt], qa[qt][dc], kf[kt][dc]);
#pragma unroll
        for (int dc = 0; dc < 2; ++dc)
#pragma unroll
            for (int qt = 0; qt < 2; ++qt)
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) mma16(dp[qt][kt], ga[qt][dc], vf[kt][dc]);
        // The transposed operands of dV and dK, in flight during the softmax.
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
            gta[dt] = ld_tile_t16(g_tile, 32 * qb, 16 * dt);
            qta[dt] = ld_tile_t16(q_tile, 32 * qb, 16 * dt);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    float pv = fast_exp2(fmaf(s[qt][kt][u], scale_log2, -l4[qt][u]));
                    if (MASK) {
                        const int row = qs + 16 * qt + 4 * L.g + u;
                        if (row < L.kw + 16 * kt + L.n) pv = 0.0f;
                    }
                    s[qt][kt][u] = pv;
                    dp[qt][kt][u] = pv * dp[qt][kt][u];
                }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            const frag pb = to_operand16<T>(s[0][kt], s[1][kt]);
            const frag sb = to_operand16<T>(dp[0][kt], dp[1][kt]);
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) {
                mma16(dv[dt][kt], gta[dt], pb);
                mma16(dk[dt][kt], qta[dt], sb);
            }
        }
    }
}

// dV or dK rows of the wavefront's 32 keys from 16 x 16 accumulators
// (acc[dt][kt]: head dimensions 16 dt .., keys 16 kt ..), times `scale`.
template <typename T>
__device__ __forceinline__ void kv_store_rows16(T* base, const KvLane& L, const f32x4 (&acc)[4][2], float scale) {
    // The lane's key column, recomputed here from the lane index (an
    // instruction pair the compiler cannot merge with the prologue's):
    // otherwise it keeps the K / V row offsets of the prologue, or the
    // column itself, live across the whole query loop for these stores and
    // spills them.
    int lane;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
    const int n = lane & 15;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
        const int key = L.kw + 16 * kt + n;
        if (key >= L.N) continue;
        T* row = base + (size_t)key * HEAD_DIM;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
            st4<T>(row + 16 * dt + 4 * L.g, acc[dt][kt][0] * scale, acc[dt][kt][1] * scale, acc[dt][kt][2] * scale,
                   acc[dt][kt][3] * scale);
    }
}

template <typename T>
__device__ __forceinline__ void kv_ordinary(const Tiles<T>& sm, const BwdArgs& p, const KvLane& L, size_t base,
                                            size_t row_base) {
    // Tiles of a step's first 64 queries: Q in t[0] / t[1], dO in t[2] / t[3];
    // of its second 64: Q in t[4] / t[5], dO in t[6] / t[7]; LSE and -D rows of
    // both in aux[0] / aux[1] (64 LSE, 64 -D, then the same for the second).
    const T* __restrict__ K = reinterpret_cast<const T*>(p.k) + base;
    const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + base;
    const __amdgpu_buffer_rsrc_t rq = slice_rsrc<T>(reinterpret_cast<const T*>(p.q) + base, L.N);
    const __amdgpu_buffer_rsrc_t rg = slice_rsrc<T>(reinterpret_cast<const T*>(p.dO) + base, L.N);
    const float* __restrict__ LSE = p.lse + row_base;
    const float* __restrict__ Dsum = p.dsum + row_base;
    static_assert(KV_KB == 1, "the ordinary program's tiles cover 32 keys per wavefront");
    typedef typename Vec<T>::x8 frag;
    // B operands of S and dP: key 16 kt + n of the wavefront, head dimensions
    // 32 dc + 8 g .. 32 dc + 8 g + 7.
    frag kf[2][2], vf[2][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
        const int key = L.kw + 16 * kt + L.n;
#pragma unroll
        for (int dc = 0; dc < 2; ++dc) {
            kf[kt][dc] = key < L.N ? ld8<T>(K + (size_t)key * HEAD_DIM + 32 * dc + 8 * L.g) : zero8<T>();
            vf[kt][dc] = key < L.N ? ld8<T>(V + (size_t)key * HEAD_DIM + 32 * dc + 8 * L.g) : zero8<T>();
        }
    }
    f32x4 dv[4][2], dk[4][2];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            dv[dt][kt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            dk[dt][kt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        }

    // Steps of two 64-query tiles (one barrier per 128 queries): the step
    // that meets the diagonal first (masked), then the rest.  Rows past N
    // arrive as zeros with LSE = +inf, so they add nothing.
    constexpr int SB = 2 * KV_BM;
    const int n_steps = (L.N - L.n0 + SB - 1) / SB;
    run_slots(
        2, 2 + n_steps - 1, [&](int i) { return i < 2 ? (i == 0 ? 0 : -1) : i - 1; },
        [&](auto buf, int t) {
            constexpr int b = decltype(buf)::value;
            const int mq = L.n0 + t * SB;
            tile_load_lds<T>(sm.t[b], rq, mq, L.w, L.lane);
            tile_load_lds<T>(sm.t[2 + b], rg, mq, L.w, L.lane);
            tile_load_lds<T>(sm.t[4 + b], rq, mq + KV_BM, L.w, L.lane);
            tile_load_lds<T>(sm.t[6 + b], rg, mq + KV_BM, L.w, L.lane);
            if (L.tid < SB) {
                const int row = mq + L.tid;
                const bool ok = row < L.N;
                float* x = sm.aux[b] + (L.tid / KV_BM) * 2 * KV_BM + (L.tid % KV_BM);
                x[0] = ok ? LSE[row] * LOG2E : INFINITY;
                x[KV_BM] = ok ? -Dsum[row] : 0.0f;
            }
        },
        [&](auto) {},
        [&](auto buf, int t, auto mask) {
            constexpr int b = decltype(buf)::value;
            const int mq = L.n0 + t * SB;
            kv_tile<T, decltype(mask)::value>(sm.t[b], sm.t[2 + b], sm.aux[b], mq, L, kf, vf, dv, dk,
                                              p.scale_log2);
            if (mq + KV_BM < L.N)
                kv_tile<T, decltype(mask)::value>(sm.t[4 + b], sm.t[6 + b], sm.aux[b] + 2 * KV_BM, mq + KV_BM, L, kf,
                                                  vf, dv, dk, p.scale_log2);
        });
    kv_store_rows16<T>(reinterpret_cast<T*>(p.dv) + base, L, dv, 1.0f);
    kv_store_rows16<T>(reinterpret_cast<T*>(p.dk) + base, L, dk, p.scale);
}

// --- fixed heads: exact per-element program (fallback) ----------------------

template <typename T>
__device__ __forceinline__ void kv_fixed_exact(const Tiles<T>& sm, const BwdArgs& p, const KvLane& L, size_t base,
                                               size_t row_base, const float* arow, const float* rrow) {
    // Tiles: dO in t[0]; LSE * log2(e) of the tile's rows and r over its
    // offsets in t[1].
    T* gt = sm.t[0];
    float* lse = reinterpret_cast<float*>(sm.t[1]);
    float* rb = lse + KV_BM;
    const T* __restrict__ dO = reinterpret_cast<const T*>(p.dO) + base;
    const float* __restrict__ LSE = p.lse + row_base;
    typedef typename Vec<T>::x8 frag;
    const int N = L.N;
    float a_key[KV_KB];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) {
        const int key = L.kw + 32 * kb + L.c;
        a_key[kb] = key < N ? arow[key] : -INFINITY;
    }
    f32x16 dv[KV_KB][2];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb)
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) dv[kb][db][v] = 0.0f;
    const int row = unit_row<T>(L.w, L.lane);
    for (int mq = L.n0; mq < N; mq += KV_BM) {
        __syncthreads();
#pragma unroll
        for (int k = 0; k < tile_units<T>(); ++k) {
            const int col = unit_col<T>(L.w, L.lane, k);
            const u32x4 z = {0u, 0u, 0u, 0u};
            const u32x4 x = mq + row < N ? ld_unit(dO + (size_t)(mq + row) * HEAD_DIM + col) : z;
            *reinterpret_cast<u32x4*>(gt + toff<T>(row, col)) = x;
        }
        if (L.tid < KV_BM) lse[L.tid] = mq + L.tid < N ? LSE[mq + L.tid] * LOG2E : INFINITY;
        for (int x = L.tid; x < KV_BAND; x += KV_THREADS) {
            const int delta = mq - L.n0 - (KV_BN - 1) + x;
            rb[x] = (delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
        }
        __syncthreads();
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            const int qs = mq + 32 * qb;
            if (qs + 31 < L.kw || qs >= N) continue;
            f32x16 pm[KV_KB];
#pragma unroll
            for (int kb = 0; kb < KV_KB; ++kb) {
                const int kl = L.kw - L.n0 + 32 * kb + L.c;  // key within the block
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int ql = 32 * qb + 8 * (v >> 2) + 4 * L.hf + (v & 3);
                    const int x = ql - kl + (KV_BN - 1);
                    pm[kb][v] = fast_exp2(fmaf(a_key[kb] + rb[x], LOG2E, -lse[ql]));
                }
            }
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                frag gta[2];
#pragma unroll
                for (int db = 0; db < 2; ++db) gta[db] = ld_tile_t<true>(gt, 32 * qb + 16 * kc, 32 * db);
#pragma unroll
                for (int kb = 0; kb < KV_KB; ++kb) {
                    const frag pb = to_operand<T>(pm[kb], 8 * kc);
#pragma unroll
                    for (int db = 0; db < 2; ++db) mma(dv[kb][db], gta[db], pb);
                }
            }
        }
    }
    float one[KV_KB];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) one[kb] = 1.0f;
    kv_store_rows<T>(reinterpret_cast<T*>(p.dv) + base, L, dv, one);
    kv_store_zero<T>(reinterpret_cast<T*>(p.dk) + base, L);
}

// --- fixed heads: factorised program ----------------------------------------

// Small per-tile values in registers between their loads (issued a tile
// ahead) and their LDS stores: log Z of one row, two band entries.
struct KvFixStage {
    float lse;    // log Z of row L.tid of the tile (L.tid < KV_BM)
    float rb[2];  // band entries
};

__device__ __forceinline__ void kvf_load(KvFixStage& st, const float* LSE, const float* rrow, int mq,
                                         const KvLane& L) {
    st.lse = (L.tid < KV_BM && mq + L.tid < L.N) ? LSE[mq + L.tid] : INFINITY;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int x = L.tid + KV_THREADS * k;
        const int delta = mq - L.n0 - (KV_BN - 1) + x;
        st.rb[k] = (x < KV_BAND && delta >= 0 && delta < L.N) ? rrow[delta] : -INFINITY;
    }
}

// gs: g of the tile's rows; band: copy s of er at s * KV_BAND_STRIDE, float32.
__device__ __forceinline__ void kvf_store(float* gs, float* band, const KvFixStage& st, const KvLane& L, float g_sh,
                                          float r_sh) {
    if (L.tid < KV_BM) gs[L.tid] = fast_exp2(fmaf(-st.lse, LOG2E, g_sh));  // 0 past N
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int x = L.tid + KV_THREADS * k;
        if (x < KV_BAND) {
            const float e = fast_exp2(fmaf(st.rb[k], LOG2E, -r_sh));
#pragma unroll
            for (int s = 0; s < BAND_COPIES; ++s)
                if (x >= s) band[s * KV_BAND_STRIDE + x - s] = e;
        }
    }
}

// dV^T += dO^T (er g) for NB batch elements at once: the weight operand of
// lane (key c, half hf) in chunk (qb, kc) is er(q - key) g(q) for its eight
// queries q, formed in float32 from the band and g and rounded once, then fed
// to the MFMAs of every batch element's dO tile (the pattern and its
// normalisers do not depend on the input).
template <typename T, int NB, bool MASK>
__device__ __forceinline__ void kvf_tile(const T* const (&dot)[NB], const float* band, const float* gs, int mq,
                                         const KvLane& L, f32x16 (&dv)[NB][KV_KB][2]) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qs = mq + 32 * qb;
        if (MASK && (qs + 31 < L.kw || qs >= L.N)) continue;
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const int col = 32 * qb + 16 * kc + 8 * L.hf;  // first query (within the tile) of this lane's slots
            const f32x4 g0 = *reinterpret_cast<const f32x4*>(gs + col);
            const f32x4 g1 = *reinterpret_cast<const f32x4*>(gs + col + 4);
            frag w[KV_KB];
#pragma unroll
            for (int kb = 0; kb < KV_KB; ++kb) {
                const int kl = L.kw - L.n0 + 32 * kb + L.c;
                const int u0 = col - kl + (KV_BN - 1);  // band index of offset (mq + col) - (n0 + kl)
                const int s = u0 & 7;
                const float* bp = band + s * KV_BAND_STRIDE + u0 - s;
                const f32x4 b0 = *reinterpret_cast<const f32x4*>(bp);
                const f32x4 b1 = *reinterpret_cast<const f32x4*>(bp + 4);
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    w[kb][t] = (T)(b0[t] * g0[t]);
                    w[kb][4 + t] = (T)(b1[t] * g1[t]);
                }
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                frag gta[2];
#pragma unroll
                for (int db = 0; db < 2; ++db) gta[db] = ld_tile_t<false>(dot[nb], 32 * qb + 16 * kc, 32 * db);
#pragma unroll
                for (int kb = 0; kb < KV_KB; ++kb)
#pragma unroll
                    for (int db = 0; db < 2; ++db) mma(dv[nb][kb][db], gta[db], w[kb]);
            }
        }
    }
}

// NB batch elements b, b + 1, .. of one fixed head and key block (slice
// offsets base + nb * slice; log Z is read from batch element b, the same
// for all).
template <typename T, int NB>
__device__ __forceinline__ void kv_fixed(const Tiles<T>& sm, const BwdArgs& p, const KvLane& L, size_t base,
                                         size_t row_base, int h) {
    // Tiles: dO of batch element nb in t[4 nb] / t[4 nb + 1] (buffer loads to
    // LDS), the float32 band in t[2] / t[3]; g of the tile's rows in aux[0] /
    // aux[1].
    const size_t slice = (size_t)p.H * p.N * HEAD_DIM;
    const size_t rows = (size_t)p.H * p.N;
    const float* __restrict__ LSE = p.lse + row_base;
    const float* __restrict__ arow = p.a + (size_t)h * p.ld_prior;
    const float* __restrict__ rrow = p.r + (size_t)h * p.ld_prior;
    const int N = L.N;

    // A: max of a over the block's keys; R: max of r over the offsets the
    // block meets (0 .. N - 1 - n0); lo: min of log Z over its rows.
    float am = -INFINITY;
    for (int j = L.tid; j < KV_BN; j += KV_THREADS)
        if (L.n0 + j < N) am = fmaxf(am, arow[L.n0 + j]);
    float rm = -INFINITY, lo = INFINITY;
    for (int j = L.tid; j < N - L.n0; j += KV_THREADS) {
        rm = fmaxf(rm, rrow[j]);
        lo = fminf(lo, LSE[L.n0 + j]);
    }
    const float A = block_max(am, sm.red);
    const float R = block_max(rm, sm.red);
    const float LO = -block_max(-lo, sm.red);
    if (!(LO - A - R >= -FAST_GUARD)) {  // some g(i) could overflow
        for (int nb = 0; nb < NB; ++nb) {
            if (nb > 0) __syncthreads();
            kv_fixed_exact<T>(sm, p, L, base + nb * slice, row_base + nb * rows, arow, rrow);
        }
        return;
    }
    const float g_sh = (A + R) * LOG2E, r_sh = R * LOG2E, a_sh = A * LOG2E;

    f32x16 dv[NB][KV_KB][2];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int kb = 0; kb < KV_KB; ++kb)
#pragma unroll
            for (int db = 0; db < 2; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) dv[nb][kb][db][v] = 0.0f;

    const int n_tiles = (N - L.n0 + KV_BM - 1) / KV_BM;
    const int n_mask = min(KV_MASK_TILES, n_tiles);
    const int P = (n_mask + 1) & ~1;
    __amdgpu_buffer_rsrc_t rg[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) rg[nb] = slice_rsrc<T>(reinterpret_cast<const T*>(p.dO) + base + nb * slice, N);
    KvFixStage st;
    run_slots(
        P, P + n_tiles - n_mask, [&](int i) { return i < P ? (i < n_mask ? i : -1) : n_mask + (i - P); },
        [&](auto buf, int t) {
            constexpr int b = decltype(buf)::value;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) tile_load_lds<T>(sm.t[4 * nb + b], rg[nb], L.n0 + t * KV_BM, L.w, L.lane);
            kvf_load(st, LSE, rrow, L.n0 + t * KV_BM, L);
        },
        [&](auto buf) {
            constexpr int b = decltype(buf)::value;
            kvf_store(sm.aux[b], reinterpret_cast<float*>(sm.t[2 + b]), st, L, g_sh, r_sh);
        },
        [&](auto buf, int t, auto mask) {
            constexpr int b = decltype(buf)::value;
            const T* dot[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) dot[nb] = sm.t[4 * nb + b];
            kvf_tile<T, NB, decltype(mask)::value>(dot, reinterpret_cast<const float*>(sm.t[2 + b]), sm.aux[b],
                                                   L.n0 + t * KV_BM, L, dv);
        });
    float ea[KV_KB];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) {
        const int key = L.kw + 32 * kb + L.c;
        ea[kb] = key < N ? fast_exp2(fmaf(arow[key], LOG2E, -a_sh)) : 0.0f;
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        kv_store_rows<T>(reinterpret_cast<T*>(p.dv) + base + nb * slice, L, dv[nb], ea);
        kv_store_zero<T>(reinterpret_cast<T*>(p.dk) + base + nb * slice, L);
    }
}

template <typename T>
__global__ __launch_bounds__(KV_THREADS) __attribute__((amdgpu_waves_per_eu(sizeof(T) == 2 ? 2 : 1))) void bwd_kv_kernel(BwdArgs p) {
    __shared__ __attribute__((aligned(16))) T t0[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t1[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t2[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t3[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t4[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t5[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t6[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t7[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) float x0[4 * KV_BM];
    __shared__ __attribute__((aligned(16))) float x1[4 * KV_BM];
    __shared__ float red[4];
    const Tiles<T> sm = {{t0, t1, t2, t3, t4, t5, t6, t7}, {x0, x1}, red};
    const SliceOf sl = slice_of(blockIdx.x, p.B, p.H, 1, [&](int k) { return (int)p.head_order[k]; });
    const int kblk = sl.level;  // ascending: longest first
    const int h = sl.h;
    const int bh = sl.b * p.H + h;
    KvLane L;
    L.tid = threadIdx.x;
    L.w = L.tid >> 6;
    L.lane = L.tid & 63;
    L.c = L.tid & 31;
    L.hf = (L.tid >> 5) & 1;
    L.n = L.tid & 15;
    L.g = (L.tid >> 4) & 3;
    L.n0 = kblk * KV_BN;
    L.kw = L.n0 + 32 * KV_KB * L.w;
    L.N = p.N;
    if ((p.fixed_mask >> h) & 1ull) {
        // Batch elements pair up (b0 = b with its low bit cleared, b0 + 1):
        // one workgroup of the pair, the one whose batch parity matches the
        // key block's, forms the pattern's weights once and applies them to
        // both, so the active workgroups alternate between the pair's two
        // places in the grid from block to block.  An unpaired last element
        // (odd B) is served alone.  The forward does not pair: its fixed
        // program forms fewer weights per product, and holding two elements'
        // accumulators costs the whole forward kernel registers.
        const int b0 = sl.b & ~1;
        const bool paired = b0 + 1 < p.B;
        if (paired && (sl.b & 1) != (kblk & 1)) return;
        const size_t base = ((size_t)b0 * p.H + h) * p.N * HEAD_DIM;
        const size_t row_base = ((size_t)b0 * p.H + h) * p.N;
        if (paired)
            kv_fixed<T, 2>(sm, p, L, base, row_base, h);
        else
            kv_fixed<T, 1>(sm, p, L, base, row_base, h);
    } else {
        kv_ordinary<T>(sm, p, L, (size_t)bh * p.N * HEAD_DIM, (size_t)bh * p.N);
    }
}

// ---------------------------------------------------------------------------
// Query-block pass (ordinary heads): workgroup = (b, h, 128 queries); 4
// wavefronts x 32 queries, streaming key tiles of 64 up to the diagonal,
// copied by buffer loads straight into double-buffered column-slab LDS tiles.
// S^T (keys x queries) puts one query per lane, so LSE and D are per-lane
// scalars and dS^T feeds the B operand of dQ^T += K^T dS^T (K^T through
// transposing LDS reads).  Tiles below the block's first query run a
// mask-free body.  Workgroups of fixed heads only write zeros.
// ---------------------------------------------------------------------------
constexpr int DQ_BM = 128;
constexpr int DQ_BN = TILE_ROWS;
constexpr int DQ_THREADS = 256;

struct DqLane {
    int tid, w, lane, c, hf, m0, q0, qq, N;
};

template <typename T, bool MASK>
__device__ __forceinline__ void dq_tile(const T* kt, const T* vt, int n0, const DqLane& L,
                                        const typename Vec<T>::x8 (&qf)[4], const typename Vec<T>::x8 (&gf)[4],
                                        float lse2, float dsum, f32x16 (&dq)[2], float scale_log2) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int k0 = n0 + 32 * kb;
        if (MASK && !(k0 < L.q0 + 32 && k0 < L.N)) continue;  // keys wholly after this wavefront's queries
        f32x16 s, dp;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            s[v] = 0.0f;
            dp[v] = 0.0f;
        }
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) {
            mma(s, ld_row<T>(kt, 32 * kb + L.c, 16 * dc + 8 * L.hf), qf[dc]);
            mma(dp, ld_row<T>(vt, 32 * kb + L.c, 16 * dc + 8 * L.hf), gf[dc]);
        }
        // K^T operands of dQ, in flight during the softmax.
        frag kta[2][2];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
            for (int db = 0; db < 2; ++db) kta[kc][db] = ld_tile_t<true>(kt, 32 * kb + 16 * kc, 32 * db);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            float pv = fast_exp2(fmaf(s[v], scale_log2, -lse2));
            if (MASK && k0 == L.q0) {
                const int kk = k0 + 8 * (v >> 2) + 4 * L.hf + (v & 3);
                if (kk > L.qq) pv = 0.0f;
            }
            s[v] = pv * (dp[v] - dsum);  // dS^T
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const frag sb = to_operand<T>(s, 8 * kc);
#pragma unroll
            for (int db = 0; db < 2; ++db) mma(dq[db], kta[kc][db], sb);
        }
    }
}

template <typename T>
__global__ __launch_bounds__(DQ_THREADS) __attribute__((amdgpu_waves_per_eu(3))) void bwd_dq_kernel(BwdArgs p) {
    __shared__ __attribute__((aligned(16))) T t0[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t1[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t2[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t3[tile_elems<T>()];
    const SliceOf sl = slice_of(blockIdx.x, p.B, p.H, 1, [&](int k) { return (int)p.head_order[k]; });
    const int qblk = p.n_blocks - 1 - sl.level;  // longest first
    const int h = sl.h;
    const int bh = sl.b * p.H + h;
    const bool fixed = (p.fixed_mask >> h) & 1ull;
    const int N = p.N;
    const size_t base = (size_t)bh * N * HEAD_DIM;
    T* __restrict__ dQ = reinterpret_cast<T*>(p.dq) + base;
    DqLane L;
    L.tid = threadIdx.x;
    L.w = L.tid >> 6;
    L.lane = L.tid & 63;
    L.c = L.tid & 31;
    L.hf = (L.tid >> 5) & 1;
    L.m0 = qblk * DQ_BM;
    L.q0 = L.m0 + 32 * L.w;
    L.qq = L.q0 + L.c;
    L.N = N;

    if (fixed) {  // the whole workgroup takes this branch
        for (int id = L.tid; id < DQ_BM * (HEAD_DIM / 8); id += DQ_THREADS) {
            const int row = L.m0 + id / (HEAD_DIM / 8);
            if (row < N) st8<T>(dQ + (size_t)row * HEAD_DIM + (id % (HEAD_DIM / 8)) * 8, zero8<T>());
        }
        return;
    }

    // Tiles: K in t0 / t1, V in t2 / t3.
    const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + base;
    const T* __restrict__ dO = reinterpret_cast<const T*>(p.dO) + base;
    const __amdgpu_buffer_rsrc_t rk = slice_rsrc<T>(reinterpret_cast<const T*>(p.k) + base, N);
    const __amdgpu_buffer_rsrc_t rv = slice_rsrc<T>(reinterpret_cast<const T*>(p.v) + base, N);

    typedef typename Vec<T>::x8 frag;
    frag qf[4], gf[4];
#pragma unroll
    for (int dc = 0; dc < 4; ++dc) {
        qf[dc] = L.qq < N ? ld8<T>(Q + (size_t)L.qq * HEAD_DIM + 16 * dc + 8 * L.hf) : zero8<T>();
        gf[dc] = L.qq < N ? ld8<T>(dO + (size_t)L.qq * HEAD_DIM + 16 * dc + 8 * L.hf) : zero8<T>();
    }
    const float lse2 = L.qq < N ? p.lse[(size_t)bh * N + L.qq] * LOG2E : INFINITY;
    float dsum;
    if (p.dq_writes_dsum) {
        // D_i = sum_c dO * O of this lane's query, from the dO fragments
        // already in registers and O's matching columns.
        const T* __restrict__ Orow = reinterpret_cast<const T*>(p.o) + base + (size_t)L.qq * HEAD_DIM;
        float part = 0.0f;
        if (L.qq < N) {
#pragma unroll
            for (int dc = 0; dc < 4; ++dc) part = dot8(ld8<T>(Orow + 16 * dc + 8 * L.hf), gf[dc], part);
        }
        dsum = pair_sum(part);
        if (L.qq < N && L.hf == 0) p.dsum[(size_t)bh * N + L.qq] = dsum;
    } else {
        dsum = L.qq < N ? p.dsum[(size_t)bh * N + L.qq] : 0.0f;
    }

    f32x16 dq[2];
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) dq[db][v] = 0.0f;

    // Slots: the tiles that meet the diagonal first (masked), then the tiles
    // wholly below the block's first query.
    const int n_tiles = (min(L.m0 + DQ_BM, N) + DQ_BN - 1) / DQ_BN;
    const int n_full = L.m0 / DQ_BN;
    const int n_mask = n_tiles - n_full;
    const int P = (n_mask + 1) & ~1;
    T* const kt[2] = {t0, t1};
    T* const vt[2] = {t2, t3};
    run_slots(
        P, P + n_full, [&](int i) { return i < P ? (i < n_mask ? n_full + i : -1) : i - P; },
        [&](auto buf, int t) {
            tile_load_lds<T>(kt[decltype(buf)::value], rk, t * DQ_BN, L.w, L.lane);
            tile_load_lds<T>(vt[decltype(buf)::value], rv, t * DQ_BN, L.w, L.lane);
        },
        [&](auto) {},
        [&](auto buf, int t, auto mask) {
            dq_tile<T, decltype(mask)::value>(kt[decltype(buf)::value], vt[decltype(buf)::value], t * DQ_BN, L, qf,
                                              gf, lse2, dsum, dq, p.scale_log2);
        });

    if (L.qq < N) {
        T* row = dQ + (size_t)L.qq * HEAD_DIM;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                st4<T>(row + 32 * db + 8 * g + 4 * L.hf, dq[db][4 * g] * p.scale, dq[db][4 * g + 1] * p.scale,
                       dq[db][4 * g + 2] * p.scale, dq[db][4 * g + 3] * p.scale);
    }
}

}  // namespace saf
