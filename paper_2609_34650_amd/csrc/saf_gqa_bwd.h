// Backward of the grouped-query hybrid layer for head dimensions 64, 96 and
// 128, for the loss sum(O * dO) (the training side of the layouts the
// grouped-query forward serves: Appendix "Replacement in pretrained models",
// subsection "GQA prefill measurements"; Appendix "Mixed-head execution
// and numerical checks", whose grouped-query path keeps every shared
// key/value head and maps each ordinary query head to its group).
//
// Q, O, dO, dQ: [B, Hq, N, D]; K, V, dK, dV: [B, Hkv, N, D]; query head h
// reads key/value head h / (Hq / Hkv).  A shared head's dK and dV are sums
// over the query heads of its group: ordinary heads add dS^T Q / sqrt(D) to
// dK and P^T dO to dV (the FlashAttention-2 recurrences of the layer's own
// backward); fixed heads add P^T dO to dV only (factorised into a Toeplitz
// band times a scaled dO, or, behind a guard, P(i, j) = exp(a[j] + r[i - j] -
// log Z(i)) per entry); they get exact zeros in dQ.
//
// Launches: the query-block pass (workgroup = (b, query head, 128 queries)),
// which also forms D_i = sum_c dO * O of the ordinary heads' rows; then the
// key-block pass (workgroup = (b, key/value head, 128 keys), one 32-key block
// per wavefront, looping over the group's query heads with dK and dV
// accumulated in registers).  At D = 128 the key-block pass is two launches,
// one for dK and one for dV: both gradients' accumulators plus the block's K
// and V fragments would not leave room for two wavefronts per SIMD.
#pragma once

#include "saf_common.h"

namespace saf {

struct GqaBwdArgs {
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
    float* dsum;  // workspace: D, [B, Hq, N], written by the query-block pass, read by the key-block pass
    uint64_t fixed_mask;
    int B, Hq, Hkv, N, ld_prior, n_blocks;
    float scale;       // 1 / sqrt(D)
    float scale_log2;  // log2(e) / sqrt(D)
    unsigned char kv_order[64];  // key/value heads by decreasing work (slice_of)
};

// ---------------------------------------------------------------------------
// Key-block pass.  A lane holds one key (l % 32) of its wavefront's 32 and,
// for ordinary heads, forms S = Q K^T with queries in accumulator rows, so P
// and dS feed the B operands of dV^T += dO^T P and dK^T += Q^T dS directly.
// K and V of the wavefront's keys stay in registers; Q and dO tiles of 64
// queries come by buffer loads straight to LDS, double-buffered.
// ---------------------------------------------------------------------------
constexpr int GKV_BN = 128;  // keys per workgroup
constexpr int GKV_BM = TILE_ROWS;  // queries per tile
constexpr int GKV_THREADS = 256;
constexpr int GKV_MASK_TILES = GKV_BN / GKV_BM;
constexpr int GKV_BAND = GKV_BM + GKV_BN - 1;  // offsets met by one tile

struct GkvLane {
    int tid, w, lane, c, hf, n0, kw, N;
};

// The gradients one key-block launch accumulates.
enum GkvPart { GKV_BOTH = 0, GKV_DK = 1, GKV_DV = 2 };
template <int D> constexpr bool gkv_split() { return D > 96; }

template <typename T, int D, int PART, bool MASK>
__device__ __forceinline__ void gkv_tile(const T* qt, const T* gt, const float* rows, int mq, const GkvLane& L,
                                         const typename Vec<T>::x8 (&kf)[D / 16],
                                         const typename Vec<T>::x8 (&vf)[D / 16], f32x16 (&dv)[D / 32],
                                         f32x16 (&dk)[D / 32], float scale_log2) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qs = mq + 32 * qb;
        if (MASK && (qs + 31 < L.kw || qs >= L.N)) continue;  // no query of this half sees these keys
        f32x16 s, dp;
#pragma unroll
        for (int v = 0; v < 16; ++v) s[v] = 0.0f;
#pragma unroll
        for (int dc = 0; dc < D / 16; ++dc) mma(s, ld_row<T>(qt, 32 * qb + L.c, 16 * dc + 8 * L.hf), kf[dc]);
        if constexpr (PART != GKV_DV) {
            // dP - D in one go: the accumulator starts at -D of its rows.
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const f32x4 nd4 = *reinterpret_cast<const f32x4*>(rows + GKV_BM + 32 * qb + 8 * g + 4 * L.hf);
#pragma unroll
                for (int u = 0; u < 4; ++u) dp[4 * g + u] = nd4[u];
            }
#pragma unroll
            for (int dc = 0; dc < D / 16; ++dc) mma(dp, ld_row<T>(gt, 32 * qb + L.c, 16 * dc + 8 * L.hf), vf[dc]);
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 l4 = *reinterpret_cast<const f32x4*>(rows + 32 * qb + 8 * g + 4 * L.hf);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int v = 4 * g + u;
                float pv = fast_exp2(fmaf(s[v], scale_log2, -l4[u]));
                if (MASK && qs + 8 * g + 4 * L.hf + u < L.kw + L.c) pv = 0.0f;
                s[v] = pv;
                if constexpr (PART != GKV_DV) dp[v] = pv * dp[v];
            }
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            if constexpr (PART != GKV_DK) {
                const frag pb = to_operand<T>(s, 8 * kc);
#pragma unroll
                for (int db = 0; db < D / 32; ++db) mma(dv[db], ld_tile_t<true>(gt, 32 * qb + 16 * kc, 32 * db), pb);
            }
            if constexpr (PART != GKV_DV) {
                const frag sb = to_operand<T>(dp, 8 * kc);
#pragma unroll
                for (int db = 0; db < D / 32; ++db) mma(dk[db], ld_tile_t<true>(qt, 32 * qb + 16 * kc, 32 * db), sb);
            }
        }
    }
}

// Fixed query head, one tile: dV^T += dO^T P with P evaluated per entry.
// gt: the dO tile; lse2: log Z * log2(e) of the tile's rows; rb: r over the
// offsets the tile meets (rb[x] = r(mq - n0 - 127 + x), -inf outside
// 0 .. N - 1, which masks keys after the query).
template <typename T, int D>
__device__ __forceinline__ void gkv_fixed_tile(const T* gt, const float* lse2, const float* rb, int mq, float a_key,
                                               const GkvLane& L, f32x16 (&dv)[D / 32]) {
    typedef typename Vec<T>::x8 frag;
    const int kl = L.kw - L.n0 + L.c;  // key within the block
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qs = mq + 32 * qb;
        if (qs + 31 < L.kw || qs >= L.N) continue;  // no query of this half sees these keys
        f32x16 pm;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse2 + 32 * qb + 8 * g + 4 * L.hf);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int ql = 32 * qb + 8 * g + 4 * L.hf + u;
                pm[4 * g + u] = fast_exp2(fmaf(a_key + rb[ql - kl + (GKV_BN - 1)], LOG2E, -l4[u]));
            }
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const frag pb = to_operand<T>(pm, 8 * kc);
#pragma unroll
            for (int db = 0; db < D / 32; ++db) mma(dv[db], ld_tile_t<true>(gt, 32 * qb + 16 * kc, 32 * db), pb);
        }
    }
}

// Fixed query head, factorised (the layer's key-block program): dV[j] +=
// ea(j) sum_i er(i - j) g(i) dO[i] with ea = exp(a - A), er = exp(r - R),
// g(i) = exp(A + R - log Z(i)) (A: maximum of a over the block's keys, R:
// maximum of r over the offsets it meets).  The dO tile comes by buffer
// loads to LDS unscaled; the Toeplitz band er is kept in float32 in LDS
// (eight shifted copies, so every 8-entry read is aligned; negative offsets
// hold 0) beside g of the tile's rows, and the weight operand er(i - j) g(i)
// is formed in float32 per chunk and rounded once; the head's sum is scaled
// by ea(j) once at the end: no exponential per entry.
constexpr int GKV_BAND_STRIDE = (GKV_BAND + 8) / 8 * 8 + 8;  // every copy 32-byte aligned

struct GkvFixStage {
    float lse;  // log Z of row L.tid of the tile (L.tid < GKV_BM)
    float rb;   // one band entry
};

__device__ __forceinline__ void gkvf_load(GkvFixStage& st, const float* LSE, const float* rrow, int mq,
                                          const GkvLane& L) {
    st.lse = (L.tid < GKV_BM && mq + L.tid < L.N) ? LSE[mq + L.tid] : INFINITY;
    const int delta = mq - L.n0 - (GKV_BN - 1) + L.tid;
    st.rb = (L.tid < GKV_BAND && delta >= 0 && delta < L.N) ? rrow[delta] : -INFINITY;
}

// gs: g of the tile's rows; band: copy s of er at s * GKV_BAND_STRIDE.
__device__ __forceinline__ void gkvf_store(float* gs, float* band, const GkvFixStage& st, const GkvLane& L,
                                           float g_sh, float r_sh) {
    if (L.tid < GKV_BM) gs[L.tid] = fast_exp2(fmaf(-st.lse, LOG2E, g_sh));  // 0 past N
    if (L.tid < GKV_BAND) {
        const float e = fast_exp2(fmaf(st.rb, LOG2E, -r_sh));
#pragma unroll
        for (int s = 0; s < BAND_COPIES; ++s)
            if (L.tid >= s) band[s * GKV_BAND_STRIDE + L.tid - s] = e;
    }
}

template <typename T, int D>
__device__ __forceinline__ void gkvf_tile(const T* dot, const float* band, const float* gs, int mq,
                                          const GkvLane& L, f32x16 (&acc)[D / 32]) {
    typedef typename Vec<T>::x8 frag;
    const int kl = L.kw - L.n0 + L.c;  // key within the block
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qs = mq + 32 * qb;
        if (qs + 31 < L.kw || qs >= L.N) continue;  // no query of this half sees these keys
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const int col = 32 * qb + 16 * kc + 8 * L.hf;  // this lane's first query within the tile
            const int u0 = col - kl + (GKV_BN - 1);       // band index of its first slot
            const int s = u0 & 7;
            const float* bp = band + s * GKV_BAND_STRIDE + u0 - s;
            const f32x4 b0 = *reinterpret_cast<const f32x4*>(bp);
            const f32x4 b1 = *reinterpret_cast<const f32x4*>(bp + 4);
            const f32x4 g0 = *reinterpret_cast<const f32x4*>(gs + col);
            const f32x4 g1 = *reinterpret_cast<const f32x4*>(gs + col + 4);
            frag wt;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                wt[t] = (T)(b0[t] * g0[t]);
                wt[4 + t] = (T)(b1[t] * g1[t]);
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db) mma(acc[db], ld_tile_t<false>(dot, 32 * qb + 16 * kc, 32 * db), wt);
        }
    }
}

template <typename T, int D>
__device__ __forceinline__ void gkv_store(T* base, const GkvLane& L, const f32x16 (&acc)[D / 32], float sc) {
    const int key = L.kw + L.c;
    if (key >= L.N) return;
    T* row = base + (size_t)key * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g)
            st4<T>(row + 32 * db + 8 * g + 4 * L.hf, acc[db][4 * g] * sc, acc[db][4 * g + 1] * sc,
                   acc[db][4 * g + 2] * sc, acc[db][4 * g + 3] * sc);
}

template <typename T, int D, int PART>
__global__ __launch_bounds__(GKV_THREADS) __attribute__((amdgpu_waves_per_eu(sizeof(T) == 2 ? 2 : 1))) void gqa_bwd_kv_kernel(
    GqaBwdArgs p) {
    static_assert((PART == GKV_BOTH) != gkv_split<D>(), "D = 128 runs the key-block pass as two launches");
    __shared__ __attribute__((aligned(16))) T q0s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T q1s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T g0s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T g1s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) float x0[2 * GKV_BM];
    __shared__ __attribute__((aligned(16))) float x1[2 * GKV_BM];
    __shared__ __attribute__((aligned(16))) float f0[GKV_BM + GKV_BAND + 1];
    __shared__ __attribute__((aligned(16))) float f1[GKV_BM + GKV_BAND + 1];
    __shared__ float red[4];
    static_assert(BAND_COPIES * GKV_BAND_STRIDE * 4 <= tile_elems<T, D>() * (int)sizeof(T),
                  "float32 band copies fit in a tile");
    const SliceOf sl = slice_of(blockIdx.x, p.B, p.Hkv, 1, [&](int k) { return (int)p.kv_order[k]; });
    const int kblk = sl.level;  // ascending: longest first
    const int b = sl.b, hkv = sl.h;
    const int group = p.Hq / p.Hkv;
    const int N = p.N;
    GkvLane L;
    L.tid = threadIdx.x;
    L.w = __builtin_amdgcn_readfirstlane(L.tid >> 6);
    L.lane = L.tid & 63;
    L.c = L.tid & 31;
    L.hf = (L.tid >> 5) & 1;
    L.n0 = kblk * GKV_BN;
    L.kw = L.n0 + 32 * L.w;
    L.N = N;
    typedef typename Vec<T>::x8 frag;
    const size_t kvbase = ((size_t)b * p.Hkv + hkv) * N * D;
    const int key = L.kw + L.c;

    f32x16 dv[D / 32], dk[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) dv[db][v] = 0.0f;
    const uint64_t all = (group == 64) ? ~0ull : ((1ull << group) - 1);
    const uint64_t gmask = (p.fixed_mask >> (hkv * group)) & all;
    const int n_tiles = (N - L.n0 + GKV_BM - 1) / GKV_BM;
    const int n_mask = min(GKV_MASK_TILES, n_tiles);
    const int P = (n_mask + 1) & ~1;
    // Fixed query heads first (only dV is live), then the ordinary ones with K
    // and V of the block's keys in registers.
    for (int i = 0; i < group; ++i) {
        if (PART == GKV_DK || !((gmask >> i) & 1ull)) continue;  // fixed heads add to dV only
        const int h = hkv * group + i;
        const size_t qbase = ((size_t)b * p.Hq + h) * N * D;
        const size_t row_base = ((size_t)b * p.Hq + h) * N;
        const float* __restrict__ LSE = p.lse + row_base;
        const __amdgpu_buffer_rsrc_t rg = slice_rsrc<T, D>(reinterpret_cast<const T*>(p.dO) + qbase, N);
        const float* arow = p.a + (size_t)h * p.ld_prior;
        const float* rrow = p.r + (size_t)h * p.ld_prior;
        const float a_key = key < N ? arow[key] : -INFINITY;
        // A: max of a over the block's keys; R: max of r over the offsets
        // the block meets (0 .. N - 1 - n0); LO: min of log Z over its rows.
        float am = -INFINITY, rm = -INFINITY, lo = INFINITY;
        for (int j = L.tid; j < GKV_BN; j += GKV_THREADS)
            if (L.n0 + j < N) am = fmaxf(am, arow[L.n0 + j]);
        for (int j = L.tid; j < N - L.n0; j += GKV_THREADS) {
            rm = fmaxf(rm, rrow[j]);
            lo = fminf(lo, LSE[L.n0 + j]);
        }
        const float A = block_max(am, red);
        const float R = block_max(rm, red);
        const float LO = -block_max(-lo, red);
        if (LO - A - R >= -FAST_GUARD) {  // no g(i) can overflow
            const float g_sh = (A + R) * LOG2E, r_sh = R * LOG2E;
            f32x16 acc[D / 32];
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[db][v] = 0.0f;
            GkvFixStage st;
            run_slots(
                P, P + n_tiles - n_mask,
                [&](int s) { return s < P ? (s < n_mask ? s : -1) : n_mask + (s - P); },
                [&](auto buf, int t) {
                    tile_load_lds<T, D>(decltype(buf)::value ? g1s : g0s, rg, L.n0 + t * GKV_BM, L.w, L.lane);
                    gkvf_load(st, LSE, rrow, L.n0 + t * GKV_BM, L);
                },
                [&](auto buf) {
                    constexpr int B_ = decltype(buf)::value;
                    gkvf_store(B_ ? x1 : x0, reinterpret_cast<float*>(B_ ? q1s : q0s), st, L, g_sh, r_sh);
                },
                [&](auto buf, int t, auto) {
                    constexpr int B_ = decltype(buf)::value;
                    gkvf_tile<T, D>(B_ ? g1s : g0s, reinterpret_cast<const float*>(B_ ? q1s : q0s), B_ ? x1 : x0,
                                    L.n0 + t * GKV_BM, L, acc);
                });
            const float ea = key < N ? fast_exp2(fmaf(a_key, LOG2E, -A * LOG2E)) : 0.0f;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) dv[db][v] = fmaf(ea, acc[db][v], dv[db][v]);
            continue;
        }
        // Exact program: dO tiles by buffer loads to LDS; each buffer's LSE
        // rows and r band are written while the other buffer is in use.
        run_slots(
            P, P + n_tiles - n_mask, [&](int s) { return s < P ? (s < n_mask ? s : -1) : n_mask + (s - P); },
            [&](auto buf, int t) {
                constexpr int B_ = decltype(buf)::value;
                const int mq = L.n0 + t * GKV_BM;
                tile_load_lds<T, D>(B_ ? g1s : g0s, rg, mq, L.w, L.lane);
                float* fr = B_ ? f1 : f0;
                if (L.tid < GKV_BM) fr[L.tid] = mq + L.tid < N ? LSE[mq + L.tid] * LOG2E : INFINITY;
                if (L.tid < GKV_BAND) {
                    const int delta = mq - L.n0 - (GKV_BN - 1) + L.tid;
                    fr[GKV_BM + L.tid] = (delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
                }
            },
            [&](auto) {},
            [&](auto buf, int t, auto) {
                constexpr int B_ = decltype(buf)::value;
                const float* fr = B_ ? f1 : f0;
                gkv_fixed_tile<T, D>(B_ ? g1s : g0s, fr, fr + GKV_BM, L.n0 + t * GKV_BM, a_key, L, dv);
            });
    }
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) dk[db][v] = 0.0f;
    if (gmask != all) {
        const T* __restrict__ K = reinterpret_cast<const T*>(p.k) + kvbase;
        const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + kvbase;
        frag kf[D / 16], vf[D / 16];
#pragma unroll
        for (int dc = 0; dc < D / 16; ++dc) {
            kf[dc] = key < N ? ld8<T>(K + (size_t)key * D + 16 * dc + 8 * L.hf) : zero8<T>();
            vf[dc] = (PART != GKV_DV && key < N) ? ld8<T>(V + (size_t)key * D + 16 * dc + 8 * L.hf) : zero8<T>();
        }
        for (int i = 0; i < group; ++i) {
            if ((gmask >> i) & 1ull) continue;
            const int h = hkv * group + i;
            const size_t qbase = ((size_t)b * p.Hq + h) * N * D;
            const size_t row_base = ((size_t)b * p.Hq + h) * N;
            const float* __restrict__ LSE = p.lse + row_base;
            const __amdgpu_buffer_rsrc_t rg = slice_rsrc<T, D>(reinterpret_cast<const T*>(p.dO) + qbase, N);
            const __amdgpu_buffer_rsrc_t rq = slice_rsrc<T, D>(reinterpret_cast<const T*>(p.q) + qbase, N);
            const float* __restrict__ Dsum = p.dsum + row_base;
            run_slots(
                P, P + n_tiles - n_mask, [&](int s) { return s < P ? (s < n_mask ? s : -1) : n_mask + (s - P); },
                [&](auto buf, int t) {
                    constexpr int B_ = decltype(buf)::value;
                    const int mq = L.n0 + t * GKV_BM;
                    tile_load_lds<T, D>(B_ ? q1s : q0s, rq, mq, L.w, L.lane);
                    tile_load_lds<T, D>(B_ ? g1s : g0s, rg, mq, L.w, L.lane);
                    if (L.tid < GKV_BM) {
                        float* xr = B_ ? x1 : x0;
                        const bool ok = mq + L.tid < N;
                        xr[L.tid] = ok ? LSE[mq + L.tid] * LOG2E : INFINITY;
                        xr[GKV_BM + L.tid] = ok ? -Dsum[mq + L.tid] : 0.0f;
                    }
                },
                [&](auto) {},
                [&](auto buf, int t, auto mask) {
                    constexpr int B_ = decltype(buf)::value;
                    gkv_tile<T, D, PART, decltype(mask)::value>(B_ ? q1s : q0s, B_ ? g1s : g0s, B_ ? x1 : x0,
                                                                L.n0 + t * GKV_BM, L, kf, vf, dv, dk, p.scale_log2);
                });
        }
    }
    if (PART != GKV_DK) gkv_store<T, D>(reinterpret_cast<T*>(p.dv) + kvbase, L, dv, 1.0f);
    if (PART != GKV_DV) gkv_store<T, D>(reinterpret_cast<T*>(p.dk) + kvbase, L, dk, p.scale);
}

// ---------------------------------------------------------------------------
// Query-block pass (ordinary query heads): S^T = K Q^T puts one query per
// lane (LSE and D are per-lane scalars) and dS^T feeds the B operand of
// dQ^T += K^T dS^T.  K and V tiles of the group's key/value head come by
// buffer loads straight to LDS, double-buffered.  Fixed heads write zeros.
// ---------------------------------------------------------------------------
constexpr int GDQ_BM = 128;
constexpr int GDQ_BN = TILE_ROWS;
constexpr int GDQ_THREADS = 256;

struct GdqLane {
    int tid, w, lane, c, hf, m0, q0, qq, N;
};

template <typename T, int D, bool MASK>
__device__ __forceinline__ void gdq_tile(const T* kt, const T* vt, int n0, const GdqLane& L,
                                         const typename Vec<T>::x8 (&qf)[D / 16],
                                         const typename Vec<T>::x8 (&gf)[D / 16], float lse2, float dsum,
                                         f32x16 (&dq)[D / 32], float scale_log2) {
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
        for (int dc = 0; dc < D / 16; ++dc) {
            mma(s, ld_row<T>(kt, 32 * kb + L.c, 16 * dc + 8 * L.hf), qf[dc]);
            mma(dp, ld_row<T>(vt, 32 * kb + L.c, 16 * dc + 8 * L.hf), gf[dc]);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            float pv = fast_exp2(fmaf(s[v], scale_log2, -lse2));
            if (MASK && k0 + 8 * (v >> 2) + 4 * L.hf + (v & 3) > L.qq) pv = 0.0f;
            s[v] = pv * (dp[v] - dsum);  // dS^T
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const frag sb = to_operand<T>(s, 8 * kc);
#pragma unroll
            for (int db = 0; db < D / 32; ++db) mma(dq[db], ld_tile_t<true>(kt, 32 * kb + 16 * kc, 32 * db), sb);
        }
    }
}

template <typename T, int D>
__global__ __launch_bounds__(GDQ_THREADS) __attribute__((amdgpu_waves_per_eu(2))) void gqa_bwd_dq_kernel(
    GqaBwdArgs p) {
    __shared__ __attribute__((aligned(16))) T k0s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T k1s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T v0s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T v1s[tile_elems<T, D>()];
    const int group = p.Hq / p.Hkv;
    const SliceOf sl = slice_of(blockIdx.x, p.B, p.Hkv, group, [&](int k) { return (int)p.kv_order[k]; });
    const int qblk = p.n_blocks - 1 - sl.level;  // longest first
    const int b = sl.b, h = sl.h;
    const int hkv = h / group;
    const int N = p.N;
    const size_t qbase = ((size_t)b * p.Hq + h) * N * D;
    const size_t kvbase = ((size_t)b * p.Hkv + hkv) * N * D;
    T* __restrict__ dQ = reinterpret_cast<T*>(p.dq) + qbase;
    GdqLane L;
    L.tid = threadIdx.x;
    L.w = __builtin_amdgcn_readfirstlane(L.tid >> 6);
    L.lane = L.tid & 63;
    L.c = L.tid & 31;
    L.hf = (L.tid >> 5) & 1;
    L.m0 = qblk * GDQ_BM;
    L.q0 = L.m0 + 32 * L.w;
    L.qq = L.q0 + L.c;
    L.N = N;

    if ((p.fixed_mask >> h) & 1ull) {  // the whole workgroup takes this branch
        for (int id = L.tid; id < GDQ_BM * (D / 8); id += GDQ_THREADS) {
            const int row = L.m0 + id / (D / 8);
            if (row < N) st8<T>(dQ + (size_t)row * D + (id % (D / 8)) * 8, zero8<T>());
        }
        return;
    }

    const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + qbase;
    const T* __restrict__ dO = reinterpret_cast<const T*>(p.dO) + qbase;
    const __amdgpu_buffer_rsrc_t rk = slice_rsrc<T, D>(reinterpret_cast<const T*>(p.k) + kvbase, N);
    const __amdgpu_buffer_rsrc_t rv = slice_rsrc<T, D>(reinterpret_cast<const T*>(p.v) + kvbase, N);
    typedef typename Vec<T>::x8 frag;
    frag qf[D / 16], gf[D / 16];
#pragma unroll
    for (int dc = 0; dc < D / 16; ++dc) {
        qf[dc] = L.qq < N ? ld8<T>(Q + (size_t)L.qq * D + 16 * dc + 8 * L.hf) : zero8<T>();
        gf[dc] = L.qq < N ? ld8<T>(dO + (size_t)L.qq * D + 16 * dc + 8 * L.hf) : zero8<T>();
    }
    const size_t row_base = ((size_t)b * p.Hq + h) * N;
    const float lse2 = L.qq < N ? p.lse[row_base + L.qq] * LOG2E : INFINITY;
    // D_i = sum_c dO * O of this lane's query, from the dO fragments already
    // in registers and O's matching columns; written for the key-block pass,
    // which runs after this one.
    float dsum;
    {
        const T* __restrict__ Orow = reinterpret_cast<const T*>(p.o) + qbase + (size_t)L.qq * D;
        float part = 0.0f;
        if (L.qq < N) {
#pragma unroll
            for (int dc = 0; dc < D / 16; ++dc) part = dot8(ld8<T>(Orow + 16 * dc + 8 * L.hf), gf[dc], part);
        }
        dsum = pair_sum(part);
        if (L.qq < N && L.hf == 0) p.dsum[row_base + L.qq] = dsum;
    }

    f32x16 dq[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) dq[db][v] = 0.0f;

    const int n_tiles = (min(L.m0 + GDQ_BM, N) + GDQ_BN - 1) / GDQ_BN;
    const int n_full = L.m0 / GDQ_BN;
    const int n_mask = n_tiles - n_full;
    const int P = (n_mask + 1) & ~1;
    run_slots(
        P, P + n_full, [&](int i) { return i < P ? (i < n_mask ? n_full + i : -1) : i - P; },
        [&](auto buf, int t) {
            constexpr int B_ = decltype(buf)::value;
            tile_load_lds<T, D>(B_ ? k1s : k0s, rk, t * GDQ_BN, L.w, L.lane);
            tile_load_lds<T, D>(B_ ? v1s : v0s, rv, t * GDQ_BN, L.w, L.lane);
        },
        [&](auto) {},
        [&](auto buf, int t, auto mask) {
            constexpr int B_ = decltype(buf)::value;
            gdq_tile<T, D, decltype(mask)::value>(B_ ? k1s : k0s, B_ ? v1s : v0s, t * GDQ_BN, L, qf, gf, lse2, dsum,
                                                  dq, p.scale_log2);
        });

    if (L.qq < N) {
        T* row = dQ + (size_t)L.qq * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                st4<T>(row + 32 * db + 8 * g + 4 * L.hf, dq[db][4 * g] * p.scale, dq[db][4 * g + 1] * p.scale,
                       dq[db][4 * g + 2] * p.scale, dq[db][4 * g + 3] * p.scale);
    }
}

}  // namespace saf
