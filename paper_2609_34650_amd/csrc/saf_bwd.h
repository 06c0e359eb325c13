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
// the forward's LSE, dP = dO V^T, D_i = rowsum(dO * O)_i (row pre-pass),
// dS = P * (dP - D), dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d).
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
// streaming query tiles of 64 from the block's first key to N.  KV_KB 32-key
// sub-blocks per wavefront: with one, a wavefront stays under 256 VGPRs and
// two of them share a SIMD.
//
// Ordinary heads: scores are formed as S (queries x keys), so a lane holds one
// key (l % 32) and 16 queries of each 32-query half: P and dS feed directly
// into the B operand of dV^T += dO^T P and dK^T += Q^T dS, whose accumulators
// again hold one key per lane.  K and V of the wavefront's keys stay in
// registers; Q and dO tiles are staged in LDS twice, row-major (A operand of S
// and dP) and transposed (A operand of the dV/dK products), in a double buffer
// filled from registers loaded one tile ahead.  The first four tiles meet the
// diagonal and run a masked body; the rest run mask-free.
//
// Fixed heads: dV[j] = sum_i P(i,j) dO[i] with P(i,j) = ea(j) er(i-j) g(i),
// ea = exp(a - A), er = exp(r - R), g(i) = exp(A + R - log Z(i)) (A: maximum
// of a over the block's keys, R: maximum of r over the offsets it meets, log Z
// from the forward's LSE).  The dO tile is staged scaled by g(i), the weight
// operand is the Toeplitz band er(i-j) read from LDS (8 shifted copies, so any
// lane's eight consecutive offsets are one aligned 16-byte read; negative
// offsets hold 0, the causal mask), and the accumulator is scaled by ea(j) at
// the end: no exponential per element.  The band is kept as a bf16 high part
// plus a bf16 low part (er - hi), two products per chunk, so each term is
// rounded once (in g * dO), as in the exact program.  If some row's log Z lies more than
// FAST_GUARD below A + R (g could overflow), the block runs the exact
// per-element program instead.  dK of a fixed head is written as zeros.
// ---------------------------------------------------------------------------
constexpr int KV_KB = 1;                 // 32-key sub-blocks per wavefront
constexpr int KV_BN = 4 * 32 * KV_KB;    // keys per workgroup
constexpr int KV_BM = 64;                // queries per tile
constexpr int KV_THREADS = 256;
constexpr int KV_PAD = 8;
constexpr int KV_MASK_TILES = KV_BN / KV_BM;  // tiles that meet the diagonal
constexpr int KV_BAND = KV_BM + KV_BN - 1;    // offsets per tile
constexpr int KV_BAND_STRIDE = (KV_BAND + 8) / 8 * 8 + 8;  // every copy 16-byte aligned

template <typename T>
struct KvOrdSmem {
    T q[2][KV_BM][HEAD_DIM + KV_PAD];
    T dO[2][KV_BM][HEAD_DIM + KV_PAD];
    T qt[2][HEAD_DIM][KV_BM + KV_PAD];    // [d][tpos(query)]
    T dOt[2][HEAD_DIM][KV_BM + KV_PAD];
    float lse[2][KV_BM];                  // LSE * log2(e); +inf past N
    float dsum[2][KV_BM];                 // D; 0 past N
};

template <typename T>
struct KvFixSmem {
    T dogt[2][HEAD_DIM][KV_BM + KV_PAD];          // (g * dO) transposed, [d][query]
    T band[2][2][BAND_COPIES][KV_BAND_STRIDE];    // [buf][hi, lo] er(delta_lo + x + s) in copy s
    float red[4];
};

template <typename T>
struct KvExactSmem {
    T dOt[HEAD_DIM][KV_BM + KV_PAD];  // [d][tpos(query)]
    float lse[KV_BM];
    float rb[KV_BAND + 1];            // r(delta_lo + x), -inf outside [0, N)
};

template <typename T>
constexpr size_t kv_smem_bytes() {
    size_t x = sizeof(KvOrdSmem<T>);
    if (sizeof(KvFixSmem<T>) > x) x = sizeof(KvFixSmem<T>);
    if (sizeof(KvExactSmem<T>) > x) x = sizeof(KvExactSmem<T>);
    return x;
}

struct KvLane {
    int tid, w, c, hf, n0, kw, N;
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

template <typename T>
struct KvStage {
    typename Vec<T>::x8 q[2], g[2];
    float lse, dsum;
};

template <typename T>
__device__ __forceinline__ void kv_load(KvStage<T>& st, const T* Q, const T* dO, const float* LSE, const float* Dsum,
                                        int mq, int N, int tid) {
    const int r2 = (tid >> 3) * 2;
    const int d8 = (tid & 7) * 8;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const bool ok = mq + r2 + k < N;
        st.q[k] = ok ? ld8<T>(Q + (size_t)(mq + r2 + k) * HEAD_DIM + d8) : zero8<T>();
        st.g[k] = ok ? ld8<T>(dO + (size_t)(mq + r2 + k) * HEAD_DIM + d8) : zero8<T>();
    }
    if (tid < KV_BM) {
        const bool ok = mq + tid < N;
        st.lse = ok ? LSE[mq + tid] * LOG2E : INFINITY;
        st.dsum = ok ? Dsum[mq + tid] : 0.0f;
    }
}

template <typename T>
__device__ __forceinline__ void kv_store(KvOrdSmem<T>& sm, int buf, const KvStage<T>& st, int tid) {
    const int r2 = (tid >> 3) * 2;
    const int d8 = (tid & 7) * 8;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        st8<T>(&sm.q[buf][r2 + k][d8], st.q[k]);
        st8<T>(&sm.dO[buf][r2 + k][d8], st.g[k]);
    }
    st_pair_t(&sm.qt[buf][d8][tpos(r2)], KV_BM + KV_PAD, st.q[0], st.q[1]);
    st_pair_t(&sm.dOt[buf][d8][tpos(r2)], KV_BM + KV_PAD, st.g[0], st.g[1]);
    if (tid < KV_BM) {
        sm.lse[buf][tid] = st.lse;
        sm.dsum[buf][tid] = st.dsum;
    }
}

template <typename T, bool MASK>
__device__ __forceinline__ void kv_tile(const KvOrdSmem<T>& sm, int buf, int mq, const KvLane& L,
                                        const typename Vec<T>::x8 (&kf)[KV_KB][4], const typename Vec<T>::x8 (&vf)[KV_KB][4],
                                        f32x16 (&dv)[KV_KB][2], f32x16 (&dk)[KV_KB][2], float scale_log2) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qs = mq + 32 * qb;
        if (MASK && (qs + 31 < L.kw || qs >= L.N)) continue;  // no query of this half sees these keys
        f32x16 s[KV_KB], dp[KV_KB];
        {
            frag qa[4];
#pragma unroll
            for (int dc = 0; dc < 4; ++dc) qa[dc] = ld8<T>(&sm.q[buf][32 * qb + L.c][16 * dc + 8 * L.hf]);
#pragma unroll
            for (int kb = 0; kb < KV_KB; ++kb) {
#pragma unroll
                for (int v = 0; v < 16; ++v) s[kb][v] = 0.0f;
#pragma unroll
                for (int dc = 0; dc < 4; ++dc) mma(s[kb], qa[dc], kf[kb][dc]);
            }
        }
        {
            frag ga[4];
#pragma unroll
            for (int dc = 0; dc < 4; ++dc) ga[dc] = ld8<T>(&sm.dO[buf][32 * qb + L.c][16 * dc + 8 * L.hf]);
#pragma unroll
            for (int kb = 0; kb < KV_KB; ++kb) {
#pragma unroll
                for (int v = 0; v < 16; ++v) dp[kb][v] = 0.0f;
#pragma unroll
                for (int dc = 0; dc < 4; ++dc) mma(dp[kb], ga[dc], vf[kb][dc]);
            }
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sm.lse[buf][32 * qb + 8 * g + 4 * L.hf]);
            const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sm.dsum[buf][32 * qb + 8 * g + 4 * L.hf]);
#pragma unroll
            for (int kb = 0; kb < KV_KB; ++kb)
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int v = 4 * g + u;
                    float pv = fast_exp2(fmaf(s[kb][v], scale_log2, -l4[u]));
                    if (MASK) {
                        const int row = qs + 8 * g + 4 * L.hf + u;
                        if (row < L.kw + 32 * kb + L.c) pv = 0.0f;
                    }
                    s[kb][v] = pv;
                    dp[kb][v] = pv * (dp[kb][v] - d4[u]);
                }
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const int col = 32 * qb + 16 * kc + 8 * L.hf;
            frag gt[2], qt[2];
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                gt[db] = ld8<T>(&sm.dOt[buf][32 * db + L.c][col]);
                qt[db] = ld8<T>(&sm.qt[buf][32 * db + L.c][col]);
            }
#pragma unroll
            for (int kb = 0; kb < KV_KB; ++kb) {
                const frag pb = to_operand<T>(s[kb], 8 * kc);
                const frag sb = to_operand<T>(dp[kb], 8 * kc);
#pragma unroll
                for (int db = 0; db < 2; ++db) {
                    mma(dv[kb][db], gt[db], pb);
                    mma(dk[kb][db], qt[db], sb);
                }
            }
        }
    }
}

template <typename T>
__device__ void kv_ordinary(void* smem, const BwdArgs& p, const KvLane& L, size_t base, size_t row_base) {
    KvOrdSmem<T>& sm = *reinterpret_cast<KvOrdSmem<T>*>(smem);
    const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + base;
    const T* __restrict__ K = reinterpret_cast<const T*>(p.k) + base;
    const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + base;
    const T* __restrict__ dO = reinterpret_cast<const T*>(p.dO) + base;
    const float* __restrict__ LSE = p.lse + row_base;
    const float* __restrict__ Dsum = p.dsum + row_base;
    typedef typename Vec<T>::x8 frag;
    frag kf[KV_KB][4], vf[KV_KB][4];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) {
        const int key = L.kw + 32 * kb + L.c;
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) {
            kf[kb][dc] = key < L.N ? ld8<T>(K + (size_t)key * HEAD_DIM + 16 * dc + 8 * L.hf) : zero8<T>();
            vf[kb][dc] = key < L.N ? ld8<T>(V + (size_t)key * HEAD_DIM + 16 * dc + 8 * L.hf) : zero8<T>();
        }
    }
    f32x16 dv[KV_KB][2], dk[KV_KB][2];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb)
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                dv[kb][db][v] = 0.0f;
                dk[kb][db][v] = 0.0f;
            }

    const int n_tiles = (L.N - L.n0 + KV_BM - 1) / KV_BM;
    KvStage<T> st;
    kv_load<T>(st, Q, dO, LSE, Dsum, L.n0, L.N, L.tid);
    kv_store<T>(sm, 0, st, L.tid);
    __syncthreads();
    for (int t = 0; t < n_tiles; ++t) {
        const bool more = t + 1 < n_tiles;
        const int mq = L.n0 + t * KV_BM;
        if (more) kv_load<T>(st, Q, dO, LSE, Dsum, mq + KV_BM, L.N, L.tid);
        if (t < KV_MASK_TILES)
            kv_tile<T, true>(sm, t & 1, mq, L, kf, vf, dv, dk, p.scale_log2);
        else
            kv_tile<T, false>(sm, t & 1, mq, L, kf, vf, dv, dk, p.scale_log2);
        if (more) kv_store<T>(sm, (t + 1) & 1, st, L.tid);
        __syncthreads();
    }
    float one[KV_KB], ks[KV_KB];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) {
        one[kb] = 1.0f;
        ks[kb] = p.scale;
    }
    kv_store_rows<T>(reinterpret_cast<T*>(p.dv) + base, L, dv, one);
    kv_store_rows<T>(reinterpret_cast<T*>(p.dk) + base, L, dk, ks);
}

// --- fixed heads: exact per-element program (fallback) ----------------------

template <typename T>
__device__ void kv_fixed_exact(void* smem, const BwdArgs& p, const KvLane& L, size_t base, size_t row_base,
                               const float* arow, const float* rrow) {
    KvExactSmem<T>& sm = *reinterpret_cast<KvExactSmem<T>*>(smem);
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
    for (int mq = L.n0; mq < N; mq += KV_BM) {
        __syncthreads();
        {
            const int r2 = (L.tid >> 3) * 2;
            const int d8 = (L.tid & 7) * 8;
            const frag g0 = mq + r2 < N ? ld8<T>(dO + (size_t)(mq + r2) * HEAD_DIM + d8) : zero8<T>();
            const frag g1 = mq + r2 + 1 < N ? ld8<T>(dO + (size_t)(mq + r2 + 1) * HEAD_DIM + d8) : zero8<T>();
            st_pair_t(&sm.dOt[d8][tpos(r2)], KV_BM + KV_PAD, g0, g1);
        }
        if (L.tid < KV_BM) sm.lse[L.tid] = mq + L.tid < N ? LSE[mq + L.tid] * LOG2E : INFINITY;
        for (int x = L.tid; x < KV_BAND; x += KV_THREADS) {
            const int delta = mq - L.n0 - (KV_BN - 1) + x;
            sm.rb[x] = (delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
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
                    pm[kb][v] = fast_exp2(fmaf(a_key[kb] + sm.rb[x], LOG2E, -sm.lse[ql]));
                }
            }
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const int col = 32 * qb + 16 * kc + 8 * L.hf;
                frag gt[2];
#pragma unroll
                for (int db = 0; db < 2; ++db) gt[db] = ld8<T>(&sm.dOt[32 * db + L.c][col]);
#pragma unroll
                for (int kb = 0; kb < KV_KB; ++kb) {
                    const frag pb = to_operand<T>(pm[kb], 8 * kc);
#pragma unroll
                    for (int db = 0; db < 2; ++db) mma(dv[kb][db], gt[db], pb);
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

template <typename T>
struct KvFixStage {
    typename Vec<T>::x8 g[2];
    float lse[2];
    float rb[2];
};

template <typename T>
__device__ __forceinline__ void kvf_load(KvFixStage<T>& st, const T* dO, const float* LSE, const float* rrow, int mq,
                                         int n0, int N, int tid) {
    const int r2 = (tid >> 3) * 2;
    const int d8 = (tid & 7) * 8;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const bool ok = mq + r2 + k < N;
        st.g[k] = ok ? ld8<T>(dO + (size_t)(mq + r2 + k) * HEAD_DIM + d8) : zero8<T>();
        st.lse[k] = ok ? LSE[mq + r2 + k] : INFINITY;
        const int x = tid + KV_THREADS * k;
        const int delta = mq - n0 - (KV_BN - 1) + x;
        st.rb[k] = (x < KV_BAND && delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
    }
}

template <typename T>
__device__ __forceinline__ void kvf_store(KvFixSmem<T>& sm, int buf, const KvFixStage<T>& st, int tid, float g_sh,
                                          float r_sh) {
    const int r2 = (tid >> 3) * 2;
    const int d8 = (tid & 7) * 8;
    const float g0 = fast_exp2(fmaf(-st.lse[0], LOG2E, g_sh));
    const float g1 = fast_exp2(fmaf(-st.lse[1], LOG2E, g_sh));
    st_pair_t_scaled(&sm.dogt[buf][d8][r2], KV_BM + KV_PAD, st.g[0], st.g[1], g0, g1);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int x = tid + KV_THREADS * k;
        if (x < KV_BAND) {
            const float e = fast_exp2(fmaf(st.rb[k], LOG2E, -r_sh));
            const T hi = (T)e;
            const T lo = (T)(e - (float)hi);
#pragma unroll
            for (int s = 0; s < BAND_COPIES; ++s)
                if (x >= s) {
                    sm.band[buf][0][s][x - s] = hi;
                    sm.band[buf][1][s][x - s] = lo;
                }
        }
    }
}

template <typename T, bool MASK>
__device__ __forceinline__ void kvf_tile(const KvFixSmem<T>& sm, int buf, int mq, const KvLane& L,
                                         f32x16 (&dv)[KV_KB][2]) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qs = mq + 32 * qb;
        if (MASK && (qs + 31 < L.kw || qs >= L.N)) continue;
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const int col = 32 * qb + 16 * kc + 8 * L.hf;  // first query (within the tile) of this lane's slots
            frag gt[2];
#pragma unroll
            for (int db = 0; db < 2; ++db) gt[db] = ld8<T>(&sm.dogt[buf][32 * db + L.c][col]);
#pragma unroll
            for (int kb = 0; kb < KV_KB; ++kb) {
                const int kl = L.kw - L.n0 + 32 * kb + L.c;
                const int u0 = col - kl + (KV_BN - 1);  // band index of offset (mq + col) - (n0 + kl)
                const int s = u0 & 7;
                const frag bh = ld8<T>(&sm.band[buf][0][s][u0 - s]);
                const frag bl = ld8<T>(&sm.band[buf][1][s][u0 - s]);
#pragma unroll
                for (int db = 0; db < 2; ++db) {
                    mma(dv[kb][db], gt[db], bh);
                    mma(dv[kb][db], gt[db], bl);
                }
            }
        }
    }
}

template <typename T>
__device__ void kv_fixed(void* smem, const BwdArgs& p, const KvLane& L, size_t base, size_t row_base, int h) {
    KvFixSmem<T>& sm = *reinterpret_cast<KvFixSmem<T>*>(smem);
    const T* __restrict__ dO = reinterpret_cast<const T*>(p.dO) + base;
    const float* __restrict__ LSE = p.lse + row_base;
    const float* __restrict__ arow = p.a + (size_t)h * p.ld_prior;
    const float* __restrict__ rrow = p.r + (size_t)h * p.ld_prior;
    const int N = L.N;

    // A: max of a over the block's keys; R: max of r over the offsets the
    // block meets (0 .. N - 1 - n0); lo: min of log Z over its rows.
    float am = L.n0 + L.tid < N ? arow[L.n0 + L.tid] : -INFINITY;
    float rm = -INFINITY, lo = INFINITY;
    for (int j = L.tid; j < N - L.n0; j += KV_THREADS) {
        rm = fmaxf(rm, rrow[j]);
        lo = fminf(lo, LSE[L.n0 + j]);
    }
    const float A = block_max(am, sm.red);
    const float R = block_max(rm, sm.red);
    const float LO = -block_max(-lo, sm.red);
    if (!(LO - A - R >= -FAST_GUARD)) {  // some g(i) could overflow
        kv_fixed_exact<T>(smem, p, L, base, row_base, arow, rrow);
        return;
    }
    const float g_sh = (A + R) * LOG2E, r_sh = R * LOG2E, a_sh = A * LOG2E;

    f32x16 dv[KV_KB][2];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb)
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) dv[kb][db][v] = 0.0f;

    const int n_tiles = (N - L.n0 + KV_BM - 1) / KV_BM;
    KvFixStage<T> st;
    kvf_load<T>(st, dO, LSE, rrow, L.n0, L.n0, N, L.tid);
    kvf_store<T>(sm, 0, st, L.tid, g_sh, r_sh);
    __syncthreads();
    for (int t = 0; t < n_tiles; ++t) {
        const bool more = t + 1 < n_tiles;
        const int mq = L.n0 + t * KV_BM;
        if (more) kvf_load<T>(st, dO, LSE, rrow, mq + KV_BM, L.n0, N, L.tid);
        if (t < KV_MASK_TILES)
            kvf_tile<T, true>(sm, t & 1, mq, L, dv);
        else
            kvf_tile<T, false>(sm, t & 1, mq, L, dv);
        if (more) kvf_store<T>(sm, (t + 1) & 1, st, L.tid, g_sh, r_sh);
        __syncthreads();
    }
    float ea[KV_KB];
#pragma unroll
    for (int kb = 0; kb < KV_KB; ++kb) {
        const int key = L.kw + 32 * kb + L.c;
        ea[kb] = key < N ? fast_exp2(fmaf(arow[key], LOG2E, -a_sh)) : 0.0f;
    }
    kv_store_rows<T>(reinterpret_cast<T*>(p.dv) + base, L, dv, ea);
    kv_store_zero<T>(reinterpret_cast<T*>(p.dk) + base, L);
}

template <typename T>
__global__ __launch_bounds__(KV_THREADS) void bwd_kv_kernel(BwdArgs p) {
    __shared__ __attribute__((aligned(16))) char smem[kv_smem_bytes<T>()];
    const int n_bh = p.B * p.H;
    const int kblk = (int)(blockIdx.x / n_bh);  // ascending: longest first
    const int bh = (int)(blockIdx.x % n_bh);
    const int h = bh % p.H;
    KvLane L;
    L.tid = threadIdx.x;
    L.w = L.tid >> 6;
    L.c = L.tid & 31;
    L.hf = (L.tid >> 5) & 1;
    L.n0 = kblk * KV_BN;
    L.kw = L.n0 + 32 * KV_KB * L.w;
    L.N = p.N;
    const size_t base = (size_t)bh * p.N * HEAD_DIM;
    const size_t row_base = (size_t)bh * p.N;
    if ((p.fixed_mask >> h) & 1ull)
        kv_fixed<T>(smem, p, L, base, row_base, h);
    else
        kv_ordinary<T>(smem, p, L, base, row_base);
}

// ---------------------------------------------------------------------------
// Query-block pass (ordinary heads): workgroup = (b, h, 128 queries); 4
// wavefronts x 32 queries, streaming key tiles of 64 up to the diagonal.
// S^T (keys x queries) puts one query per lane, so LSE and D are per-lane
// scalars and dS^T feeds the B operand of dQ^T += K^T dS^T.  Workgroups of
// fixed heads only write zeros.
// ---------------------------------------------------------------------------
constexpr int DQ_BM = 128;
constexpr int DQ_BN = 64;
constexpr int DQ_THREADS = 256;
constexpr int DQ_PAD = 8;

template <typename T>
struct DqSmem {
    T k[DQ_BN][HEAD_DIM + DQ_PAD];
    T v[DQ_BN][HEAD_DIM + DQ_PAD];
    T kt[HEAD_DIM][DQ_BN + DQ_PAD];
};

template <typename T>
__global__ __launch_bounds__(DQ_THREADS) void bwd_dq_kernel(BwdArgs p) {
    __shared__ DqSmem<T> sm;

    const int n_bh = p.B * p.H;
    const int qblk = p.n_blocks - 1 - (int)(blockIdx.x / n_bh);  // longest first
    const int bh = (int)(blockIdx.x % n_bh);
    const int h = bh % p.H;
    const bool fixed = (p.fixed_mask >> h) & 1ull;
    const int N = p.N;
    const size_t base = (size_t)bh * N * HEAD_DIM;
    T* __restrict__ dQ = reinterpret_cast<T*>(p.dq) + base;

    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int lane = tid & 63;
    const int c = lane & 31;
    const int hf = lane >> 5;
    const int m0 = qblk * DQ_BM;
    const int q0 = m0 + 32 * w;
    const int qq = q0 + c;

    if (fixed) {  // the whole workgroup takes this branch
        for (int id = tid; id < DQ_BM * (HEAD_DIM / 8); id += DQ_THREADS) {
            const int row = m0 + id / (HEAD_DIM / 8);
            if (row < N) st8<T>(dQ + (size_t)row * HEAD_DIM + (id % (HEAD_DIM / 8)) * 8, zero8<T>());
        }
        return;
    }

    const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + base;
    const T* __restrict__ K = reinterpret_cast<const T*>(p.k) + base;
    const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + base;
    const T* __restrict__ dO = reinterpret_cast<const T*>(p.dO) + base;

    typedef typename Vec<T>::x8 frag;
    frag qf[4], gf[4];
#pragma unroll
    for (int dc = 0; dc < 4; ++dc) {
        qf[dc] = qq < N ? ld8<T>(Q + (size_t)qq * HEAD_DIM + 16 * dc + 8 * hf) : zero8<T>();
        gf[dc] = qq < N ? ld8<T>(dO + (size_t)qq * HEAD_DIM + 16 * dc + 8 * hf) : zero8<T>();
    }
    const float lse2 = qq < N ? p.lse[(size_t)bh * N + qq] * LOG2E : INFINITY;
    const float dq_row = qq < N ? p.dsum[(size_t)bh * N + qq] : 0.0f;

    f32x16 dq[2];
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) dq[db][v] = 0.0f;

    const int n_end = min(m0 + DQ_BM, N);
    for (int n0 = 0; n0 < n_end; n0 += DQ_BN) {
        __syncthreads();
        {
            const int k2 = (tid >> 3) * 2;
            const int d8 = (tid & 7) * 8;
            const bool v0 = n0 + k2 < N, v1 = n0 + k2 + 1 < N;
            frag x0 = v0 ? ld8<T>(K + (size_t)(n0 + k2) * HEAD_DIM + d8) : zero8<T>();
            frag x1 = v1 ? ld8<T>(K + (size_t)(n0 + k2 + 1) * HEAD_DIM + d8) : zero8<T>();
            st8<T>(&sm.k[k2][d8], x0);
            st8<T>(&sm.k[k2 + 1][d8], x1);
            const int pos = tpos(k2);
#pragma unroll
            for (int t = 0; t < 8; ++t) st2<T>(&sm.kt[d8 + t][pos], x0[t], x1[t]);
            frag y0 = v0 ? ld8<T>(V + (size_t)(n0 + k2) * HEAD_DIM + d8) : zero8<T>();
            frag y1 = v1 ? ld8<T>(V + (size_t)(n0 + k2 + 1) * HEAD_DIM + d8) : zero8<T>();
            st8<T>(&sm.v[k2][d8], y0);
            st8<T>(&sm.v[k2 + 1][d8], y1);
        }
        __syncthreads();

        bool act[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int k0 = n0 + 32 * kb;
            act[kb] = (k0 < q0 + 32) && (k0 < N);
        }
        if (!act[0]) continue;

#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            if (!act[kb]) continue;
            const int k0 = n0 + 32 * kb;
            f32x16 s, dp;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                s[v] = 0.0f;
                dp[v] = 0.0f;
            }
#pragma unroll
            for (int dc = 0; dc < 4; ++dc) {
                mma(s, ld8<T>(&sm.k[32 * kb + c][16 * dc + 8 * hf]), qf[dc]);
                mma(dp, ld8<T>(&sm.v[32 * kb + c][16 * dc + 8 * hf]), gf[dc]);
            }
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                float pv = fast_exp2(s[v] * p.scale_log2 - lse2);
                if (k0 == q0) {
                    const int kidx = k0 + 8 * (v >> 2) + 4 * hf + (v & 3);
                    if (kidx > qq) pv = 0.0f;
                }
                s[v] = pv * (dp[v] - dq_row);  // dS^T
            }
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const frag sb = to_operand<T>(s, 8 * kc);
#pragma unroll
                for (int db = 0; db < 2; ++db)
                    mma(dq[db], ld8<T>(&sm.kt[32 * db + c][32 * kb + 16 * kc + 8 * hf]), sb);
            }
        }
    }

    if (qq < N) {
        T* row = dQ + (size_t)qq * HEAD_DIM;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                st4<T>(row + 32 * db + 8 * g + 4 * hf, dq[db][4 * g] * p.scale, dq[db][4 * g + 1] * p.scale,
                       dq[db][4 * g + 2] * p.scale, dq[db][4 * g + 3] * p.scale);
    }
}

}  // namespace saf
