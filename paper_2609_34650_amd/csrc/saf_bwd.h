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
// Key-block pass: workgroup = (b, h, 128 keys); 4 wavefronts x 32 keys each,
// streaming query tiles of 64 from the block's first key to N.
//
// Scores are formed as S (queries x keys), so a lane holds one key (l % 32)
// and 16 queries of each 32-query half: P and dS feed directly into the B
// operand of dV^T += dO^T P and dK^T += Q^T dS, whose accumulators again hold
// one key per lane.  K and V of the wavefront's keys stay in registers; Q and
// dO tiles are staged in LDS twice, row-major (A operand of S and dP) and
// transposed (A operand of the dV/dK products).
// ---------------------------------------------------------------------------
constexpr int KV_BN = 128;  // keys per workgroup
constexpr int KV_BM = 64;   // queries per tile
constexpr int KV_THREADS = 256;
constexpr int KV_PAD = 8;

template <typename T>
struct KvSmem {
    T q[KV_BM][HEAD_DIM + KV_PAD];
    T dO[KV_BM][HEAD_DIM + KV_PAD];
    T qt[HEAD_DIM][KV_BM + KV_PAD];
    T dOt[HEAD_DIM][KV_BM + KV_PAD];
    float lse[KV_BM];            // LSE * log2(e); +inf past N
    float dsum[KV_BM];           // D; 0 past N
    float rb[KV_BM + KV_BN];     // fixed head: r over the tile's offsets
};

template <typename T>
__global__ __launch_bounds__(KV_THREADS) void bwd_kv_kernel(BwdArgs p) {
    __shared__ KvSmem<T> sm;

    const int n_bh = p.B * p.H;
    const int kblk = (int)(blockIdx.x / n_bh);  // ascending: longest first
    const int bh = (int)(blockIdx.x % n_bh);
    const int h = bh % p.H;
    const bool fixed = (p.fixed_mask >> h) & 1ull;
    const int N = p.N;
    const size_t base = (size_t)bh * N * HEAD_DIM;
    const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + base;
    const T* __restrict__ K = reinterpret_cast<const T*>(p.k) + base;
    const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + base;
    const T* __restrict__ dO = reinterpret_cast<const T*>(p.dO) + base;
    T* __restrict__ dK = reinterpret_cast<T*>(p.dk) + base;
    T* __restrict__ dV = reinterpret_cast<T*>(p.dv) + base;
    const float* __restrict__ LSE = p.lse + (size_t)bh * N;
    const float* __restrict__ Dsum = p.dsum + (size_t)bh * N;
    const float* __restrict__ rrow = fixed ? p.r + (size_t)h * p.ld_prior : nullptr;

    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int lane = tid & 63;
    const int c = lane & 31;
    const int hf = lane >> 5;
    const int n0 = kblk * KV_BN;
    const int k0w = n0 + 32 * w;  // first key of this wavefront
    const int kk = k0w + c;       // this lane's key

    typedef typename Vec<T>::x8 frag;
    frag kf[4], vf[4];
    float a_key = 0.0f;
    if (!fixed) {
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) {
            kf[dc] = kk < N ? ld8<T>(K + (size_t)kk * HEAD_DIM + 16 * dc + 8 * hf) : zero8<T>();
            vf[dc] = kk < N ? ld8<T>(V + (size_t)kk * HEAD_DIM + 16 * dc + 8 * hf) : zero8<T>();
        }
    } else {
        a_key = kk < N ? p.a[(size_t)h * p.ld_prior + kk] : -INFINITY;
    }

    f32x16 dv[2], dk[2];
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            dv[db][v] = 0.0f;
            dk[db][v] = 0.0f;
        }

    for (int mq = n0; mq < N; mq += KV_BM) {
        __syncthreads();
        {
            const int r2 = (tid >> 3) * 2;  // query rows (r2, r2 + 1) of the tile
            const int d8 = (tid & 7) * 8;
            const int pos = tpos(r2);
            const bool v0 = mq + r2 < N, v1 = mq + r2 + 1 < N;
            if (!fixed) {
                frag x0 = v0 ? ld8<T>(Q + (size_t)(mq + r2) * HEAD_DIM + d8) : zero8<T>();
                frag x1 = v1 ? ld8<T>(Q + (size_t)(mq + r2 + 1) * HEAD_DIM + d8) : zero8<T>();
                st8<T>(&sm.q[r2][d8], x0);
                st8<T>(&sm.q[r2 + 1][d8], x1);
#pragma unroll
                for (int t = 0; t < 8; ++t) st2<T>(&sm.qt[d8 + t][pos], x0[t], x1[t]);
            }
            frag g0 = v0 ? ld8<T>(dO + (size_t)(mq + r2) * HEAD_DIM + d8) : zero8<T>();
            frag g1 = v1 ? ld8<T>(dO + (size_t)(mq + r2 + 1) * HEAD_DIM + d8) : zero8<T>();
            if (!fixed) {
                st8<T>(&sm.dO[r2][d8], g0);
                st8<T>(&sm.dO[r2 + 1][d8], g1);
            }
#pragma unroll
            for (int t = 0; t < 8; ++t) st2<T>(&sm.dOt[d8 + t][pos], g0[t], g1[t]);
        }
        if (tid < KV_BM) {
            const int qi = mq + tid;
            sm.lse[tid] = qi < N ? LSE[qi] * LOG2E : INFINITY;
            sm.dsum[tid] = (!fixed && qi < N) ? Dsum[qi] : 0.0f;
        }
        if (fixed) {
            // Offsets i - j over the tile: mq - n0 - 127 .. mq - n0 + 63.
            for (int x = tid; x < KV_BM + KV_BN - 1; x += KV_THREADS) {
                const int delta = mq - n0 - (KV_BN - 1) + x;
                sm.rb[x] = (delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
            }
        }
        __syncthreads();

        // 32-query halves of the tile that hold a query >= some key of this
        // wavefront (both start at multiples of 32).
        bool act[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            const int qs = mq + 32 * qb;
            act[qb] = (qs >= k0w) && (qs < N);
        }
        if (!act[0] && !act[1]) continue;

        f32x16 pm[2], dsm[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            if (!act[qb]) continue;
            const int qs = mq + 32 * qb;
            if (!fixed) {
#pragma unroll
                for (int v = 0; v < 16; ++v) pm[qb][v] = 0.0f;
#pragma unroll
                for (int dc = 0; dc < 4; ++dc)
                    mma(pm[qb], ld8<T>(&sm.q[32 * qb + c][16 * dc + 8 * hf]), kf[dc]);
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sm.lse[32 * qb + 8 * g + 4 * hf]);
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        pm[qb][4 * g + u] = fast_exp2(pm[qb][4 * g + u] * p.scale_log2 - l4[u]);
                }
            } else {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sm.lse[32 * qb + 8 * g + 4 * hf]);
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int ql = 32 * qb + 8 * g + 4 * hf + u;   // query within tile
                        const int x = ql - (kk - n0) + (KV_BN - 1);    // band index of (mq + ql) - kk
                        pm[qb][4 * g + u] = fast_exp2((a_key + sm.rb[x]) * LOG2E - l4[u]);
                    }
                }
            }
            if (qs == k0w) {  // diagonal: queries before the key see nothing of it
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int qi = qs + 8 * (v >> 2) + 4 * hf + (v & 3);
                    if (qi < kk) pm[qb][v] = 0.0f;
                }
            }
            if (!fixed) {
                f32x16 dp;
#pragma unroll
                for (int v = 0; v < 16; ++v) dp[v] = 0.0f;
#pragma unroll
                for (int dc = 0; dc < 4; ++dc)
                    mma(dp, ld8<T>(&sm.dO[32 * qb + c][16 * dc + 8 * hf]), vf[dc]);
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sm.dsum[32 * qb + 8 * g + 4 * hf]);
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        dsm[qb][4 * g + u] = pm[qb][4 * g + u] * (dp[4 * g + u] - d4[u]);
                }
            }
        }

#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            if (!act[qb]) continue;
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const int col = 32 * qb + 16 * kc + 8 * hf;
                const frag pb = to_operand<T>(pm[qb], 8 * kc);
#pragma unroll
                for (int db = 0; db < 2; ++db) mma(dv[db], ld8<T>(&sm.dOt[32 * db + c][col]), pb);
                if (!fixed) {
                    const frag sb = to_operand<T>(dsm[qb], 8 * kc);
#pragma unroll
                    for (int db = 0; db < 2; ++db) mma(dk[db], ld8<T>(&sm.qt[32 * db + c][col]), sb);
                }
            }
        }
    }

    if (kk < N) {
        T* dvrow = dV + (size_t)kk * HEAD_DIM;
        T* dkrow = dK + (size_t)kk * HEAD_DIM;
        const float ks = fixed ? 0.0f : p.scale;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int col = 32 * db + 8 * g + 4 * hf;
                st4<T>(dvrow + col, dv[db][4 * g], dv[db][4 * g + 1], dv[db][4 * g + 2], dv[db][4 * g + 3]);
                st4<T>(dkrow + col, dk[db][4 * g] * ks, dk[db][4 * g + 1] * ks, dk[db][4 * g + 2] * ks,
                       dk[db][4 * g + 3] * ks);
            }
    }
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
