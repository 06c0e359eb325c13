// Forward of the hybrid causal-attention layer: one launch for all heads.
//
// Workgroup = (batch b, head h, block of 128 queries); 4 wavefronts, each
// owning 32 consecutive queries.  The head's flag picks the path of the whole
// workgroup (Appendix "Mixed-head execution and numerical checks": one
// program per batch element, head and query block, a head-state flag selects
// the computation, outputs keep the original head order).
//
// Both paths stream key tiles of 64 from key 0 up to the block's last query
// (causal tile skipping: tiles wholly in the future of a wavefront's queries
// are skipped by that wavefront) and keep, per query, a running maximum m and
// sum l of the base-2 exponentials plus an unnormalised output, the online
// softmax of FlashAttention-2 that the paper uses for ordinary heads.
//
// Scores are formed transposed, S^T (keys x queries), so that the
// accumulator of lane l holds one query (l % 32) and 16 of its keys: the
// per-query statistics stay in the lane (one cross-half exchange per tile for
// the maximum), the exponentials go straight into the B operand of
// O^T += V^T P^T, and O^T again holds one query per lane.
//
//   ordinary head: S = Q K^T / sqrt(d) (bf16/fp32 MFMA, K tile in LDS,
//                  Q in registers), LSE = log sum_j exp(S_ij)
//   fixed head:    S_ij = a[j] + r[i - j] gathered from LDS copies of a and
//                  of the r band the tile touches (Eq. compact-prior; no
//                  1/sqrt(d), no Q or K reads), LSE = log Z(i)
#pragma once

#include "saf_common.h"

namespace saf {

constexpr int FWD_BM = 128;  // queries per workgroup
constexpr int FWD_BN = 64;   // keys per tile
constexpr int FWD_THREADS = 256;
constexpr int LDS_PAD = 8;   // elements appended to each LDS row

template <typename T>
struct FwdSmem {
    T k[FWD_BN][HEAD_DIM + LDS_PAD];    // K tile, [key][d]
    T vt[HEAD_DIM][FWD_BN + LDS_PAD];   // V tile transposed, [d][tpos(key)]
    float a[FWD_BN];                    // fixed head: a of the tile's keys
    float rb[FWD_BM + FWD_BN];          // fixed head: r over the tile's offsets
};

struct FwdArgs {
    const void* q;
    const void* k;
    const void* v;
    const float* a;
    const float* r;
    void* o;
    float* lse;
    uint64_t fixed_mask;
    int B, H, N, ld_prior, n_qblocks;
    float scale_log2;  // log2(e) / sqrt(d)
};

template <typename T>
__global__ __launch_bounds__(FWD_THREADS) void fwd_kernel(FwdArgs p) {
    __shared__ FwdSmem<T> sm;

    const int n_bh = p.B * p.H;
    // Longest blocks first: block index -> query block in descending order.
    const int qblk = p.n_qblocks - 1 - (int)(blockIdx.x / n_bh);
    const int bh = (int)(blockIdx.x % n_bh);
    const int h = bh % p.H;
    const bool fixed = (p.fixed_mask >> h) & 1ull;
    const int N = p.N;
    const size_t base = (size_t)bh * N * HEAD_DIM;
    const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + base;
    const T* __restrict__ K = reinterpret_cast<const T*>(p.k) + base;
    const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + base;
    T* __restrict__ O = reinterpret_cast<T*>(p.o) + base;
    float* __restrict__ LSE = p.lse + (size_t)bh * N;
    const float* __restrict__ arow = fixed ? p.a + (size_t)h * p.ld_prior : nullptr;
    const float* __restrict__ rrow = fixed ? p.r + (size_t)h * p.ld_prior : nullptr;

    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int lane = tid & 63;
    const int c = lane & 31;
    const int hf = lane >> 5;
    const int m0 = qblk * FWD_BM;
    const int q0 = m0 + 32 * w;  // first query of this wavefront
    const int qq = q0 + c;       // this lane's query

    typedef typename Vec<T>::x8 frag;
    frag qf[4];
    if (!fixed) {
#pragma unroll
        for (int dc = 0; dc < 4; ++dc)
            qf[dc] = qq < N ? ld8<T>(Q + (size_t)qq * HEAD_DIM + 16 * dc + 8 * hf) : zero8<T>();
    }

    f32x16 oacc[2];
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[db][v] = 0.0f;
    float m_run = NEG_BIG;
    float l_run = 0.0f;  // this lane's share of the row sum

    const int n_end = min(m0 + FWD_BM, N);
    for (int n0 = 0; n0 < n_end; n0 += FWD_BN) {
        __syncthreads();
        if (!fixed) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int id = tid + FWD_THREADS * i;
                const int row = id >> 3;
                const int col = (id & 7) * 8;
                frag x = (n0 + row < N) ? ld8<T>(K + (size_t)(n0 + row) * HEAD_DIM + col) : zero8<T>();
                st8<T>(&sm.k[row][col], x);
            }
        }
        {
            const int k2 = (tid >> 3) * 2;  // key pair (k2, k2 + 1)
            const int d8 = (tid & 7) * 8;
            frag x0 = (n0 + k2 < N) ? ld8<T>(V + (size_t)(n0 + k2) * HEAD_DIM + d8) : zero8<T>();
            frag x1 = (n0 + k2 + 1 < N) ? ld8<T>(V + (size_t)(n0 + k2 + 1) * HEAD_DIM + d8) : zero8<T>();
            const int pos = tpos(k2);
#pragma unroll
            for (int t = 0; t < 8; ++t) st2<T>(&sm.vt[d8 + t][pos], x0[t], x1[t]);
        }
        if (fixed) {
            if (tid < FWD_BN) sm.a[tid] = (n0 + tid < N) ? arow[n0 + tid] : -INFINITY;
            // Offsets i - j over the tile: m0 - n0 - 63 .. m0 - n0 + 127.
            for (int x = tid; x < FWD_BM + FWD_BN - 1; x += FWD_THREADS) {
                const int delta = m0 - n0 - (FWD_BN - 1) + x;
                sm.rb[x] = (delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
            }
        }
        __syncthreads();

        // 32-key sub-blocks of this tile that hold a key <= some query of
        // this wavefront (both start at multiples of 32).
        bool act[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int k0 = n0 + 32 * kb;
            act[kb] = (k0 < q0 + 32) && (k0 < N);
        }
        if (!act[0]) continue;

        f32x16 s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            if (!act[kb]) continue;
            const int k0 = n0 + 32 * kb;
            if (!fixed) {
#pragma unroll
                for (int v = 0; v < 16; ++v) s[kb][v] = 0.0f;
#pragma unroll
                for (int dc = 0; dc < 4; ++dc)
                    mma(s[kb], ld8<T>(&sm.k[32 * kb + c][16 * dc + 8 * hf]), qf[dc]);
#pragma unroll
                for (int v = 0; v < 16; ++v) s[kb][v] *= p.scale_log2;
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int kl = 32 * kb + 8 * (v >> 2) + 4 * hf + (v & 3);  // key within tile
                    const int x = (qq - m0) - kl + (FWD_BN - 1);               // band index of qq - (n0 + kl)
                    s[kb][v] = (sm.a[kl] + sm.rb[x]) * LOG2E;
                }
            }
            if (k0 == q0) {  // diagonal sub-block: hide keys after the query
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int kk = k0 + 8 * (v >> 2) + 4 * hf + (v & 3);
                    if (kk > qq) s[kb][v] = -INFINITY;
                }
            }
        }

        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            if (!act[kb]) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kb][v]);
        }
        mx = fmaxf(mx, xor32(mx));
        const float m_new = fmaxf(m_run, mx);
        const float alpha = fast_exp2(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[db][v] *= alpha;

#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            if (!act[kb]) continue;
            float ls = 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float e = fast_exp2(s[kb][v] - m_new);
                s[kb][v] = e;
                ls += e;
            }
            l_run += ls;
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const frag pb = to_operand<T>(s[kb], 8 * kc);
#pragma unroll
                for (int db = 0; db < 2; ++db)
                    mma(oacc[db], ld8<T>(&sm.vt[32 * db + c][32 * kb + 16 * kc + 8 * hf]), pb);
            }
        }
    }

    const float l_tot = l_run + xor32(l_run);
    if (qq < N) {
        const float inv = 1.0f / l_tot;
        T* orow = O + (size_t)qq * HEAD_DIM;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                st4<T>(orow + 32 * db + 8 * g + 4 * hf, oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv,
                       oacc[db][4 * g + 2] * inv, oacc[db][4 * g + 3] * inv);
        if (hf == 0) LSE[qq] = (m_run + __log2f(l_tot)) * LN2;
    }
}

}  // namespace saf
