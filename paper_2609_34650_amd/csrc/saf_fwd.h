// Forward of the hybrid causal-attention layer: one launch for all heads.
//
// Workgroup = (batch b, head h, block of 256 queries); 4 wavefronts, each
// owning 64 consecutive queries as two 32-query column blocks.  The head's
// flag picks the program of the whole workgroup (Appendix "Mixed-head
// execution and numerical checks": one program per batch element, head and
// query block, a head-state flag selects the computation, outputs keep the
// original head order).
//
// Every product streams one operand from LDS and keeps the other in
// registers.  A 32x32x16 MFMA takes 32 cycles and its LDS operand is 1 KB, so
// with one 32-wide register block the four SIMDs would need all of the CU's
// LDS bandwidth (128 bytes per clock); with two register blocks per wavefront
// every LDS fragment feeds two MFMAs and LDS runs at half that.
//
// Ordinary heads (Eqs. standard-head): FlashAttention-2 tiling with online
// softmax, the scheme the paper uses for ordinary heads.  Scores are formed
// transposed, S^T = K Q^T (keys x queries), so the accumulator of lane l holds
// one query (l % 32) and 16 of its keys: the running maximum and sum stay in
// the lane (one exchange with the other lane half per tile), the
// exponentials go straight into the B operand of O^T += V^T P^T, and O^T
// again holds one query per lane.  K and V tiles of 64 keys are copied from
// memory straight into column-slab LDS tiles by buffer loads (rows past N
// arrive as zeros), double-buffered so the next tile is in flight while this
// one is used; V^T comes from transposing LDS reads.  Tiles below the block's
// diagonal run a mask-free body.  Probabilities are formed against the
// running maximum as it stands; only when a sub-block's partial sum shows
// that its scores exceed that maximum by a wide margin is the maximum
// recomputed and the accumulator rescaled, so most tiles do neither.
//
// Fixed heads (Eq. compact-prior): P(i,j) = exp(a[j] + r[i-j]) / Z(i) factors
// as ea(j) * er(i-j) / Z'(i) with ea = exp(a - A*), er = exp(r - R*) and
// A*, R* the maxima of a and r over the positions the block touches.  V
// tiles come by buffer loads straight to LDS; the Toeplitz band er(i-j) is
// kept in float32 in LDS beside ea of the tile's keys, and each chunk's
// weight operand er(i-j) ea(j) is formed in float32 and rounded once -- no
// exponential, no score and no softmax per element; a band entry of a
// negative offset is 0, which is the causal mask.  The same float32 weights
// are summed into Z'(i) as they are formed, so the block writes O = acc / Z'
// and log Z = A* + R* + ln Z' itself (the paper precomputes the normalisers;
// here no pre-pass is needed).  This is exact up to rounding as long as no
// row's terms all underflow; a block where the largest of a row's diagonal
// and sink terms lies more than FAST_GUARD below A* + R* runs the exact
// per-element program instead, an online softmax that also writes log Z.
#pragma once

#include "saf_common.h"

namespace saf {

constexpr int FWD_BM = 256;  // queries per workgroup
constexpr int FWD_QW = 64;   // queries per wavefront (two 32-query blocks)
constexpr int FWD_BN = 64;   // keys per tile
constexpr int FWD_THREADS = 256;
// A sub-block's probabilities are taken against the running maximum as it
// stands; the maximum is only raised (and the accumulators rescaled) when a
// lane's partial sum over the sub-block exceeds this bound, so no
// probability exceeds it either.  Values up to 2^20 are harmless in float32
// sums and in bf16 operands (same exponent range).
constexpr float RESCALE_SUM = 1048576.0f;
constexpr int FWD_BAND = FWD_BM + FWD_BN - 1;            // offsets met by one tile
constexpr int FWD_BAND_STRIDE = (FWD_BAND + 7) / 8 * 8 + 8;  // every copy 16-byte aligned
static_assert(FWD_THREADS / 64 * FWD_QW == FWD_BM, "wavefronts cover the query block");
static_assert(BAND_COPIES * FWD_BAND_STRIDE * 2 <= tile_elems<bf16>() * 2, "band copies fit in a tile");
static_assert((FWD_BN + FWD_BAND) * 4 <= tile_elems<bf16>() * 2, "exact-program a and r fit in a tile");
static_assert(FWD_BAND <= 2 * FWD_THREADS, "two band entries per thread");

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
    unsigned char head_order[64];  // ordinary heads, then fixed heads (slice_of)
};

// Per-lane geometry of one workgroup: the wavefront's queries are q0 .. q0+63,
// query block qb covers q0 + 32*qb .. +31, and this lane's query in it is
// q0 + 32*qb + c.
struct FwdLane {
    int tid, w, lane, c, hf, m0, q0, N;
};

template <typename T>
__device__ __forceinline__ void store_rows(T* O, float* LSE, const FwdLane& L, int qq, const f32x16 (&oacc)[2],
                                           float inv, float lse, bool write_lse) {
    if (qq >= L.N) return;
    T* orow = O + (size_t)qq * HEAD_DIM;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g)
            st4<T>(orow + 32 * db + 8 * g + 4 * L.hf, oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv,
                   oacc[db][4 * g + 2] * inv, oacc[db][4 * g + 3] * inv);
    if (write_lse && L.hf == 0) LSE[qq] = lse;
}

// ---------------------------------------------------------------------------
// Ordinary heads
// ---------------------------------------------------------------------------

// Raise the running maxima of both query blocks to at least mx (log2
// units) and rescale the row sums and accumulators to match.
__device__ __forceinline__ void ord_rescale(const float (&mx)[2], float (&m_run)[2], float (&l_run)[2],
                                            f32x16 (&oacc)[2][2]) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float m_new = fmaxf(m_run[qb], mx[qb]);
        const float alpha = fast_exp2(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[qb][db][v] *= alpha;
    }
}

// exp2(s * sl2 - m) for both query blocks, with this lane's partial sums.
__device__ __forceinline__ void ord_probs(const f32x16 (&s)[2], const float (&m_run)[2], float sl2, f32x16 (&pr)[2],
                                          float (&ts)[2]) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float neg_m = -m_run[qb];
        float t0 = 0.0f, t1 = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; v += 2) {
            pr[qb][v] = fast_exp2(fmaf(s[qb][v], sl2, neg_m));
            pr[qb][v + 1] = fast_exp2(fmaf(s[qb][v + 1], sl2, neg_m));
            t0 += pr[qb][v];
            t1 += pr[qb][v + 1];
        }
        ts[qb] = t0 + t1;
    }
}

// One 64-key tile, as two 32-key sub-blocks kb processed one after the
// other (a scheduling barrier keeps their live ranges apart).  s[qb]: scores
// of the sub-block's 32 keys (rows) against query block qb (columns).  MASK:
// the tile meets the diagonal; keys after a query are hidden by one compare
// per score (no branches, so the masked body schedules like the plain one).
// A sub-block wholly after the wavefront's queries is skipped.
template <typename T, bool MASK>
__device__ __forceinline__ void ord_tile(const T* kt, const T* vt, int n0, const FwdLane& L,
                                         const typename Vec<T>::x8 (&qf)[2][4], f32x16 (&oacc)[2][2],
                                         float (&m_run)[2], float (&l_run)[2], float sl2) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int k0 = n0 + 32 * kb;
        if (MASK && k0 > L.q0 + FWD_QW - 1) break;
        f32x16 s[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int v = 0; v < 16; ++v) s[qb][v] = 0.0f;
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) {
            const frag kf = ld_row<T>(kt, 32 * kb + L.c, 16 * dc + 8 * L.hf);
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) mma(s[qb], kf, qf[qb][dc]);
        }
        if (MASK) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const int qq = L.q0 + 32 * qb + L.c;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int kk = k0 + 8 * (v >> 2) + 4 * L.hf + (v & 3);
                    s[qb][v] = kk > qq ? -INFINITY : s[qb][v];
                }
            }
        }
        // Probabilities against the running maximum; the maximum itself is
        // only recomputed when some lane's partial sum shows that this
        // sub-block exceeds it by a wide margin (or on the first visible
        // sub-block, where the maximum is still NEG_BIG and the sums are inf).
        f32x16 pr[2];
        float ts[2];
        ord_probs(s, m_run, sl2, pr, ts);
        if (__any(ts[0] > RESCALE_SUM || ts[1] > RESCALE_SUM)) {
            float mx[2];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                float m = vmax(s[qb][0], s[qb][1]);
#pragma unroll
                for (int v = 2; v < 16; v += 2) m = vmax(vmax(m, s[qb][v]), s[qb][v + 1]);
                mx[qb] = pair_max(m) * sl2;
            }
            ord_rescale(mx, m_run, l_run, oacc);
            ord_probs(s, m_run, sl2, pr, ts);
        }
        frag pb[2][2];  // [qb][kc]
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            l_run[qb] += ts[qb];  // float32 row sum, before rounding to the operand type
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) pb[qb][kc] = to_operand<T>(pr[qb], 8 * kc);
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                const frag vf = ld_tile_t<true>(vt, 32 * kb + 16 * kc, 32 * db);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) mma(oacc[qb][db], vf, pb[qb][kc]);
            }
        __builtin_amdgcn_sched_barrier(0);
    }
}

template <typename T>
__device__ __forceinline__ void fwd_ordinary(const Tiles<T>& sm, const FwdArgs& p, const FwdLane& L, size_t base,
                                             size_t row_base) {
    // Tiles: K in t[0] / t[1], V in t[2] / t[3] (two buffers each).
    const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + base;
    const __amdgpu_buffer_rsrc_t rk = slice_rsrc<T>(reinterpret_cast<const T*>(p.k) + base, L.N);
    const __amdgpu_buffer_rsrc_t rv = slice_rsrc<T>(reinterpret_cast<const T*>(p.v) + base, L.N);
    typedef typename Vec<T>::x8 frag;
    frag qf[2][4];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qq = L.q0 + 32 * qb + L.c;
#pragma unroll
        for (int dc = 0; dc < 4; ++dc)
            qf[qb][dc] = qq < L.N ? ld8<T>(Q + (size_t)qq * HEAD_DIM + 16 * dc + 8 * L.hf) : zero8<T>();
    }
    f32x16 oacc[2][2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[qb][db][v] = 0.0f;
    float m_run[2] = {NEG_BIG, NEG_BIG};
    float l_run[2] = {0.0f, 0.0f};  // this lane's share of each row sum

    // Slots: first the tiles that meet the diagonal (masked), then the tiles
    // wholly below the block's first query (mask-free).
    const int n_tiles = (min(L.m0 + FWD_BM, L.N) + FWD_BN - 1) / FWD_BN;
    const int n_full = L.m0 / FWD_BN;
    const int n_mask = n_tiles - n_full;  // 1 .. 4
    const int P = (n_mask + 1) & ~1;
    run_slots(
        P, P + n_full, [&](int i) { return i < P ? (i < n_mask ? n_full + i : -1) : i - P; },
        [&](auto buf, int t) {
            tile_load_lds<T>(sm.t[decltype(buf)::value], rk, t * FWD_BN, L.w, L.lane);
            tile_load_lds<T>(sm.t[2 + decltype(buf)::value], rv, t * FWD_BN, L.w, L.lane);
        },
        [&](auto) {},
        [&](auto buf, int t, auto mask) {
            ord_tile<T, decltype(mask)::value>(sm.t[decltype(buf)::value], sm.t[2 + decltype(buf)::value],
                                               t * FWD_BN, L, qf, oacc, m_run, l_run, p.scale_log2);
        });
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float l_tot = pair_sum(l_run[qb]);
        store_rows<T>(reinterpret_cast<T*>(p.o) + base, p.lse + row_base, L, L.q0 + 32 * qb + L.c, oacc[qb],
                      1.0f / l_tot, (m_run[qb] + __log2f(l_tot)) * LN2, true);
    }
}

// ---------------------------------------------------------------------------
// Fixed heads, exact per-element program (fallback)
// ---------------------------------------------------------------------------

template <typename T>
__device__ __forceinline__ void fwd_fixed_exact(const Tiles<T>& sm, const FwdArgs& p, const FwdLane& L, size_t base,
                                                size_t row_base, const float* arow, const float* rrow) {
    // Tiles: V in t[0]; a of the tile's keys and r over its offsets in t[1].
    T* vt = sm.t[0];
    float* as = reinterpret_cast<float*>(sm.t[1]);
    float* rb = as + FWD_BN;  // rb[x] = r(m0 - n0 - 63 + x)
    const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + base;
    typedef typename Vec<T>::x8 frag;
    const int N = L.N;
    f32x16 oacc[2][2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[qb][db][v] = 0.0f;
    float m_run[2] = {NEG_BIG, NEG_BIG};
    float l_run[2] = {0.0f, 0.0f};
    const int n_end = min(L.m0 + FWD_BM, N);
    const int row = unit_row<T>(L.w, L.lane);
    for (int n0 = 0; n0 < n_end; n0 += FWD_BN) {
        __syncthreads();
#pragma unroll
        for (int k = 0; k < tile_units<T>(); ++k) {
            const int col = unit_col<T>(L.w, L.lane, k);
            const u32x4 z = {0u, 0u, 0u, 0u};
            const u32x4 x = n0 + row < N ? ld_unit(V + (size_t)(n0 + row) * HEAD_DIM + col) : z;
            *reinterpret_cast<u32x4*>(vt + toff<T>(row, col)) = x;
        }
        if (L.tid < FWD_BN) as[L.tid] = (n0 + L.tid < N) ? arow[n0 + L.tid] : -INFINITY;
        for (int x = L.tid; x < FWD_BAND; x += FWD_THREADS) {
            const int delta = L.m0 - n0 - (FWD_BN - 1) + x;
            rb[x] = (delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
        }
        __syncthreads();
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            const int qs = L.q0 + 32 * qb;
            if (!(n0 <= qs + 31)) continue;  // tile wholly after this query block
            const int ql = qs + L.c - L.m0;  // query within the block
            f32x16 s[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int kl = 32 * kb + 8 * (v >> 2) + 4 * L.hf + (v & 3);
                    s[kb][v] = (as[kl] + rb[ql - kl + (FWD_BN - 1)]) * LOG2E;
                }
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kb][v]);
            mx = pair_max(mx);
            const float m_new = fmaxf(m_run[qb], mx);
            const float alpha = fast_exp2(m_run[qb] - m_new);
            m_run[qb] = m_new;
            l_run[qb] *= alpha;
#pragma unroll
            for (int db = 0; db < 2; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) oacc[qb][db][v] *= alpha;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const float e = fast_exp2(s[kb][v] - m_new);
                    s[kb][v] = e;
                    l_run[qb] += e;
                }
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    const frag pb = to_operand<T>(s[kb], 8 * kc);
#pragma unroll
                    for (int db = 0; db < 2; ++db)
                        mma(oacc[qb][db], ld_tile_t<true>(vt, 32 * kb + 16 * kc, 32 * db), pb);
                }
            }
        }
    }
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float l_tot = pair_sum(l_run[qb]);
        store_rows<T>(reinterpret_cast<T*>(p.o) + base, p.lse + row_base, L, L.q0 + 32 * qb + L.c, oacc[qb],
                      1.0f / l_tot, (m_run[qb] + __log2f(l_tot)) * LN2, true);
    }
}

// ---------------------------------------------------------------------------
// Fixed heads, factorised program
// ---------------------------------------------------------------------------

// Small per-tile values in registers between their loads (issued a tile
// ahead) and their LDS stores: a of one key, two band entries.  V tiles come
// by buffer loads straight to LDS, unscaled.
struct FixStage {
    float a;      // a of key n0 + L.tid (L.tid < FWD_BN)
    float rb[2];  // band entries
};

// Band entry u of the tile at n0 holds offset (m0 - n0 + FWD_BM - 1) - u.
__device__ __forceinline__ void fix_load(FixStage& st, const float* arow, const float* rrow, int n0,
                                         const FwdLane& L) {
    st.a = (L.tid < FWD_BN && n0 + L.tid < L.N) ? arow[n0 + L.tid] : -INFINITY;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int u = L.tid + FWD_THREADS * k;
        const int delta = L.m0 - n0 + (FWD_BM - 1) - u;
        st.rb[k] = (u < FWD_BAND && delta >= 0 && delta < L.N) ? rrow[delta] : -INFINITY;
    }
}

// eas: ea of the tile's keys; band: copy s of er (float32) at
// s * FWD_BAND_STRIDE, FIX_BAND_COPIES copies (16-byte reads of float32 need
// four).
constexpr int FIX_BAND_COPIES = 4;
static_assert(FIX_BAND_COPIES * FWD_BAND_STRIDE * 4 <= tile_elems<bf16>() * 2, "float32 band copies fit in a tile");

__device__ __forceinline__ void fix_store(float* eas, float* band, const FixStage& st, const FwdLane& L, float a_sh,
                                          float r_sh) {
    if (L.tid < FWD_BN) eas[L.tid] = fast_exp2(fmaf(st.a, LOG2E, -a_sh));  // 0 past N
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int u = L.tid + FWD_THREADS * k;
        if (u < FWD_BAND) {
            const float e = fast_exp2(fmaf(st.rb[k], LOG2E, -r_sh));
#pragma unroll
            for (int s = 0; s < FIX_BAND_COPIES; ++s)
                if (u >= s) band[s * FWD_BAND_STRIDE + u - s] = e;
        }
    }
}

// O^T += V^T (band ea)^T: four 16-key chunks; the weight operand of lane
// (query column c, half hf) in chunk G is band entries u0 .. u0 + 7 times ea
// of keys 16G + 8hf .. 16G + 8hf + 7, formed in float32 and rounded once.
// z[qb] collects this lane's share of the row sum Z'(i) of the float32
// weights (the other lane half holds the other eight keys of each chunk).
template <typename T, bool MASK>
__device__ __forceinline__ void fix_tile(const T* vs, const float* band, const float* eas, int n0, const FwdLane& L,
                                         f32x16 (&oacc)[2][2], float (&z)[2]) {
    typedef typename Vec<T>::x8 frag;
#pragma unroll
    for (int G = 0; G < 4; ++G) {
        if (MASK && n0 + 16 * G > L.q0 + FWD_QW - 1) continue;  // chunk wholly after this wavefront's queries
        frag vf[2];
#pragma unroll
        for (int db = 0; db < 2; ++db) vf[db] = ld_tile_t<false>(vs, 16 * G, 32 * db);
        const f32x4 e0 = *reinterpret_cast<const f32x4*>(eas + 16 * G + 8 * L.hf);
        const f32x4 e1 = *reinterpret_cast<const f32x4*>(eas + 16 * G + 8 * L.hf + 4);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            if (MASK && n0 + 16 * G > L.q0 + 32 * qb + 31) continue;
            const int ql = L.q0 - L.m0 + 32 * qb + L.c;  // query within the block
            const int u0 = (FWD_BM - 1) - ql + 16 * G + 8 * L.hf;
            const int s = u0 & (FIX_BAND_COPIES - 1);
            const float* bp = band + s * FWD_BAND_STRIDE + u0 - s;
            const f32x4 b0 = *reinterpret_cast<const f32x4*>(bp);
            const f32x4 b1 = *reinterpret_cast<const f32x4*>(bp + 4);
            frag w;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const float x0 = b0[t] * e0[t], x1 = b1[t] * e1[t];
                w[t] = (T)x0;
                w[4 + t] = (T)x1;
                z[qb] += x0 + x1;
            }
#pragma unroll
            for (int db = 0; db < 2; ++db) mma(oacc[qb][db], vf[db], w);
        }
    }
}

template <typename T>
__device__ __forceinline__ void fwd_fixed(const Tiles<T>& sm, const FwdArgs& p, const FwdLane& L, size_t base,
                                          size_t row_base, int h) {
    // Tiles: V in t[0] / t[1], the float32 band in t[2] / t[3], ea in aux.
    const T* __restrict__ V = reinterpret_cast<const T*>(p.v) + base;
    const float* __restrict__ arow = p.a + (size_t)h * p.ld_prior;
    const float* __restrict__ rrow = p.r + (size_t)h * p.ld_prior;
    const int N = L.N;
    const int m1 = min(L.m0 + FWD_BM, N);

    // Shifts: maxima of a and r over the positions this block touches.
    float am = -INFINITY, rm = -INFINITY;
    for (int j = L.tid; j < m1; j += FWD_THREADS) {
        am = fmaxf(am, arow[j]);
        rm = fmaxf(rm, rrow[j]);
    }
    const float A = block_max(am, sm.red);
    const float R = block_max(rm, sm.red);
    // Guard: every row's diagonal or sink term within FAST_GUARD of A + R,
    // so Z'(i) >= exp(-FAST_GUARD) and no row underflows.
    bool ok = true;
    if (L.tid < FWD_BM && L.m0 + L.tid < N) {
        const int i = L.m0 + L.tid;
        ok = fmaxf(arow[i] + rrow[0], arow[0] + rrow[i]) - A - R >= -FAST_GUARD;
    }
    if (!__syncthreads_and(ok)) {
        fwd_fixed_exact<T>(sm, p, L, base, row_base, arow, rrow);
        return;
    }
    const float a_sh = A * LOG2E, r_sh = R * LOG2E;

    f32x16 oacc[2][2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[qb][db][v] = 0.0f;

    const int n_tiles = (m1 + FWD_BN - 1) / FWD_BN;
    const int n_full = L.m0 / FWD_BN;
    const int n_mask = n_tiles - n_full;
    const int P = (n_mask + 1) & ~1;
    const __amdgpu_buffer_rsrc_t rv = slice_rsrc<T>(V, N);
    float z[2] = {0.0f, 0.0f};
    FixStage st;
    run_slots(
        P, P + n_full, [&](int i) { return i < P ? (i < n_mask ? n_full + i : -1) : i - P; },
        [&](auto buf, int t) {
            tile_load_lds<T>(sm.t[decltype(buf)::value], rv, t * FWD_BN, L.w, L.lane);
            fix_load(st, arow, rrow, t * FWD_BN, L);
        },
        [&](auto buf) {
            constexpr int b = decltype(buf)::value;
            fix_store(sm.aux[b], reinterpret_cast<float*>(sm.t[2 + b]), st, L, a_sh, r_sh);
        },
        [&](auto buf, int t, auto mask) {
            constexpr int b = decltype(buf)::value;
            fix_tile<T, decltype(mask)::value>(sm.t[b], reinterpret_cast<const float*>(sm.t[2 + b]), sm.aux[b],
                                               t * FWD_BN, L, oacc, z);
        });
    // O(i) = acc(i) / Z'(i) and log Z(i) = A + R + ln Z'(i), with Z'(i) the
    // sum of the same float32 weights (the guard keeps it above e^-40).
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float zt = pair_sum(z[qb]);
        store_rows<T>(reinterpret_cast<T*>(p.o) + base, p.lse + row_base, L, L.q0 + 32 * qb + L.c, oacc[qb],
                      1.0f / zt, A + R + __log2f(zt) * LN2, true);
    }
}

// ---------------------------------------------------------------------------
// Fixed-head normaliser pass (the compact fitter's log Z of each step):
// LSE[b, h, i] = log Z(i) for every batch
// element b (Z depends on a and r only).  Workgroup = (fixed head, 32 rows);
// eight threads share a row and each sums a 64-key slice of every 512-key
// tile: Z'(i) = sum_j ea(j) er(i - j) in float32, with ea = exp(a - A_t) and
// er = exp(r - R_t) shifted by the tile's maxima A_t, R_t; the tiles combine
// online under the largest shift M seen so far, so log Z = M + log Z'.  A
// row whose Z' ends below 2^-80 (its terms underflowed) is summed exactly,
// with a running maximum.  A budget of six wavefronts per SIMD (about 80
// VGPRs): the fitter launches 1536 workgroups per step, and left free the
// scheduler hoists every LDS read of the key loop into registers (164
// VGPRs, three wavefronts per SIMD, 7 % slower).
// ---------------------------------------------------------------------------
constexpr int NORM_THREADS = 256;
constexpr int NORM_ROWS = 32;
constexpr int NORM_PARTS = NORM_THREADS / NORM_ROWS;  // threads per row
constexpr int NORM_KT = 512;                          // keys per tile
constexpr int NORM_PART_KEYS = NORM_KT / NORM_PARTS;  // 64
constexpr int NORM_BAND = NORM_ROWS + NORM_KT - 1;    // offsets per tile

struct NormArgs {
    const float* a;
    const float* r;
    float* lse;
    int B, H, N, ld_prior, n_rblocks, n_fixed;
    unsigned char heads[64];  // the fixed heads, ascending
};

__global__ __launch_bounds__(NORM_THREADS) __attribute__((amdgpu_waves_per_eu(6))) void fixed_lse_kernel(
    NormArgs p) {
    __shared__ __attribute__((aligned(16))) float ea_s[NORM_KT];
    __shared__ float er_s[NORM_BAND + 1];
    __shared__ float red[2][4];
    __shared__ float zs[NORM_PARTS][NORM_ROWS];
    const int rblk = p.n_rblocks - 1 - (int)(blockIdx.x / p.n_fixed);  // longest first
    const int h = p.heads[blockIdx.x % p.n_fixed];
    const int tid = threadIdx.x;
    const int row = tid % NORM_ROWS;
    const int part = tid / NORM_ROWS;
    const int N = p.N;
    const float* __restrict__ arow = p.a + (size_t)h * p.ld_prior;
    const float* __restrict__ rrow = p.r + (size_t)h * p.ld_prior;
    const int i0 = rblk * NORM_ROWS;
    const int m1 = min(i0 + NORM_ROWS, N);
    const int i = i0 + row;

    float M = -INFINITY;  // shift of S (uniform over the workgroup)
    float S = 0.0f;       // this thread's share of Z(i) * exp(-M)
    for (int j0 = 0; j0 < m1; j0 += NORM_KT) {
        float av[NORM_KT / NORM_THREADS], rv[3];
        float amx = -INFINITY, rmx = -INFINITY;
#pragma unroll
        for (int k = 0; k < NORM_KT / NORM_THREADS; ++k) {
            const int j = j0 + tid + NORM_THREADS * k;
            av[k] = j < m1 ? arow[j] : -INFINITY;
            amx = fmaxf(amx, av[k]);
        }
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const int x = tid + NORM_THREADS * k;  // er_s[x] = er(i0 - j0 - 511 + x)
            const int delta = i0 - j0 - (NORM_KT - 1) + x;
            rv[k] = (x < NORM_BAND && delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
            rmx = fmaxf(rmx, rv[k]);
        }
        amx = wave_max(amx);
        rmx = wave_max(rmx);
        if ((tid & 63) == 0) {
            red[0][tid >> 6] = amx;
            red[1][tid >> 6] = rmx;
        }
        __syncthreads();
        const float At = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
        const float Rt = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3]));
#pragma unroll
        for (int k = 0; k < NORM_KT / NORM_THREADS; ++k)
            ea_s[tid + NORM_THREADS * k] = fast_exp2((av[k] - At) * LOG2E);
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const int x = tid + NORM_THREADS * k;
            if (x < NORM_BAND) er_s[x] = fast_exp2((rv[k] - Rt) * LOG2E);
        }
        __syncthreads();
        const float ct = At + Rt;
        if (ct > M) {
            S *= fast_exp2((M - ct) * LOG2E);
            M = ct;
        }
        const int jb = part * NORM_PART_KEYS;
        const int xb = row - jb + (NORM_KT - 1);  // er_s index of key j0 + jb for row i
        float z0 = 0.0f, z1 = 0.0f, z2 = 0.0f, z3 = 0.0f;
#pragma unroll
        for (int m = 0; m < NORM_PART_KEYS; m += 4) {
            const f32x4 e = *reinterpret_cast<const f32x4*>(&ea_s[jb + m]);
            z0 = fmaf(e[0], er_s[xb - m], z0);
            z1 = fmaf(e[1], er_s[xb - m - 1], z1);
            z2 = fmaf(e[2], er_s[xb - m - 2], z2);
            z3 = fmaf(e[3], er_s[xb - m - 3], z3);
        }
        S = fmaf((z0 + z1) + (z2 + z3), fast_exp2((ct - M) * LOG2E), S);
        __syncthreads();
    }
    zs[part][row] = S;
    __syncthreads();
    if (part != 0 || i >= N) return;
    float z = 0.0f;
#pragma unroll
    for (int q = 0; q < NORM_PARTS; ++q) z += zs[q][row];
    float lse;
    if (z >= 0x1p-80f) {
        lse = M + __log2f(z) * LN2;
    } else {
        float m = -INFINITY, s = 0.0f;
        for (int j = 0; j <= i; ++j) {
            const float x = arow[j] + rrow[i - j];
            if (x > m) {
                s = s * expf(m - x) + 1.0f;
                m = x;
            } else {
                s += expf(x - m);
            }
        }
        lse = m + logf(s);
    }
    for (int b = 0; b < p.B; ++b) p.lse[((size_t)b * p.H + h) * N + i] = lse;
}

// ---------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(FWD_THREADS) __attribute__((amdgpu_waves_per_eu(2))) void fwd_kernel(FwdArgs p) {
    __shared__ __attribute__((aligned(16))) T t0[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t1[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t2[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T t3[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) float ea0[FWD_BN];
    __shared__ __attribute__((aligned(16))) float ea1[FWD_BN];
    __shared__ float red[4];
    const Tiles<T> sm = {{t0, t1, t2, t3}, {ea0, ea1}, red};
    // Longest blocks first: level -> query block in descending order.
    const SliceOf sl = slice_of(blockIdx.x, p.B, p.H, 1, [&](int k) { return (int)p.head_order[k]; });
    const int qblk = p.n_qblocks - 1 - sl.level;
    const int h = sl.h;
    const int bh = sl.b * p.H + h;
    const bool fixed = (p.fixed_mask >> h) & 1ull;
    FwdLane L;
    L.tid = threadIdx.x;
    L.w = L.tid >> 6;
    L.lane = L.tid & 63;
    L.c = L.tid & 31;
    L.hf = (L.tid >> 5) & 1;
    L.m0 = qblk * FWD_BM;
    L.q0 = L.m0 + FWD_QW * L.w;
    L.N = p.N;
    const size_t base = (size_t)bh * p.N * HEAD_DIM;
    const size_t row_base = (size_t)bh * p.N;
    if (fixed)
        fwd_fixed<T>(sm, p, L, base, row_base, h);
    else
        fwd_ordinary<T>(sm, p, L, base, row_base);
}

}  // namespace saf
