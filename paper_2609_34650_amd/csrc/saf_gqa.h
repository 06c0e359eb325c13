// Forward of the hybrid layer with grouped-query attention and head
// dimensions 64, 96 or 128 (the layouts of the paper's grouped-query prefill
// measurement and of its 1B model's head width: Appendix "Replacement in
// pretrained models", subsection "GQA prefill measurements"; Appendix "1B
// training and evaluation"; and Appendix "Mixed-head execution and numerical
// checks", where the grouped-query implementation drops the replaced heads'
// query projections but keeps every shared key and value head).
//
// Q, O: [B, Hq, N, D]; K, V: [B, Hkv, N, D]; query head h reads key/value
// head h / (Hq / Hkv).  A fixed query head reads only V of its group.
//
// Workgroup = (batch b, query head h, block of 128 queries), 4 wavefronts of
// 32 queries (one query per lane column c, as in the layer's forward: scores
// are formed transposed, S^T = K Q^T, keys in accumulator rows).  K and V
// tiles of 64 keys go to column-slab LDS tiles D wide by buffer loads straight
// to LDS, double-buffered; the tiles that meet the diagonal come first with a
// per-score causal compare.
//   Ordinary head: online softmax (running maximum raised when a sub-block
//   exceeds it, accumulator and sum rescaled), O^T += V^T P^T on MFMA, LSE =
//   m + ln l.
//   Fixed head, factorised (as in the layer forward): P(i, j) =
//   ea(j) er(i - j) / Z'(i) with ea = exp(a - A), er = exp(r - R) and A, R
//   the maxima of a and r over the block's positions.  V tiles come by
//   buffer loads to LDS unscaled, and the weight operand is the Toeplitz
//   band er (float32 in LDS, eight shifted copies keep every 8-entry read
//   aligned) times ea of the chunk's keys, formed in float32 and rounded
//   once: no exponential per entry.  The same weights are summed into Z'(i),
//   so O = acc / Z' and LSE = log Z = A + R + ln Z' come out of this kernel.
//   A block where some row's diagonal and sink terms both lie more than
//   FAST_GUARD below A + R takes the exact per-entry program: the logits
//   a[j] + r[i - j] (the tile's a values and r band staged in LDS) through
//   an online softmax, as for an ordinary head's scores.
#pragma once

#include "saf_common.h"

namespace saf {

constexpr int GQA_BM = 128;  // queries per workgroup
constexpr int GQA_BN = 64;   // keys per tile
constexpr int GQA_THREADS = 256;
constexpr int GQA_BAND = GQA_BM + GQA_BN - 1;  // offsets met by one tile
constexpr int GQA_BAND_STRIDE = (GQA_BAND + 7) / 8 * 8 + 8;  // every band copy 16-byte aligned
static_assert(GQA_BAND <= GQA_THREADS, "one band entry per thread");

struct GqaArgs {
    const void* q;
    const void* k;
    const void* v;
    const float* a;
    const float* r;
    void* o;
    float* lse;
    uint64_t fixed_mask;
    int B, Hq, Hkv, N, ld_prior, n_qblocks;
    float scale_log2;  // log2(e) / sqrt(D)
    // Key/value heads in order of decreasing work (an ordinary query head
    // weighs 2, a fixed one 1), for slice_of's XCD assignment.
    unsigned char kv_order[64];
};

struct GqaLane {
    int tid, w, lane, c, hf, m0, q0, N;
};

// One 64-key tile (two 32-key sub-blocks) of an ordinary head.
template <typename T, int D, bool MASK>
__device__ __forceinline__ void gqa_ord_tile(const T* kt, const T* vt, int n0, const GqaLane& L,
                                             const typename Vec<T>::x8 (&qf)[D / 16], f32x16 (&oacc)[D / 32],
                                             float& m_run, float& l_run, float sl2) {
    typedef typename Vec<T>::x8 frag;
    const int qq = L.q0 + L.c;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int k0 = n0 + 32 * kb;
        if (MASK && k0 > L.q0 + 31) break;  // sub-block wholly after the wavefront's queries
        f32x16 s;
#pragma unroll
        for (int v = 0; v < 16; ++v) s[v] = 0.0f;
#pragma unroll
        for (int dc = 0; dc < D / 16; ++dc) mma(s, ld_row<T>(kt, 32 * kb + L.c, 16 * dc + 8 * L.hf), qf[dc]);
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            if (MASK) {
                const int kk = k0 + 8 * (v >> 2) + 4 * L.hf + (v & 3);
                s[v] = kk > qq ? -INFINITY : s[v];
            }
            mx = vmax(mx, s[v]);
        }
        mx = pair_max(mx) * sl2;
        if (mx > m_run) {  // raise the running maximum, rescale (per lane; both halves agree)
            const float alpha = fast_exp2(m_run - mx);
            m_run = mx;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) oacc[db][v] *= alpha;
        }
        f32x16 pr;
        float t = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            pr[v] = fast_exp2(fmaf(s[v], sl2, -m_run));
            t += pr[v];
        }
        l_run += t;
        frag pb[2];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) pb[kc] = to_operand<T>(pr, 8 * kc);
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
            for (int db = 0; db < D / 32; ++db) mma(oacc[db], ld_tile_t<true>(vt, 32 * kb + 16 * kc, 32 * db), pb[kc]);
    }
}

// One 64-key tile of a fixed head, exact program: the logits a[j] + r[i - j]
// of each 32-key sub-block (as[k]: a of the tile's key k; rb[x]:
// r(m0 - n0 - 63 + x)) go through the same online softmax as an ordinary
// head's scores (running maximum raised when a sub-block exceeds it).
template <typename T, int D, bool MASK>
__device__ __forceinline__ void gqa_fix_tile(const T* vt, const float* as, const float* rb, int n0, const GqaLane& L,
                                             f32x16 (&oacc)[D / 32], float& m_run, float& l_run) {
    typedef typename Vec<T>::x8 frag;
    const int qq = L.q0 + L.c;
    const int ql = qq - L.m0;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int k0 = n0 + 32 * kb;
        if (MASK && k0 > L.q0 + 31) break;
        f32x16 sc;
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int kl = 32 * kb + 8 * (v >> 2) + 4 * L.hf + (v & 3);  // key within the tile
            float x = (as[kl] + rb[ql - kl + (GQA_BN - 1)]) * LOG2E;
            if (MASK && n0 + kl > qq) x = -INFINITY;
            sc[v] = x;
            mx = vmax(mx, x);
        }
        mx = pair_max(mx);
        if (mx > m_run) {
            const float alpha = fast_exp2(m_run - mx);
            m_run = mx;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) oacc[db][v] *= alpha;
        }
        f32x16 pr;
        float t = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            pr[v] = fast_exp2(sc[v] - m_run);
            t += pr[v];
        }
        l_run += t;
        frag pb[2];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) pb[kc] = to_operand<T>(pr, 8 * kc);
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
            for (int db = 0; db < D / 32; ++db) mma(oacc[db], ld_tile_t<true>(vt, 32 * kb + 16 * kc, 32 * db), pb[kc]);
    }
}

// Factorised fixed program: V tiles come by buffer loads to LDS unscaled;
// per tile, ea of its 64 keys and the band er of the offsets it meets go
// through registers (loaded a tile ahead) into LDS, ea in float32 beside the
// a values of the exact program, the band as eight shifted float32 copies in
// the unused K tile.
struct GqaFixStage {
    float a;   // a of key n0 + L.tid (L.tid < GQA_BN)
    float rb;  // one band entry
};

// Band entry u of the tile at n0 holds er at offset (m0 - n0 + 127) - u.
__device__ __forceinline__ void gqa_fix_load(GqaFixStage& st, const float* arow, const float* rrow, int n0,
                                             const GqaLane& L) {
    st.a = (L.tid < GQA_BN && n0 + L.tid < L.N) ? arow[n0 + L.tid] : -INFINITY;
    const int delta = L.m0 - n0 + (GQA_BM - 1) - L.tid;
    st.rb = (L.tid < GQA_BAND && delta >= 0 && delta < L.N) ? rrow[delta] : -INFINITY;
}

__device__ __forceinline__ void gqa_fix_store(float* eas, float* band, const GqaFixStage& st, const GqaLane& L,
                                              float a_sh, float r_sh) {
    if (L.tid < GQA_BN) eas[L.tid] = fast_exp2(fmaf(st.a, LOG2E, -a_sh));  // 0 past N
    if (L.tid < GQA_BAND) {
        const float e = fast_exp2(fmaf(st.rb, LOG2E, -r_sh));
#pragma unroll
        for (int s = 0; s < BAND_COPIES; ++s)
            if (L.tid >= s) band[s * GQA_BAND_STRIDE + L.tid - s] = e;
    }
}

// O^T += V^T (band ea)^T over one tile: four 16-key chunks; the weight
// operand of lane (c, hf) in chunk G is band entries u0 .. u0 + 7 (u0 =
// 127 - ql + 16G + 8hf, read from copy u0 % 8 at an aligned address) times
// ea of keys 16G + 8hf .. 16G + 8hf + 7, formed in float32 and rounded once.
// Offsets below zero hold 0, which masks the keys after the query.
// z collects this lane's share of the row sum Z'(i) of the float32 weights.
template <typename T, int D, bool MASK>
__device__ __forceinline__ void gqa_band_tile(const T* vs, const float* band, const float* eas, int n0,
                                              const GqaLane& L, f32x16 (&oacc)[D / 32], float& z) {
    typedef typename Vec<T>::x8 frag;
    const int ql = L.q0 - L.m0 + L.c;
#pragma unroll
    for (int G = 0; G < 4; ++G) {
        if (MASK && n0 + 16 * G > L.q0 + 31) continue;  // chunk wholly after this wavefront's queries
        const int u0 = (GQA_BM - 1) - ql + 16 * G + 8 * L.hf;
        const int s = u0 & 7;
        const float* bp = band + s * GQA_BAND_STRIDE + u0 - s;
        const f32x4 b0 = *reinterpret_cast<const f32x4*>(bp);
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(bp + 4);
        const f32x4 e0 = *reinterpret_cast<const f32x4*>(eas + 16 * G + 8 * L.hf);
        const f32x4 e1 = *reinterpret_cast<const f32x4*>(eas + 16 * G + 8 * L.hf + 4);
        frag b;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const float x0 = b0[t] * e0[t], x1 = b1[t] * e1[t];
            b[t] = (T)x0;
            b[4 + t] = (T)x1;
            z += x0 + x1;
        }
#pragma unroll
        for (int db = 0; db < D / 32; ++db) mma(oacc[db], ld_tile_t<false>(vs, 16 * G, 32 * db), b);
    }
}

template <typename T, int D>
__global__ __launch_bounds__(GQA_THREADS) __attribute__((amdgpu_waves_per_eu(2))) void gqa_fwd_kernel(GqaArgs p) {
    __shared__ __attribute__((aligned(16))) T k0s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T k1s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T v0s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) T v1s[tile_elems<T, D>()];
    __shared__ __attribute__((aligned(16))) float ab0[GQA_BN + GQA_BAND + 1];
    __shared__ __attribute__((aligned(16))) float ab1[GQA_BN + GQA_BAND + 1];
    __shared__ float red[8];
    static_assert(BAND_COPIES * GQA_BAND_STRIDE * 4 <= tile_elems<T, D>() * (int)sizeof(T),
                  "float32 band copies fit in a K tile");
    // Longest query blocks first; slices = (batch, key/value head).
    const int group = p.Hq / p.Hkv;
    const SliceOf sl = slice_of(blockIdx.x, p.B, p.Hkv, group, [&](int k) { return (int)p.kv_order[k]; });
    const int qblk = p.n_qblocks - 1 - sl.level;
    const int b = sl.b, h = sl.h;
    const int bh = b * p.Hq + h;
    const int hkv = h / group;
    const bool fixed = (p.fixed_mask >> h) & 1ull;
    GqaLane L;
    L.tid = threadIdx.x;
    L.w = __builtin_amdgcn_readfirstlane(L.tid >> 6);
    L.lane = L.tid & 63;
    L.c = L.tid & 31;
    L.hf = (L.tid >> 5) & 1;
    L.m0 = qblk * GQA_BM;
    L.q0 = L.m0 + 32 * L.w;
    L.N = p.N;
    const int N = p.N;
    const size_t qbase = (size_t)bh * N * D;
    const size_t kvbase = ((size_t)b * p.Hkv + hkv) * N * D;
    const size_t row_base = (size_t)bh * N;
    const __amdgpu_buffer_rsrc_t rk = slice_rsrc<T, D>(reinterpret_cast<const T*>(p.k) + kvbase, N);
    const __amdgpu_buffer_rsrc_t rv = slice_rsrc<T, D>(reinterpret_cast<const T*>(p.v) + kvbase, N);
    typedef typename Vec<T>::x8 frag;
    const int qq = L.q0 + L.c;

    f32x16 oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[db][v] = 0.0f;

    const int n_tiles = (min(L.m0 + GQA_BM, N) + GQA_BN - 1) / GQA_BN;
    const int n_full = L.m0 / GQA_BN;
    const int n_mask = n_tiles - n_full;  // 1 or 2
    const int P = (n_mask + 1) & ~1;
    auto tile_of = [&](int i) { return i < P ? (i < n_mask ? n_full + i : -1) : i - P; };
    float row_scale = 1.0f, lse_out = 0.0f;
    if (!fixed) {
        const T* __restrict__ Q = reinterpret_cast<const T*>(p.q) + qbase;
        frag qf[D / 16];
#pragma unroll
        for (int dc = 0; dc < D / 16; ++dc)
            qf[dc] = qq < N ? ld8<T>(Q + (size_t)qq * D + 16 * dc + 8 * L.hf) : zero8<T>();
        float m_run = NEG_BIG, l_run = 0.0f;
        run_slots(
            P, P + n_full, tile_of,
            [&](auto buf, int t) {
                constexpr int B_ = decltype(buf)::value;
                tile_load_lds<T, D>(B_ ? k1s : k0s, rk, t * GQA_BN, L.w, L.lane);
                tile_load_lds<T, D>(B_ ? v1s : v0s, rv, t * GQA_BN, L.w, L.lane);
            },
            [&](auto) {},
            [&](auto buf, int t, auto mask) {
                constexpr int B_ = decltype(buf)::value;
                gqa_ord_tile<T, D, decltype(mask)::value>(B_ ? k1s : k0s, B_ ? v1s : v0s, t * GQA_BN, L, qf, oacc,
                                                          m_run, l_run, p.scale_log2);
            });
        const float l_tot = pair_sum(l_run);
        row_scale = 1.0f / l_tot;
        lse_out = (m_run + __log2f(l_tot)) * LN2;
    } else {
        const float* arow = p.a + (size_t)h * p.ld_prior;
        const float* rrow = p.r + (size_t)h * p.ld_prior;
        const int m1 = min(L.m0 + GQA_BM, N);
        float am = -INFINITY, rm = -INFINITY;
        for (int j = L.tid; j < m1; j += GQA_THREADS) {
            am = fmaxf(am, arow[j]);
            rm = fmaxf(rm, rrow[j]);
        }
        const float A = block_max(am, red);
        const float R = block_max(rm, red + 4);
        bool ok = true;
        if (L.tid < GQA_BM && L.m0 + L.tid < N) {
            const int i = L.m0 + L.tid;
            ok = fmaxf(arow[i] + rrow[0], arow[0] + rrow[i]) - A - R >= -FAST_GUARD;
        }
        if (__syncthreads_and(ok)) {
            // K is never read for a fixed head: its tiles hold the band.
            const float a_sh = A * LOG2E, r_sh = R * LOG2E;
            float z = 0.0f;
            GqaFixStage st;
            run_slots(
                P, P + n_full, tile_of,
                [&](auto buf, int t) {
                    tile_load_lds<T, D>(decltype(buf)::value ? v1s : v0s, rv, t * GQA_BN, L.w, L.lane);
                    gqa_fix_load(st, arow, rrow, t * GQA_BN, L);
                },
                [&](auto buf) {
                    constexpr int B_ = decltype(buf)::value;
                    gqa_fix_store(B_ ? ab1 : ab0, reinterpret_cast<float*>(B_ ? k1s : k0s), st, L, a_sh, r_sh);
                },
                [&](auto buf, int t, auto mask) {
                    constexpr int B_ = decltype(buf)::value;
                    gqa_band_tile<T, D, decltype(mask)::value>(B_ ? v1s : v0s,
                                                               reinterpret_cast<const float*>(B_ ? k1s : k0s),
                                                               B_ ? ab1 : ab0, t * GQA_BN, L, oacc, z);
                });
            // O = acc / Z' and log Z = A + R + ln Z' (the guard keeps Z' above e^-40).
            const float zt = pair_sum(z);
            row_scale = 1.0f / zt;
            lse_out = A + R + __log2f(zt) * LN2;
        } else {
            float m_run = NEG_BIG, l_run = 0.0f;
            run_slots(
            P, P + n_full, tile_of,
            [&](auto buf, int t) {
                constexpr int B_ = decltype(buf)::value;
                tile_load_lds<T, D>(B_ ? v1s : v0s, rv, t * GQA_BN, L.w, L.lane);
                // The tile's a values, then r over offsets m0 - n0 - 63 .. m0 - n0 + 127.
                float* ab = B_ ? ab1 : ab0;
                const int n0 = t * GQA_BN;
                for (int x = L.tid; x < GQA_BN + GQA_BAND; x += GQA_THREADS) {
                    float val;
                    if (x < GQA_BN) {
                        val = n0 + x < N ? arow[n0 + x] : -INFINITY;
                    } else {
                        const int delta = L.m0 - n0 - (GQA_BN - 1) + (x - GQA_BN);
                        val = (delta >= 0 && delta < N) ? rrow[delta] : -INFINITY;
                    }
                    ab[x] = val;
                }
            },
            [&](auto) {},
            [&](auto buf, int t, auto mask) {
                constexpr int B_ = decltype(buf)::value;
                const float* ab = B_ ? ab1 : ab0;
                gqa_fix_tile<T, D, decltype(mask)::value>(B_ ? v1s : v0s, ab, ab + GQA_BN, t * GQA_BN, L, oacc,
                                                          m_run, l_run);
            });
            const float l_tot = pair_sum(l_run);
            row_scale = 1.0f / l_tot;
            lse_out = (m_run + __log2f(l_tot)) * LN2;
        }
    }
    if (qq < N) {
        T* orow = reinterpret_cast<T*>(p.o) + qbase + (size_t)qq * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                st4<T>(orow + 32 * db + 8 * g + 4 * L.hf, oacc[db][4 * g] * row_scale,
                       oacc[db][4 * g + 1] * row_scale, oacc[db][4 * g + 2] * row_scale,
                       oacc[db][4 * g + 3] * row_scale);
        if (L.hf == 0) p.lse[row_base + qq] = lse_out;
    }
}

}  // namespace saf
