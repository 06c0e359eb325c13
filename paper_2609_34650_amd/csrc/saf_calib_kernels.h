// Calibration statistics of the ordinary heads (Section "Calibration and head
// selection"): the running mean attention, per-entry squared deviations and
// the entropy sum from which the variance score (Eq. variance-score) and the
// forward-KL score (Eq. forward-kl-score) follow, and the absolute-position
// and relative-distance marginals of the mean (Eq. fit-objective).  No
// per-input T x T matrix ever reaches memory: each workgroup keeps one
// 128 x 128 tile of the statistics in registers while it streams the
// calibration inputs of the call through it, recomputing that input's
// attention weights from Q, K and the forward's LSE.
//
// Accumulation (calib_accum_kernel): workgroup = (head h, query tile I, key
// tile J), 4 wavefronts.  Wavefront w owns the 32 keys J*128 + 32w .. +31
// (one per lane column c) and all 128 queries of the tile as four 32-row
// blocks, so each lane holds 64 entries of the tile.  For every input b the
// scores S = Q K^T come from the MFMA with Q rows as the A operand and K rows
// as the B operand (keys as columns), so a lane's accumulator entries sit in
// one key column: stores of the statistics are 128-byte row runs.  Per entry
// the weight p = exp2(S * log2(e)/sqrt(d) - LSE * log2(e)) updates the running
// mean and squared-deviation sum with Welford's recurrence (n = inputs seen
// so far, including this one):
//     delta = p - mean;  mean += delta / n;  m2 += delta * (p - mean),
// which stays accurate when the variance is small next to the mean, and the
// lane's entropy partial gathers p * log2(p).  Q and K tiles of the next input
// are copied into LDS (buffer loads straight to LDS) while this one is used.
// Tiles above the diagonal hold zeros (written on the first call only);
// diagonal tiles mask keys after the query, and a wavefront skips its row
// blocks that lie wholly above the diagonal.
//
// Finalisation (calib_final_kernel, calib_scores_kernel): one pass over the
// lower triangle of the mean and m2.  Thread j of a 256-column group sums, over
// a chunk of 256 rows, column j of the mean (eta_abs(j)), the diagonal
// i - k = j of the mean (eta_rel(j); consecutive threads read consecutive
// addresses of each row), m2 and mean * ln(mean); chunk partials are added
// atomically (float32 for the marginals, float64 for the two scalars).
#pragma once

#include "saf_common.h"

namespace saf {

constexpr int CAL_TILE = 128;     // queries and keys per workgroup tile
constexpr int CAL_THREADS = 256;
constexpr int CAL_FIN_COLS = 256;  // columns per finalisation workgroup
constexpr int CAL_FIN_ROWS = 256;  // rows per finalisation workgroup
// LSE stand-in for rows past T: every weight of such a row is exp2(-huge) = 0
// and its entropy term 0 * finite = 0.
constexpr float CAL_ROW_PAD = 1.0e30f;

struct CalibArgs {
    const void* q;      // [B, H, T, 64]
    const void* k;      // [B, H, T, 64]
    const float* lse;   // [B, H, T], natural log
    float* mean;        // [H, T, T]
    float* m2;          // [H, T, T]
    double* ent;        // [H]
    int B, H, T, n_seen, n_tiles;
    float scale_log2;   // log2(e) / sqrt(d)
};

struct CalibFinalArgs {
    const float* mean;
    const float* m2;
    const double* ent;
    float* eta_abs;     // [H, T]
    float* eta_rel;     // [H, T]
    float* s_var;       // [H]
    float* s_kl;        // [H]
    double* acc;        // [H, 2]: sum of m2, sum of mean * ln(mean)
    int H, T, n_total, n_cgroups, n_rchunks;
};

__global__ void calib_fill_kernel(float* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0.0f;
}
__global__ void calib_fill_kernel(double* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0.0;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
    return x;
}
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
    return x;
}

struct CalLane {
    int w, lane, c, hf;
    int row0, col0;  // first query / key of the tile
    int T;
};

// Stream inputs b of the call through one diagonal (MASK) or sub-diagonal tile.
template <typename T, bool MASK, typename Q0, typename Q1, typename K0, typename K1, typename LS>
__device__ __forceinline__ void calib_input(Q0 qa, Q1 qb, K0 ka, K1 kb, LS ls, int b, const CalibArgs& p,
                                            const CalLane& L, f32x16 (&mean)[4], f32x16 (&m2)[4], float& ent) {
    typedef typename Vec<T>::x8 frag;
    const T* kt = (L.w >> 1) ? kb : ka;
    frag kf[4];
#pragma unroll
    for (int dc = 0; dc < 4; ++dc) kf[dc] = ld_row<T>(kt, 32 * (L.w & 1) + L.c, 16 * dc + 8 * L.hf);
    const float rn = 1.0f / (float)(p.n_seen + b + 1);
    const float sl2 = p.scale_log2;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        if (MASK && rb < L.w) continue;  // wholly above the diagonal
        const T* qt = (rb >> 1) ? qb : qa;
        f32x16 s;
#pragma unroll
        for (int v = 0; v < 16; ++v) s[v] = 0.0f;
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) mma(s, ld_row<T>(qt, 32 * (rb & 1) + L.c, 16 * dc + 8 * L.hf), kf[dc]);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 l4 = *reinterpret_cast<const f32x4*>(ls + 32 * rb + 8 * g + 4 * L.hf);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int v = 4 * g + u;
                const float x = fmaf(s[v], sl2, -l4[u]);
                float pv = fast_exp2(x);
                // Diagonal tile: key 32w + c against query 32rb + 8g + 4hf + u.
                if (MASK && rb == L.w && L.c > 8 * g + 4 * L.hf + u) pv = 0.0f;
                ent = fmaf(pv, x, ent);
                const float d1 = pv - mean[rb][v];
                mean[rb][v] = fmaf(d1, rn, mean[rb][v]);
                m2[rb][v] = fmaf(d1, pv - mean[rb][v], m2[rb][v]);
            }
        }
    }
}

template <typename T>
__global__ __launch_bounds__(CAL_THREADS) __attribute__((amdgpu_waves_per_eu(2))) void calib_accum_kernel(
    CalibArgs p) {
    __shared__ __attribute__((aligned(16))) T q0a[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T q0b[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T k0a[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T k0b[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T q1a[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T q1b[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T k1a[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T k1b[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) float ls0[CAL_TILE];
    __shared__ __attribute__((aligned(16))) float ls1[CAL_TILE];

    const int nt2 = p.n_tiles * p.n_tiles;
    const int h = (int)(blockIdx.x / nt2);
    const int tile = (int)(blockIdx.x % nt2);
    const int I = tile / p.n_tiles;
    const int J = tile % p.n_tiles;
    const int tid = threadIdx.x;
    CalLane L;
    L.w = __builtin_amdgcn_readfirstlane(tid >> 6);
    L.lane = tid & 63;
    L.c = tid & 31;
    L.hf = (tid >> 5) & 1;
    L.row0 = I * CAL_TILE;
    L.col0 = J * CAL_TILE;
    L.T = p.T;
    const size_t plane = (size_t)h * p.T * p.T;
    float* __restrict__ Mg = p.mean + plane;
    float* __restrict__ M2g = p.m2 + plane;
    const int col = L.col0 + 32 * L.w + L.c;
    auto row_of = [&](int rb, int v) { return L.row0 + 32 * rb + 8 * (v >> 2) + 4 * L.hf + (v & 3); };

    f32x16 mean[4], m2[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            mean[rb][v] = 0.0f;
            m2[rb][v] = 0.0f;
        }
    auto store = [&]() {
        if (col >= L.T) return;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = row_of(rb, v);
                if (row < L.T) {
                    Mg[(size_t)row * L.T + col] = mean[rb][v];
                    M2g[(size_t)row * L.T + col] = m2[rb][v];
                }
            }
    };
    if (J > I) {  // above the diagonal: zeros, written once
        if (p.n_seen == 0) store();
        return;
    }
    if (p.n_seen > 0 && col < L.T) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = row_of(rb, v);
                if (row < L.T) {
                    mean[rb][v] = Mg[(size_t)row * L.T + col];
                    m2[rb][v] = M2g[(size_t)row * L.T + col];
                }
            }
    }

    float ent = 0.0f;
    auto issue = [&](auto buf, int b) {
        constexpr int B_ = decltype(buf)::value;
        const size_t slice = (size_t)(b * p.H + h) * p.T;
        const int row = L.row0 + tid;
        // The LSE load goes first so that waiting for it leaves the tile
        // copies in flight.
        const float lv = (tid < CAL_TILE && row < L.T) ? p.lse[slice + row] * LOG2E : CAL_ROW_PAD;
        const __amdgpu_buffer_rsrc_t rq =
            slice_rsrc<T>(reinterpret_cast<const T*>(p.q) + slice * HEAD_DIM, L.T);
        const __amdgpu_buffer_rsrc_t rk =
            slice_rsrc<T>(reinterpret_cast<const T*>(p.k) + slice * HEAD_DIM, L.T);
        tile_load_lds<T>(B_ ? q1a : q0a, rq, L.row0, L.w, L.lane);
        tile_load_lds<T>(B_ ? q1b : q0b, rq, L.row0 + TILE_ROWS, L.w, L.lane);
        tile_load_lds<T>(B_ ? k1a : k0a, rk, L.col0, L.w, L.lane);
        tile_load_lds<T>(B_ ? k1b : k0b, rk, L.col0 + TILE_ROWS, L.w, L.lane);
        if (tid < CAL_TILE) (B_ ? ls1 : ls0)[tid] = lv;
    };
    auto compute = [&](auto buf, int b, auto mask) {
        constexpr int B_ = decltype(buf)::value;
        constexpr bool M_ = decltype(mask)::value;
        if (B_)
            calib_input<T, M_>(q1a, q1b, k1a, k1b, ls1, b, p, L, mean, m2, ent);
        else
            calib_input<T, M_>(q0a, q0b, k0a, k0b, ls0, b, p, L, mean, m2, ent);
    };
    const bool diag = (I == J);
    const int P = diag ? (p.B + 1) & ~1 : 0;
    run_slots(
        P, diag ? P : p.B, [&](int i) { return i < p.B ? i : -1; }, issue, [&](auto) {}, compute);
    store();
    const float e = wave_sum(ent);
    if (L.lane == 0 && e != 0.0f) atomicAdd(p.ent + h, (double)e * (double)LN2);
}

__global__ __launch_bounds__(CAL_FIN_COLS) void calib_final_kernel(CalibFinalArgs p) {
    const int per_head = p.n_rchunks * p.n_cgroups;
    const int h = (int)(blockIdx.x / per_head);
    const int rem = (int)(blockIdx.x % per_head);
    const int i0 = (rem / p.n_cgroups) * CAL_FIN_ROWS;
    const int j = (rem % p.n_cgroups) * CAL_FIN_COLS + (int)threadIdx.x;
    const int j_first = (rem % p.n_cgroups) * CAL_FIN_COLS;
    if (j_first > i0 + CAL_FIN_ROWS - 1) return;  // the whole block lies above the diagonal
    const int T = p.T;
    const size_t plane = (size_t)h * T * T;
    const float* __restrict__ M = p.mean + plane;
    const float* __restrict__ M2 = p.m2 + plane;
    float col = 0.0f, dg = 0.0f, m2s = 0.0f, mlm = 0.0f;
    const int i_end = min(i0 + CAL_FIN_ROWS, T);
    if (j < T) {
        for (int i = max(i0, j); i < i_end; ++i) {
            const size_t rowoff = (size_t)i * T;
            const float mv = M[rowoff + j];
            col += mv;
            m2s += M2[rowoff + j];
            mlm += mv > 0.0f ? mv * __logf(mv) : 0.0f;
            dg += M[rowoff + (i - j)];
        }
        if (max(i0, j) < i_end) {
            atomicAdd(p.eta_abs + (size_t)h * T + j, col);
            atomicAdd(p.eta_rel + (size_t)h * T + j, dg);
        }
    }
    const double s0 = wave_sum((double)m2s);
    const double s1 = wave_sum((double)mlm);
    if ((threadIdx.x & 63) == 0) {
        atomicAdd(p.acc + 2 * h, s0);
        atomicAdd(p.acc + 2 * h + 1, s1);
    }
}

__global__ void calib_scores_kernel(CalibFinalArgs p) {
    const int h = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (h >= p.H) return;
    const double T = (double)p.T;
    const double n = (double)p.n_total;
    p.s_var[h] = p.n_total > 1 ? (float)(p.acc[2 * h] / ((n - 1.0) * T * T)) : __builtin_nanf("");
    p.s_kl[h] = (float)(p.ent[h] / (n * T) - p.acc[2 * h + 1] / T);
}

}  // namespace saf
