// Calibration statistics of the ordinary heads (Section "Calibration and head
// selection"): the running mean attention, the squared deviations and the
// entropy sum from which the variance score (Eq. variance-score) and the
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
// one key column: loads and stores of the statistics are 128-byte row runs.
// Per entry the weight p = exp(S / sqrt(d) - LSE) updates the running mean
// with Welford's recurrence (n = inputs seen so far, including this one):
//     delta = p - mean;  mean += delta / n;  inc += delta * (p - mean),
// where inc, the growth of the entry's sum of squared deviations over this
// call, depends only on the running mean (no cancellation when the variance
// is small next to the mean).  The call adds inc to the per-entry sums when
// the caller keeps them, and its total to the head's scalar sum, which is
// all the variance score needs.  The lane's entropy partial gathers
// p * ln(p).  Q and K tiles of the next input are copied into LDS (buffer
// loads straight to LDS) while this one is used.  Tiles above the diagonal
// hold zeros (written on the first call only); diagonal tiles mask keys after
// the query (a wavefront skips its row blocks that lie wholly above the
// diagonal), and the last row of tiles masks rows past T.
//
// Each tile's entropy and squared-deviation sums live in a slot of its own in
// the state (float64), so no two workgroups ever write the same address.
//
// Finalisation (calib_final_kernel, calib_scores_kernel): one pass over the
// lower triangle of the mean.  Thread j of a 256-column group sums, over a
// chunk of 256 rows, column j (eta_abs(j)), the diagonal i - k = j
// (eta_rel(j); consecutive threads read consecutive addresses of each row) and
// mean * ln(mean).  Chunk partials of the marginals are added atomically in
// float32 (at most T/256 adds per address); the block's mean * ln(mean) sum
// goes to a slot of its own; one workgroup per head then sums the slots.
#pragma once

#include "saf_common.h"

namespace saf {

constexpr int CAL_TILE = 128;     // queries and keys per workgroup tile
constexpr int CAL_THREADS = 256;
constexpr int CAL_FIN_COLS = 256;  // columns per finalisation workgroup
constexpr int CAL_FIN_ROWS = 256;  // rows per finalisation workgroup

struct CalibArgs {
    const void* q;      // [B, H, T, 64]
    const void* k;      // [B, H, T, 64]
    const float* lse;   // [B, H, T], natural log
    float* mean;        // [H, T, T]
    float* m2;          // [H, T, T] or null
    double* stats;      // [H, n_tiles, n_tiles, 2]: per tile, sum of A ln A and of squared deviations
    int B, H, T, n_seen, n_tiles;
    float scale;        // 1 / sqrt(d)
};

struct CalibFinalArgs {
    const float* mean;
    const double* stats;  // as in CalibArgs
    float* eta_abs;       // [H, T]
    float* eta_rel;       // [H, T]
    float* s_var;         // [H]
    float* s_kl;          // [H]
    double* part;         // [H, n_rchunks, n_cgroups]: sum of mean * ln(mean) per block
    int H, T, n_total, n_tiles, n_cgroups, n_rchunks;
};

__global__ void calib_fill_kernel(float* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0.0f;
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

// Fold input b into the tile.  ls holds the input's LSE rows (natural log;
// 0 past T).  MASK: the tile needs per-entry checks -- keys after the query on
// a diagonal tile, rows at or past T (rows_valid < 128) on the last row of
// tiles.
template <typename T, bool MASK, bool M2, typename Q0, typename Q1, typename K0, typename K1, typename LS,
          typename INC>
__device__ __forceinline__ void calib_input(Q0 qa, Q1 qb, K0 ka, K1 kb, LS ls, int b, const CalibArgs& p,
                                            const CalLane& L, bool diag, int rows_valid, f32x16 (&mean)[4],
                                            INC& inc, float& inc_s, float& ent) {
    const T* kt = (L.w >> 1) ? kb : ka;
    const float rn = 1.0f / (float)(p.n_seen + b + 1);
    const float scale = p.scale;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        if (MASK && diag && rb < L.w) continue;  // wholly above the diagonal
        const T* qt = (rb >> 1) ? qb : qa;
        f32x16 s;
#pragma unroll
        for (int v = 0; v < 16; ++v) s[v] = 0.0f;
        // K's fragments are read again for every row block (the kernel is
        // bound by the state traffic, not by LDS), so they do not hold 16
        // registers across the whole input.
#pragma unroll
        for (int dc = 0; dc < 4; ++dc)
            mma(s, ld_row<T>(qt, 32 * (rb & 1) + L.c, 16 * dc + 8 * L.hf),
                ld_row<T>(kt, 32 * (L.w & 1) + L.c, 16 * dc + 8 * L.hf));
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 l4 = *reinterpret_cast<const f32x4*>(ls + 32 * rb + 8 * g + 4 * L.hf);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int v = 4 * g + u;
                const float x = fmaf(s[v], scale, -l4[u]);  // ln p
                float pv = fast_exp2(x * LOG2E);
                if (MASK) {
                    // Entry (query 32rb + 8g + 4hf + u, key 32w + c) of the tile.
                    const int r = 32 * rb + 8 * g + 4 * L.hf + u;
                    if ((diag && 32 * L.w + L.c > r) || r >= rows_valid) pv = 0.0f;
                }
                ent = fmaf(pv, x, ent);
                const float d1 = pv - mean[rb][v];
                mean[rb][v] = fmaf(d1, rn, mean[rb][v]);
                if constexpr (M2)
                    inc[rb][v] = fmaf(d1, pv - mean[rb][v], inc[rb][v]);
                else
                    inc_s = fmaf(d1, pv - mean[rb][v], inc_s);
            }
        }
    }
}

template <typename T, bool M2>
__global__ __launch_bounds__(CAL_THREADS) __attribute__((amdgpu_waves_per_eu(M2 ? 2 : 3))) void calib_accum_kernel(
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
    __shared__ float red[8];

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
    // Statistics of the tile: a wavefront-uniform base (the tile's first row)
    // plus a 32-bit per-lane offset; the row step of entry (rb, v) is a
    // uniform multiple of T.
    const size_t tile_base = (size_t)h * p.T * p.T + (size_t)L.row0 * p.T;
    float* __restrict__ Mg = p.mean + tile_base;
    float* __restrict__ M2g = M2 ? p.m2 + tile_base : nullptr;
    const int col = L.col0 + 32 * L.w + L.c;
    auto row_of = [&](int rb, int v) { return L.row0 + 32 * rb + 8 * (v >> 2) + 4 * L.hf + (v & 3); };
    auto row_step = [&](int rb, int v) { return (32 * rb + 8 * (v >> 2) + (v & 3)) * L.T; };
    // A fresh copy of the lane offset for each pass over the tile, so that
    // the compiler does not keep the first pass's addresses live to the last.
    auto lane_off = [&]() {
        int o = 4 * L.hf * L.T + col;
        asm volatile("" : "+v"(o));
        return o;
    };

    // Per-entry increments of the squared deviations only when they are
    // kept; otherwise one running sum per lane.
    f32x16 mean[4], inc[M2 ? 4 : 1];
    float inc_s = 0.0f;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            mean[rb][v] = 0.0f;
            if constexpr (M2) inc[rb][v] = 0.0f;
        }
    double* slot = p.stats + 2 * (size_t)blockIdx.x;
    const bool diag = (I == J);
    const int rows_valid = min(CAL_TILE, L.T - L.row0);
    if (J > I) {  // above the diagonal: zeros, written once
        if (p.n_seen == 0 && tid < 2) slot[tid] = 0.0;
        if (p.n_seen == 0 && col < L.T) {
            const int lo = lane_off();
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    if (row_of(rb, v) < L.T) {
                        Mg[lo + row_step(rb, v)] = 0.0f;
                        if (M2g) M2g[lo + row_step(rb, v)] = 0.0f;
                    }
                }
        }
        return;
    }
    if (p.n_seen > 0 && col < L.T) {
        const int lo = lane_off();
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                if (row_of(rb, v) < L.T) mean[rb][v] = Mg[lo + row_step(rb, v)];
    }

    float ent = 0.0f;
    // Copies of input b: Q rows and K rows of the tile into column-slab tiles,
    // its LSE rows into a float array (rows past T arrive as 0 and are masked).
    auto issue = [&](auto buf, int b) {
        constexpr int B_ = decltype(buf)::value;
        const size_t slice = (size_t)(b * p.H + h) * p.T;
        const __amdgpu_buffer_rsrc_t rq =
            slice_rsrc<T>(reinterpret_cast<const T*>(p.q) + slice * HEAD_DIM, L.T);
        const __amdgpu_buffer_rsrc_t rk =
            slice_rsrc<T>(reinterpret_cast<const T*>(p.k) + slice * HEAD_DIM, L.T);
        tile_load_lds<T>(B_ ? q1a : q0a, rq, L.row0, L.w, L.lane);
        tile_load_lds<T>(B_ ? q1b : q0b, rq, L.row0 + TILE_ROWS, L.w, L.lane);
        tile_load_lds<T>(B_ ? k1a : k0a, rk, L.col0, L.w, L.lane);
        tile_load_lds<T>(B_ ? k1b : k0b, rk, L.col0 + TILE_ROWS, L.w, L.lane);
        if (L.w < 2) {
            const __amdgpu_buffer_rsrc_t rl =
                __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.lse + slice), (short)0, L.T * 4, 0x00020000);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (lds_void*)((B_ ? ls1 : ls0) + 64 * L.w), 4,
                                                     (L.row0 + 64 * L.w + L.lane) * 4, 0, 0, 0);
        }
    };
    const bool masked = diag || rows_valid < CAL_TILE;
    if constexpr (M2) {
        // Per-entry increments take 64 more registers: two workgroups per CU,
        // so the inputs are double-buffered (one loads while one is folded in).
        auto compute = [&](auto buf, int b, auto mask) {
            constexpr int B_ = decltype(buf)::value;
            constexpr bool M_ = decltype(mask)::value;
            if (B_)
                calib_input<T, M_, M2>(q1a, q1b, k1a, k1b, ls1, b, p, L, diag, rows_valid, mean, inc, inc_s, ent);
            else
                calib_input<T, M_, M2>(q0a, q0b, k0a, k0b, ls0, b, p, L, diag, rows_valid, mean, inc, inc_s, ent);
        };
        const int P = masked ? (p.B + 1) & ~1 : 0;
        run_slots(P, P ? P : p.B, [&](int i) { return i < p.B ? i : -1; }, issue, [&](auto) {}, compute);
    } else {
        // One buffer of input tiles (35 KB of LDS for bf16), so that three
        // workgroups fit on a CU: each input is loaded, then folded in.
        for (int b = 0; b < p.B; ++b) {
            issue(Buf0{}, b);
            __syncthreads();
            if (masked)
                calib_input<T, true, M2>(q0a, q0b, k0a, k0b, ls0, b, p, L, diag, rows_valid, mean, inc, inc_s, ent);
            else
                calib_input<T, false, M2>(q0a, q0b, k0a, k0b, ls0, b, p, L, diag, rows_valid, mean, inc, inc_s,
                                          ent);
            __syncthreads();
        }
    }

    float inc_sum = M2 ? 0.0f : inc_s;
    if (col < L.T) {
        const int lo = lane_off();
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                if (row_of(rb, v) < L.T) {
                    const int at = lo + row_step(rb, v);
                    Mg[at] = mean[rb][v];
                    if constexpr (M2) {
                        M2g[at] = p.n_seen > 0 ? M2g[at] + inc[rb][v] : inc[rb][v];
                        inc_sum += inc[rb][v];
                    }
                }
            }
    }
    // The tile's two sums go to its own slot of the state: no atomics, and
    // the result does not depend on the order in which workgroups finish.
    const float e = wave_sum(ent);
    const float q = wave_sum(inc_sum);
    if (L.lane == 0) {
        red[2 * L.w] = e;
        red[2 * L.w + 1] = q;
    }
    __syncthreads();
    if (tid < 2) {
        const float t = red[tid] + red[tid + 2] + red[tid + 4] + red[tid + 6];
        const double add = (double)t;
        slot[tid] = p.n_seen > 0 ? slot[tid] + add : add;
    }
}

__global__ __launch_bounds__(CAL_FIN_COLS) void calib_final_kernel(CalibFinalArgs p) {
    __shared__ double red[CAL_FIN_COLS / 64];
    const int per_head = p.n_rchunks * p.n_cgroups;
    const int h = (int)(blockIdx.x / per_head);
    const int rem = (int)(blockIdx.x % per_head);
    const int i0 = (rem / p.n_cgroups) * CAL_FIN_ROWS;
    const int j_first = (rem % p.n_cgroups) * CAL_FIN_COLS;
    const int j = j_first + (int)threadIdx.x;
    if (j_first > i0 + CAL_FIN_ROWS - 1) {  // the whole block lies above the diagonal
        if (threadIdx.x == 0) p.part[blockIdx.x] = 0.0;
        return;
    }
    const int T = p.T;
    const float* __restrict__ M = p.mean + (size_t)h * T * T;
    float col = 0.0f, dg = 0.0f, mlm = 0.0f;
    const int i_end = min(i0 + CAL_FIN_ROWS, T);
    const int i_beg = max(i0, j);
    if (j < T && i_beg < i_end) {
        // Eight rows per step: sixteen independent loads in flight per thread.
        int i = i_beg;
        for (; i + 8 <= i_end; i += 8) {
            float mv[8], dv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const size_t rowoff = (size_t)(i + u) * T;
                mv[u] = M[rowoff + j];
                dv[u] = M[rowoff + (i + u - j)];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                col += mv[u];
                dg += dv[u];
                mlm += mv[u] > 0.0f ? mv[u] * __logf(mv[u]) : 0.0f;
            }
        }
        for (; i < i_end; ++i) {
            const size_t rowoff = (size_t)i * T;
            const float mv = M[rowoff + j];
            col += mv;
            dg += M[rowoff + (i - j)];
            mlm += mv > 0.0f ? mv * __logf(mv) : 0.0f;
        }
        atomicAdd(p.eta_abs + (size_t)h * T + j, col);
        atomicAdd(p.eta_rel + (size_t)h * T + j, dg);
    }
    const double s1 = wave_sum((double)mlm);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s1;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
#pragma unroll
        for (int w = 0; w < CAL_FIN_COLS / 64; ++w) t += red[w];
        p.part[blockIdx.x] = t;
    }
}

// One workgroup per head: sums the per-tile slots of the state and the
// finalisation blocks' partials, then forms the two scores.
__global__ __launch_bounds__(256) void calib_scores_kernel(CalibFinalArgs p) {
    __shared__ double red[3][4];
    const int h = (int)blockIdx.x;
    const int n_slots = p.n_tiles * p.n_tiles;
    const int n_parts = p.n_rchunks * p.n_cgroups;
    const double* st = p.stats + 2 * (size_t)h * n_slots;
    const double* pt = p.part + (size_t)h * n_parts;
    double e = 0.0, q = 0.0, m = 0.0;
    for (int i = (int)threadIdx.x; i < n_slots; i += 256) {
        e += st[2 * i];
        q += st[2 * i + 1];
    }
    for (int i = (int)threadIdx.x; i < n_parts; i += 256) m += pt[i];
    e = wave_sum(e);
    q = wave_sum(q);
    m = wave_sum(m);
    if ((threadIdx.x & 63) == 0) {
        red[0][threadIdx.x >> 6] = e;
        red[1][threadIdx.x >> 6] = q;
        red[2][threadIdx.x >> 6] = m;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const double E = red[0][0] + red[0][1] + red[0][2] + red[0][3];
        const double Qs = red[1][0] + red[1][1] + red[1][2] + red[1][3];
        const double Ms = red[2][0] + red[2][1] + red[2][2] + red[2][3];
        const double T = (double)p.T;
        const double n = (double)p.n_total;
        p.s_var[h] = p.n_total > 1 ? (float)(Qs / ((n - 1.0) * T * T)) : __builtin_nanf("");
        p.s_kl[h] = (float)(E / (n * T) - Ms / T);
    }
}

}  // namespace saf
