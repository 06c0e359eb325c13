// Compact fit of fixed patterns (Section "Fixed-pattern construction and
// fitting", Eq. fit-objective; the fitting step of Algorithm "calibration";
// Appendix "Compact fitting and storage").
//
// Targets: the mean attention of a head, its causal entries floored at 1e-9
// and each row renormalised, Pi(i, j) = max(A(i, j), floor) / s(i).  One pass
// gives the row sums s(i) (fit_rowsum_kernel, one wavefront per row); a second
// pass (fit_target_kernel) gives eta_abs (column sums of Pi), eta_rel (its
// diagonal sums) and sum Pi ln Pi, with the access pattern of the calibration
// finalisation: thread j of a 256-column group walks a chunk of 256 rows
// down column j and down diagonal i - k = j (both coalesced); chunk partials
// of the marginals are added atomically, the entropy partial goes to a slot of
// its own.
//
// Fitter: alpha = 0, rho(delta) = log max(eta_rel(delta) / (T - delta),
// floor), then Adam steps on Eq. fit-objective.  One step is three launches
// for all heads at once: the row normalisers log Z(i) (the forward's
// fixed_lse_kernel, with one batch element), the marginals of the fitted
// pattern (fit_marginals_kernel: column and diagonal sums of
// P(i, j) = exp(alpha(j) + rho(i - j) - log Z(i)), the same walk as above,
// one exponential per visited entry), and the update (fit_adam_kernel: the
// gradient (marginal - eta) / T, Adam's moments and step; it also clears the
// marginal sums for the next step).  fit_kl_kernel forms the acceptance KL,
// L + (1/T) sum Pi ln Pi with L = (1/T)(sum_i log Z(i) - eta_abs . alpha -
// eta_rel . rho), in float64.
#pragma once

#include "saf_common.h"

namespace saf {

constexpr int FIT_COLS = 256;  // columns per marginal workgroup
constexpr int FIT_ROWS = 256;  // rows per marginal workgroup
constexpr float FIT_ADAM_BETA1 = 0.9f;
constexpr float FIT_ADAM_BETA2 = 0.999f;
constexpr float FIT_ADAM_EPS = 1e-8f;

struct FitArgs {
    const float* mean;   // [H, T, T] (targets only)
    float* rowsum;       // [H, T]
    float* eta_abs;      // [H, T]
    float* eta_rel;      // [H, T]
    double* part;        // [H, n_rchunks * n_cgroups]: per block sum of Pi ln Pi
    double* neg_entropy; // [H]
    float* alpha;        // [H, T]
    float* rho;          // [H, T]
    float* m;            // [2, H, T]: Adam first moments of alpha, rho
    float* v;            // [2, H, T]: second moments
    float* col;          // [H, T]: column sums of the fitted pattern
    float* diag;         // [H, T]: its diagonal sums
    float* logz;         // [H, T]
    float* kl;           // [H]
    float floor_value, lr, bc1, bc2;  // bias corrections 1 - beta^t of this step
    int H, T, n_cgroups, n_rchunks;
};

__device__ __forceinline__ float fit_wave_sum(float x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
    return x;
}
__device__ __forceinline__ double fit_wave_sum(double x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
    return x;
}

// s(i) = sum_{j <= i} max(A(i, j), floor): one wavefront per row.
__global__ __launch_bounds__(256) void fit_rowsum_kernel(FitArgs p) {
    const int rows_per_head = (p.T + 3) / 4;
    const int h = (int)(blockIdx.x / rows_per_head);
    const int i = (int)(blockIdx.x % rows_per_head) * 4 + (int)(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (i >= p.T) return;
    const float* row = p.mean + ((size_t)h * p.T + i) * p.T;
    float s = 0.0f;
    for (int j = lane; j <= i; j += 64) s += fmaxf(row[j], p.floor_value);
    s = fit_wave_sum(s);
    if (lane == 0) p.rowsum[(size_t)h * p.T + i] = s;
}

// Block (head, 256-row chunk, 256-column group); see the header comment.
__global__ __launch_bounds__(FIT_COLS) void fit_target_kernel(FitArgs p) {
    __shared__ double red[FIT_COLS / 64];
    const int per_head = p.n_rchunks * p.n_cgroups;
    const int h = (int)(blockIdx.x / per_head);
    const int rem = (int)(blockIdx.x % per_head);
    const int i0 = (rem / p.n_cgroups) * FIT_ROWS;
    const int j_first = (rem % p.n_cgroups) * FIT_COLS;
    const int j = j_first + (int)threadIdx.x;
    if (j_first > i0 + FIT_ROWS - 1) {  // the whole block lies above the diagonal
        if (threadIdx.x == 0) p.part[blockIdx.x] = 0.0;
        return;
    }
    const int T = p.T;
    const float* __restrict__ M = p.mean + (size_t)h * T * T;
    const float* __restrict__ s = p.rowsum + (size_t)h * T;
    const float fl = p.floor_value;
    float colsum = 0.0f, dg = 0.0f, ent = 0.0f;
    const int i_end = min(i0 + FIT_ROWS, T);
    const int i_beg = max(i0, j);
    if (j < T && i_beg < i_end) {
        for (int i = i_beg; i < i_end; ++i) {
            const size_t rowoff = (size_t)i * T;
            const float inv = 1.0f / s[i];
            const float pc = fmaxf(M[rowoff + j], fl) * inv;
            colsum += pc;
            ent += pc * __logf(pc);
            dg += fmaxf(M[rowoff + (i - j)], fl) * inv;
        }
        atomicAdd(p.eta_abs + (size_t)h * T + j, colsum);
        atomicAdd(p.eta_rel + (size_t)h * T + j, dg);
    }
    const double e = fit_wave_sum((double)ent);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = e;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
#pragma unroll
        for (int w = 0; w < FIT_COLS / 64; ++w) t += red[w];
        p.part[blockIdx.x] = t;
    }
}

// neg_entropy[h] = sum of the head's block partials; one workgroup per head.
__global__ __launch_bounds__(256) void fit_entropy_kernel(FitArgs p) {
    __shared__ double red[4];
    const int h = (int)blockIdx.x;
    const int n = p.n_rchunks * p.n_cgroups;
    double t = 0.0;
    for (int k = (int)threadIdx.x; k < n; k += 256) t += p.part[(size_t)h * n + k];
    t = fit_wave_sum(t);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = t;
    __syncthreads();
    if (threadIdx.x == 0) p.neg_entropy[h] = (red[0] + red[1]) + (red[2] + red[3]);
}

// alpha = 0, rho = log max(eta_rel / (T - delta), floor); moments and
// marginal sums cleared.
__global__ void fit_init_kernel(FitArgs p) {
    const size_t n = (size_t)p.H * p.T;
    for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
        const int delta = (int)(k % p.T);
        p.alpha[k] = 0.0f;
        p.rho[k] = logf(fmaxf(p.eta_rel[k] / (float)(p.T - delta), p.floor_value));
        p.m[k] = 0.0f;
        p.m[n + k] = 0.0f;
        p.v[k] = 0.0f;
        p.v[n + k] = 0.0f;
        p.col[k] = 0.0f;
        p.diag[k] = 0.0f;
    }
}

// Column and diagonal sums of P(i, j) = exp(alpha(j) + rho(i - j) - log Z(i)).
// The block's rho and alpha values (offsets and keys i - j for its rows and
// columns: 511 of each) and its rows' log Z are staged in LDS first, so the
// walk reads consecutive LDS words across a wavefront.
//
// Factorised form (no exponential per entry): with A and R the maxima of
// alpha and rho over the values the block touches, P(i, j) = ea(j) er(i - j)
// w(i), ea = exp(alpha - A), er = exp(rho - R), w(i) = exp(A + R - log Z(i)),
// so column j's sum is ea(j) sum_i er(i - j) w(i) and diagonal d's sum is
// er(d) sum_i ea(i - d) w(i): two multiply-adds per row, with ea, er and w
// staged in LDS instead of the raw values (entries at negative positions are
// 0, which masks i < j).  Every term is at most 1, so ea and er cannot
// overflow; w can, when a row's log Z lies far below A + R, and a block with
// such a row (more than FAST_GUARD below) evaluates every entry exactly.
// In the factorised form each staged array is kept as four copies, copy m
// shifted by m entries, so that a lane's four consecutive entries (whose
// alignment is fixed per lane) are one aligned 16-byte read; the copies sit
// FIT_STAGE floats apart (a stride that keeps those reads free of bank
// conflicts).  The exact form uses copy 0 only.
constexpr int FIT_STAGE = 2 * FIT_COLS + 16;

__global__ __launch_bounds__(FIT_COLS) void fit_marginals_kernel(FitArgs p) {
    __shared__ __attribute__((aligned(16))) float rs[4 * FIT_STAGE];
    __shared__ __attribute__((aligned(16))) float as[4 * FIT_STAGE];
    __shared__ __attribute__((aligned(16))) float zs[FIT_ROWS];
    __shared__ float red[4];
    const int per_head = p.n_rchunks * p.n_cgroups;
    const int h = (int)(blockIdx.x / per_head);
    const int rem = (int)(blockIdx.x % per_head);
    const int i0 = (rem / p.n_cgroups) * FIT_ROWS;
    const int j_first = (rem % p.n_cgroups) * FIT_COLS;
    if (j_first > i0 + FIT_ROWS - 1) return;  // the whole block lies above the diagonal
    const int T = p.T;
    const int tid = (int)threadIdx.x;
    const int j = j_first + tid;
    const bool col_ok = j < T;
    const float* __restrict__ al = p.alpha + (size_t)h * T;
    const float* __restrict__ rh = p.rho + (size_t)h * T;
    const float* __restrict__ lz = p.logz + (size_t)h * T;
    // Staged index x holds position base + x, base = i0 - j_first - (FIT_COLS - 1).
    const int base = i0 - j_first - (FIT_COLS - 1);
    float rv[2], av[2];
    bool in[2];
    float am = col_ok ? al[j] : -INFINITY, rm = col_ok ? rh[j] : -INFINITY;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int q = base + tid + FIT_COLS * k;
        in[k] = q >= 0 && q < T;
        rv[k] = in[k] ? rh[q] : 0.0f;
        av[k] = in[k] ? al[q] : 0.0f;
        if (in[k]) {
            am = fmaxf(am, av[k]);
            rm = fmaxf(rm, rv[k]);
        }
    }
    const bool row_ok = i0 + tid < T;
    const float zv = row_ok ? lz[i0 + tid] : 0.0f;
    const float A = block_max(am, red);
    const float R = block_max(rm, red);
    const bool fast = __syncthreads_and(!row_ok || A + R - zv <= FAST_GUARD);
    const float aj = col_ok ? al[j] : 0.0f;  // column j's alpha
    const float rj = col_ok ? rh[j] : 0.0f;  // diagonal j's rho
    const int off = j_first - j + (FIT_COLS - 1);  // staged index of position i - j is (i - i0) + off
    const int r_beg = max(0, j - i0);               // rows i >= j
    float c = 0.0f, d = 0.0f;
    if (fast) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int x = tid + FIT_COLS * k;
            const float er = in[k] ? fast_exp2((rv[k] - R) * LOG2E) : 0.0f;
            const float ea = in[k] ? fast_exp2((av[k] - A) * LOG2E) : 0.0f;
#pragma unroll
            for (int m = 0; m < 4; ++m)
                if (x >= m) {
                    rs[m * FIT_STAGE + x - m] = er;
                    as[m * FIT_STAGE + x - m] = ea;
                }
        }
        zs[tid] = row_ok ? fast_exp2((A + R - zv) * LOG2E) : 0.0f;
        __syncthreads();
        if (!col_ok) return;
        // Rows from r_beg rounded down to a multiple of 4 (the rows below
        // r_beg meet staged zeros); rows past T have w = 0.  Entry r + off
        // of the staged arrays is entry r + off - m of copy m, m = off mod 4.
        const int m = off & 3;
        const float* rsm = rs + m * FIT_STAGE + off - m;
        const float* asm_ = as + m * FIT_STAGE + off - m;
        float c1 = 0.0f, d1 = 0.0f;
        for (int r = r_beg & ~3; r < FIT_ROWS; r += 4) {
            const f32x4 w4 = *reinterpret_cast<const f32x4*>(zs + r);
            const f32x4 e4 = *reinterpret_cast<const f32x4*>(rsm + r);
            const f32x4 a4 = *reinterpret_cast<const f32x4*>(asm_ + r);
            c = fmaf(e4[0], w4[0], c);
            d = fmaf(a4[0], w4[0], d);
            c1 = fmaf(e4[1], w4[1], c1);
            d1 = fmaf(a4[1], w4[1], d1);
            c = fmaf(e4[2], w4[2], c);
            d = fmaf(a4[2], w4[2], d);
            c1 = fmaf(e4[3], w4[3], c1);
            d1 = fmaf(a4[3], w4[3], d1);
        }
        c = (c + c1) * fast_exp2((aj - A) * LOG2E);
        d = (d + d1) * fast_exp2((rj - R) * LOG2E);
    } else {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            rs[tid + FIT_COLS * k] = rv[k];
            as[tid + FIT_COLS * k] = av[k];
        }
        zs[tid] = zv;
        __syncthreads();
        if (!col_ok) return;
        const int n_rows = min(FIT_ROWS, T - i0);
        const float aj2 = aj * LOG2E, rj2 = rj * LOG2E;
        float c1 = 0.0f, d1 = 0.0f;
        int r = r_beg;
        for (; r + 2 <= n_rows; r += 2) {
            const float z0 = zs[r] * LOG2E, z1 = zs[r + 1] * LOG2E;
            c += fast_exp2(fmaf(rs[r + off], LOG2E, aj2 - z0));
            c1 += fast_exp2(fmaf(rs[r + 1 + off], LOG2E, aj2 - z1));
            d += fast_exp2(fmaf(as[r + off], LOG2E, rj2 - z0));
            d1 += fast_exp2(fmaf(as[r + 1 + off], LOG2E, rj2 - z1));
        }
        if (r < n_rows) {
            const float z0 = zs[r] * LOG2E;
            c += fast_exp2(fmaf(rs[r + off], LOG2E, aj2 - z0));
            d += fast_exp2(fmaf(as[r + off], LOG2E, rj2 - z0));
        }
        c += c1;
        d += d1;
    }
    if (r_beg < min(FIT_ROWS, T - i0)) {
        atomicAdd(p.col + (size_t)h * T + j, c);
        atomicAdd(p.diag + (size_t)h * T + j, d);
    }
}

// One Adam step on alpha and rho; clears the marginal sums it read.
__global__ void fit_adam_kernel(FitArgs p) {
    const size_t n = (size_t)p.H * p.T;
    const float invT = 1.0f / (float)p.T;
    for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
        const float g0 = (p.col[k] - p.eta_abs[k]) * invT;
        const float g1 = (p.diag[k] - p.eta_rel[k]) * invT;
        p.col[k] = 0.0f;
        p.diag[k] = 0.0f;
        float* th[2] = {p.alpha, p.rho};
        const float g[2] = {g0, g1};
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const size_t at = (size_t)q * n + k;
            const float mq = FIT_ADAM_BETA1 * p.m[at] + (1.0f - FIT_ADAM_BETA1) * g[q];
            const float vq = FIT_ADAM_BETA2 * p.v[at] + (1.0f - FIT_ADAM_BETA2) * g[q] * g[q];
            p.m[at] = mq;
            p.v[at] = vq;
            const float mhat = mq / p.bc1;
            const float vhat = vq / p.bc2;
            th[q][k] -= p.lr * mhat / (sqrtf(vhat) + FIT_ADAM_EPS);
        }
    }
}

// kl[h] = (sum_i log Z(i) - eta_abs . alpha - eta_rel . rho + sum Pi ln Pi) / T.
__global__ __launch_bounds__(256) void fit_kl_kernel(FitArgs p) {
    __shared__ double red[4];
    const int h = (int)blockIdx.x;
    const size_t base = (size_t)h * p.T;
    double t = 0.0;
    for (int k = (int)threadIdx.x; k < p.T; k += 256)
        t += (double)p.logz[base + k] - (double)p.eta_abs[base + k] * p.alpha[base + k] -
             (double)p.eta_rel[base + k] * p.rho[base + k];
    t = fit_wave_sum(t);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = t;
    __syncthreads();
    if (threadIdx.x == 0)
        p.kl[h] = (float)(((red[0] + red[1]) + (red[2] + red[3]) + p.neg_entropy[h]) / (double)p.T);
}

__global__ void fit_fill_kernel(float* q, size_t n) {
    for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x)
        q[k] = 0.0f;
}

}  // namespace saf
