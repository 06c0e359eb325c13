// Gradients of trainable fixed patterns (Appendix "Pattern content and
// trainability": the variant that keeps optimising alpha and rho after
// replacement).  For a fixed head, with logits L(i, j) = a[j] + r[i - j],
// P = softmax_causal(L), O = P V and the loss sum(O * dO):
//     dP = dO V^T,  D_i = rowsum(dO * O)_i,  dL = P * (dP - D),
//     da[j] = sum_i dL(i, j),  dr[delta] = sum_{i - j = delta} dL(i, j),
// each summed over the batch (a and r are shared by every batch element).
//
// Workgroup = (batch b, fixed head, block of 128 keys, chunk of query
// tiles), 4 wavefronts of 32 keys (one per lane column c), streaming the
// chunk's query tiles of 64 rows (the block's tiles run from its first key to
// N; cutting them into chunks of at most 16 tiles keeps the workgroups of the
// first key blocks from setting the kernel's duration alone).  dP comes from the MFMA with dO rows as the A
// operand (from LDS) and the wavefront's V rows as the B operand (registers),
// so a lane's accumulator entries are 16 queries of its key: dL summed down
// the lane is the key's share of da.  P is recomputed per entry as
// exp(a[j] + r[i - j] - log Z(i)) with log Z from the forward's LSE and the
// offsets' r values from an LDS band copied per tile.  dr needs sums along
// the diagonals of each 32 x 32 block of dL: a wavefront writes the block
// into its own LDS scratch skewed so that each scratch row holds (parts of)
// two diagonals (rows padded to 36 floats), sums the rows with 16-byte reads
// and adds the diagonal sums into the wavefront's ring of 256 floats indexed
// by offset mod 256 (distinct lanes, distinct slots: no atomics; LDS atomic
// adds per entry were six times slower than the whole rest of the kernel).  Tile t touches offsets 64t - 127 .. 64t + 63, so once tile t is
// done the offsets below 64(t+1) - 127 are final; the next tile stores their
// sum over the four rings into the workgroup's own row of partial sums and
// clears the slots, which the tile after it is the first to reuse.  Plain stores, no global atomics:
// every workgroup of a head reaches the same offsets at about the same time,
// and atomic adds on one address serialise.  A second kernel sums the partial
// rows over batch elements and key blocks (and the da partials over batch
// elements).  The dO tile, the tile's LSE and D rows and the r band are
// copied by buffer loads straight to LDS (rows or offsets outside 0 .. N-1
// arrive as 0 and are masked), double-buffered over tiles.  A second kernel
// sums the partial rows (and writes the ordinary heads' zeros).
#pragma once

#include "saf_common.h"

namespace saf {

constexpr int PAT_BN = 128;      // keys per workgroup
constexpr int PAT_BM = TILE_ROWS;  // queries per tile
constexpr int PAT_THREADS = 256;
constexpr int PAT_BAND = 192;    // r entries per tile (offsets 64t - 127 .. 64t + 64)
constexpr int PAT_RING = 256;    // dr ring slots
constexpr int PAT_SCR = 36;      // scratch row stride (floats): 16-byte aligned rows, conflict-free skewed writes
static_assert(PAT_BM + PAT_BN - 1 <= PAT_BAND, "a tile's offsets fit in the band");
static_assert(PAT_BAND + PAT_BM <= PAT_RING, "live offsets never share a ring slot");

struct PatArgs {
    const void* v;
    const void* dO;
    const float* lse;
    const float* dsum;   // D, [B, H, N]
    const float* a;
    const float* r;
    float* da;           // [H, N]
    float* dr;           // [H, N]
    float* da_part;      // [B, n_fixed, n_chunks, N]: per chunk, its key block's keys
    float* dr_part;      // [B, n_fixed, n_kblocks, n_chunks, part_len]: per chunk, its offsets
    int B, H, N, ld_prior, n_fixed, n_kblocks;
    int chunk_tiles;     // query tiles per chunk
    int n_chunks;        // chunks of the longest key block (the grid's y extent)
    int part_len;        // 64 * chunk_tiles + 127: offsets one chunk touches
    unsigned char heads[64];  // the fixed heads
    unsigned char fixed_index[64];  // head -> its index in heads, or 255 for an ordinary head
};

// Query tiles of key block J, and its chunks.
__host__ __device__ inline int pat_tiles(int J, int N) { return (N - J * PAT_BN + PAT_BM - 1) / PAT_BM; }
__host__ __device__ inline int pat_chunks(int J, int N, int chunk_tiles) {
    return (pat_tiles(J, N) + chunk_tiles - 1) / chunk_tiles;
}

// One query tile t (queries q0 .. q0+63, q0 = k0 + 64 t) against the
// wavefront's 32 keys.  MASK: the tile meets the diagonal or runs past N.
// scr: the wavefront's 32 x PAT_SCR scratch; ring: its 256 offset slots.
//
// Each 32 x 32 block of dL is written into the scratch skewed: entry (row r,
// column c) goes to scratch row (r - c) mod 32, column c, so scratch row k
// holds diagonal k in its columns c < 32 - k and diagonal k - 32 in the
// rest.  Lane k (and lane k + 32, for the other half of the columns) then
// reads its row with four 16-byte loads and splits the sum at column 32 - k.
// w_lo[e]: 1 if column 16 (lane / 32) + e of scratch row lane % 32 holds
// the row's first diagonal, else 0 (fixed per lane).
template <typename T, bool MASK>
__device__ __forceinline__ void pat_tile(const T* gt, const float* rows, const float* band, float* scr, float* ring,
                                         int t, int q0, int k0, int w, int c, int hf, int lane, int N,
                                         const typename Vec<T>::x8 (&vf)[4], const float (&w_lo)[16], float a_key,
                                         float& da_acc) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        // Rows of this block all precede the wavefront's first key.
        if (MASK && 2 * t + rb < w) continue;
        // dP - D in one go: the accumulator starts at -D of its rows.
        f32x16 dp;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 d4 = *reinterpret_cast<const f32x4*>(rows + PAT_BM + 32 * rb + 8 * g + 4 * hf);
#pragma unroll
            for (int u = 0; u < 4; ++u) dp[4 * g + u] = -d4[u];
        }
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) mma(dp, ld_row<T>(gt, 32 * rb + c, 16 * dc + 8 * hf), vf[dc]);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 l4 = *reinterpret_cast<const f32x4*>(rows + 32 * rb + 8 * g + 4 * hf);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int v = 4 * g + u;
                const int r = 8 * g + 4 * hf + u;                  // row within the block
                const int bi = 32 * rb + r - 32 * w - c + (PAT_BN - 1);  // band index of i - j
                float pv = fast_exp2((a_key - l4[u] + band[bi]) * LOG2E);
                if (MASK && (32 * rb + r < 32 * w + c - 64 * t || q0 + 32 * rb + r >= N)) pv = 0.0f;
                const float dl = pv * dp[v];
                da_acc += dl;
                scr[((r - c) & 31) * PAT_SCR + c] = dl;
            }
        }
        // The wavefront's own LDS writes above are visible to its later reads.
        const int k = lane & 31;
        const int half = lane >> 5;  // columns 16 half .. 16 half + 15
        const float* src = scr + k * PAT_SCR + 16 * half;
        float s_lo = 0.0f, s_all = 0.0f;  // diagonal k; both diagonals
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const f32x4 x = *reinterpret_cast<const f32x4*>(src + 4 * q);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                s_lo = fmaf(x[e], w_lo[4 * q + e], s_lo);
                s_all += x[e];
            }
        }
        float s_hi = s_all - s_lo;  // diagonal k - 32
        s_lo += __shfl_xor(s_lo, 32);
        s_hi += __shfl_xor(s_hi, 32);
        // Lane k adds diagonal k, lane k + 32 diagonal k - 32 (k >= 1).
        const int d = half ? k - 32 : k;
        const int delta = 64 * t + 32 * rb - 32 * w + d;
        if ((half == 0 || k > 0) && delta >= 0) ring[delta & (PAT_RING - 1)] += half ? s_hi : s_lo;
    }
}

template <typename T>
__global__ __launch_bounds__(PAT_THREADS) void bwd_pattern_kernel(PatArgs p) {
    __shared__ __attribute__((aligned(16))) T g0[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) T g1[tile_elems<T>()];
    __shared__ __attribute__((aligned(16))) float rows0[2 * PAT_BM];  // LSE, then D
    __shared__ __attribute__((aligned(16))) float rows1[2 * PAT_BM];
    __shared__ __attribute__((aligned(16))) float band0[PAT_BAND];
    __shared__ __attribute__((aligned(16))) float band1[PAT_BAND];
    __shared__ __attribute__((aligned(16))) float scratch[4][32 * PAT_SCR];
    __shared__ float ring[4][PAT_RING];

    const int per_block = p.B * p.n_fixed;
    const int kblk = (int)(blockIdx.x / per_block);  // ascending: longest first
    const int rem = (int)(blockIdx.x % per_block);
    const int chunk = (int)blockIdx.y;
    const int N = p.N;
    const int n_tiles = pat_tiles(kblk, N);
    const int t0 = chunk * p.chunk_tiles;  // this chunk's tiles: t0 .. t1-1
    if (t0 >= n_tiles) return;             // the key block ends before this chunk
    const int t1 = min(t0 + p.chunk_tiles, n_tiles);
    const int b = rem / p.n_fixed;
    const int hidx = rem % p.n_fixed;
    const int h = p.heads[hidx];
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int c = tid & 31;
    const int hf = (tid >> 5) & 1;
    const int k0 = kblk * PAT_BN;
    const int key = k0 + 32 * w + c;
    const size_t slice = (size_t)(b * p.H + h) * N;
    const T* V = reinterpret_cast<const T*>(p.v) + slice * HEAD_DIM;
    const float* arow = p.a + (size_t)h * p.ld_prior;
    const float* rrow = p.r + (size_t)h * p.ld_prior;

    for (int i = tid; i < 4 * PAT_RING; i += PAT_THREADS) ring[i / PAT_RING][i % PAT_RING] = 0.0f;
    typedef typename Vec<T>::x8 frag;
    frag vf[4];
#pragma unroll
    for (int dc = 0; dc < 4; ++dc) vf[dc] = key < N ? ld8<T>(V + (size_t)key * HEAD_DIM + 16 * dc + 8 * hf) : zero8<T>();
    const float a_key = key < N ? arow[key] : -INFINITY;
    float w_lo[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) w_lo[e] = 16 * (lane >> 5) + e < 32 - (lane & 31) ? 1.0f : 0.0f;

    const __amdgpu_buffer_rsrc_t rg = slice_rsrc<T>(reinterpret_cast<const T*>(p.dO) + slice * HEAD_DIM, N);
    const __amdgpu_buffer_rsrc_t rl =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.lse + slice), (short)0, N * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t rd =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.dsum + slice), (short)0, N * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t rr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(rrow), (short)0, N * 4, 0x00020000);

    // Masked tiles: the two that meet the diagonal (first chunk only) and a
    // last tile that runs past N (last chunk only).
    const int m_lo = t0 == 0 ? min(PAT_BN / PAT_BM, t1) : 0;
    const bool ragged_end = t1 == n_tiles && (N - k0) % PAT_BM != 0 && t1 - 1 >= t0 + m_lo;
    float da_acc = 0.0f;
    auto issue = [&](auto buf, int t) {
        constexpr int B_ = decltype(buf)::value;
        const int q0 = k0 + PAT_BM * t;
        tile_load_lds<T>(B_ ? g1 : g0, rg, q0, w, lane);
        // Five 64-entry copies: LSE rows, D rows, three parts of the r band
        // (offsets q0 - k0 - 127 .. q0 - k0 + 64; negative ones arrive as 0).
        float* rows = B_ ? rows1 : rows0;
        float* band = B_ ? band1 : band0;
        if (w == 0) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (lds_void*)rows, 4, (q0 + lane) * 4, 0, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, (lds_void*)(rows + PAT_BM), 4, (q0 + lane) * 4, 0, 0, 0);
        } else {
            const int off = q0 - k0 - (PAT_BN - 1) + 64 * (w - 1) + lane;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rr, (lds_void*)(band + 64 * (w - 1)), 4, off * 4, 0, 0, 0);
        }
    };
    const size_t part = (size_t)(b * p.n_fixed + hidx);
    // This chunk's offsets start at 64 t0 - 127 (entry 0 of its row).
    const int delta0 = PAT_BM * t0 - (PAT_BN - 1);
    float* dr_row = p.dr_part + ((part * p.n_kblocks + kblk) * p.n_chunks + chunk) * (size_t)p.part_len;
    const int max_delta = N - 1 - k0;
    auto flush = [&](int lo, int count) {
        // Offsets lo .. lo+count-1 are final: store them and clear their slots.
        if (tid < count) {
            const int delta = lo + tid;
            if (delta >= 0 && delta <= max_delta) {
                const int s = delta & (PAT_RING - 1);
                dr_row[delta - delta0] = (ring[0][s] + ring[1][s]) + (ring[2][s] + ring[3][s]);
                ring[0][s] = 0.0f;
                ring[1][s] = 0.0f;
                ring[2][s] = 0.0f;
                ring[3][s] = 0.0f;
            }
        }
    };
    auto compute = [&](auto buf, int t, auto mask) {
        constexpr int B_ = decltype(buf)::value;
        if (t > t0) flush(PAT_BM * t - (PAT_BM + PAT_BN - 1), PAT_BM);  // final after tile t-1
        pat_tile<T, decltype(mask)::value>(B_ ? g1 : g0, B_ ? rows1 : rows0, B_ ? band1 : band0, scratch[w],
                                           ring[w], t, k0 + PAT_BM * t, k0, w, c, hf, lane, N, vf, w_lo, a_key, da_acc);
    };
    // Tiles in order.  run_slots wants the masked slots first, so a ragged
    // last tile gets a masked pass of its own after the others.
    const int plain_end = ragged_end ? t1 - 1 : t1;
    const int P = (m_lo + 1) & ~1;
    run_slots(
        P, P + (plain_end - t0 - m_lo),
        [&](int i) { return i < P ? (i < m_lo ? t0 + i : -1) : t0 + m_lo + (i - P); }, issue, [&](auto) {},
        compute);
    int t_last = plain_end - 1;
    if (ragged_end) {
        // Buffer 0 is free after the barrier that closed the last slot.
        issue(Buf0{}, t1 - 1);
        __syncthreads();
        compute(Buf0{}, t1 - 1, std::true_type{});
        __syncthreads();
        t_last = t1 - 1;
    }
    flush(PAT_BM * t_last - (PAT_BN - 1), PAT_BM + PAT_BN - 1);
    const float da_key = pair_sum(da_acc);
    if (hf == 0 && key < N) p.da_part[(part * p.n_chunks + chunk) * N + key] = da_key;
}

// da[h][j] = sum over batch elements and over the chunks of j's key block of
// da_part; dr[h][delta] = sum over batch elements, over the key blocks J with
// 128 J <= N - 1 - delta and over the (one or two) chunks of J whose offsets
// include delta, of dr_part.  Workgroup = (head, 8 positions): 32 groups
// of 8 threads take every 32nd key block (and chunk) of every batch
// element, then group 0 adds the 32 partial sums in a fixed order and
// stores the result, so the output does not depend on scheduling.  Rows of
// ordinary heads get zeros.  Consecutive threads read consecutive addresses.
constexpr int PRED_X = 8;                 // positions per workgroup
constexpr int PRED_G = 256 / PRED_X;      // thread groups per position

__global__ __launch_bounds__(256) void pat_reduce_kernel(PatArgs p) {
    __shared__ float red[2][PRED_G][PRED_X];
    const int per_head = (p.N + PRED_X - 1) / PRED_X;
    const int h = (int)(blockIdx.x / per_head);
    const int xl = (int)threadIdx.x % PRED_X;
    const int jg = (int)threadIdx.x / PRED_X;
    const int x = (int)(blockIdx.x % per_head) * PRED_X + xl;
    const int N = p.N;
    const int hidx = p.fixed_index[h];
    float sa = 0.0f, sr = 0.0f;
    if (hidx < p.n_fixed && x < N) {
        const int cq = PAT_BM * p.chunk_tiles;  // queries per chunk
        const int nc_key = pat_chunks(x / PAT_BN, N, p.chunk_tiles);
        const int n_j = (N - 1 - x) / PAT_BN + 1;  // key blocks that reach offset x
        const int ca = x / cq;                    // the chunk whose own queries give offset x
        const int c0 = ca * p.chunk_tiles;  // first tile of chunk ca
        const int c1 = c0 + p.chunk_tiles;  // first tile of chunk ca + 1
        for (int b = 0; b < p.B; ++b) {
            const size_t part = (size_t)(b * p.n_fixed + hidx);
            for (int ch = jg; ch < nc_key; ch += PRED_G) sa += p.da_part[(part * p.n_chunks + ch) * N + x];
            const float* rows_b = p.dr_part + part * p.n_kblocks * p.n_chunks * (size_t)p.part_len;
#pragma unroll 2
            for (int J = jg; J < n_j; J += PRED_G) {
                const int tiles = (N - J * PAT_BN + PAT_BM - 1) / PAT_BM;  // chunk ch exists iff ch * chunk_tiles < tiles
                const float* rows = rows_b + (size_t)J * p.n_chunks * p.part_len;
                if (c0 < tiles) sr += rows[(size_t)ca * p.part_len + (x - (cq * ca - (PAT_BN - 1)))];
                if (c1 < tiles && x >= cq * (ca + 1) - (PAT_BN - 1))
                    sr += rows[(size_t)(ca + 1) * p.part_len + (x - (cq * (ca + 1) - (PAT_BN - 1)))];
            }
        }
    }
    red[0][jg][xl] = sa;
    red[1][jg][xl] = sr;
    __syncthreads();
    if (jg == 0 && x < N) {
        float ta = 0.0f, tr = 0.0f;
#pragma unroll
        for (int g = 0; g < PRED_G; ++g) {
            ta += red[0][g][xl];
            tr += red[1][g][xl];
        }
        p.da[(size_t)h * N + x] = ta;
        p.dr[(size_t)h * N + x] = tr;
    }
}

__global__ void pat_fill_kernel(float* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0.0f;
}

}  // namespace saf
