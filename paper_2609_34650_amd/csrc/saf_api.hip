// Host side of libsaf.so: argument checks and kernel launches for the C ABI
// declared in include/saf.h, include/saf_calib.h, include/saf_fit.h and
// include/saf_measure.h.  No allocation, no synchronisation; the only global
// state is the per-device address of the no-allocation backward's scratch
// array, looked up once per device.
#include "saf.h"
#include "saf_calib.h"
#include "saf_fit.h"
#include "saf_measure.h"

#include <math.h>
#include <algorithm>
#include <mutex>
#include <stdint.h>

#include "saf_bwd.h"
#include "saf_calib_kernels.h"
#include "saf_fit_kernels.h"
#include "saf_fwd.h"
#include "saf_gqa.h"
#include "saf_gqa_bwd.h"
#include "saf_measure_kernels.h"
#include "saf_pattern.h"

#define SAF_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

// Kernels address one (batch, head) slice of N x 64 elements through a buffer
// resource with 32-bit byte offsets, so a slice must stay below 2^31 bytes.
constexpr int kMaxN = 1 << 24;      // bf16: 2^24 rows x 128 B = 2^31 B
constexpr int kMaxNF32 = 1 << 23;   // float32: 2^23 rows x 256 B = 2^31 B

struct Problem {
    uint64_t fixed_mask = 0;
    bool any_fixed = false;
    bool any_ordinary = false;
    bool empty = false;
};

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

// Checks shared by forward and backward.  Fills `pr`; SAF_OK with pr->empty
// set means there is nothing to do.
saf_status_t check_common(saf_dtype_t dt, const uint8_t* head_is_fixed, const float* a, const float* r,
                          int ld_prior, int B, int H, int N, int d, Problem* pr) {
    if (dt != SAF_DTYPE_F32 && dt != SAF_DTYPE_BF16) return SAF_ERR_UNSUPPORTED;
    if (B < 0 || H < 0 || N < 0 || d < 0) return SAF_ERR_SHAPE;
    if (d != saf::HEAD_DIM) return SAF_ERR_UNSUPPORTED;
    if (H > 64) return SAF_ERR_UNSUPPORTED;
    if (N > (dt == SAF_DTYPE_F32 ? kMaxNF32 : kMaxN)) return SAF_ERR_SHAPE;
    // The largest grid is the backward row pre-pass: one workgroup per 32 rows.
    if ((int64_t)B * H * ((N + 31) / 32) > INT32_MAX) return SAF_ERR_SHAPE;
    if (B == 0 || H == 0 || N == 0) {
        pr->empty = true;
        return SAF_OK;
    }
    if (head_is_fixed == nullptr) return SAF_ERR_NULL;
    for (int h = 0; h < H; ++h) {
        if (head_is_fixed[h] > 1) return SAF_ERR_FLAG;
        if (head_is_fixed[h]) {
            pr->fixed_mask |= (1ull << h);
            pr->any_fixed = true;
        } else {
            pr->any_ordinary = true;
        }
    }
    if (pr->any_fixed) {
        if (a == nullptr || r == nullptr) return SAF_ERR_MISSING_PRIOR;
        if (ld_prior < N) return SAF_ERR_SHAPE;
    }
    return SAF_OK;
}

saf_status_t launched() { return hipGetLastError() == hipSuccess ? SAF_OK : SAF_ERR_LAUNCH; }

// Pattern gradients: D [B,H,N], then da partials [B,H,chunks,N], then dr
// partials [B,H,key blocks,chunks,64*chunk_tiles+127] (H bounds the number of
// fixed heads), each part 256-byte aligned.  Chunks of 16 query tiles, more
// when N is so long that the grid's y extent would pass 1024.
struct PatGeom {
    int n_kblocks, chunk_tiles, n_chunks, part_len;
};
PatGeom pattern_geometry(int N) {
    PatGeom g;
    g.n_kblocks = (N + saf::PAT_BN - 1) / saf::PAT_BN;
    const int tiles = (N + saf::PAT_BM - 1) / saf::PAT_BM;
    g.chunk_tiles = tiles > 16 * 1024 ? (tiles + 1023) / 1024 : 16;
    g.n_chunks = (tiles + g.chunk_tiles - 1) / g.chunk_tiles;
    g.part_len = saf::PAT_BM * g.chunk_tiles + saf::PAT_BN - 1;
    return g;
}
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
size_t pattern_workspace_bytes(int B, int H, int N) {
    const PatGeom g = pattern_geometry(N);
    const size_t bh = (size_t)B * H;
    return align256(bh * N * 4) + align256(bh * g.n_chunks * N * 4) +
           align256(bh * g.n_kblocks * g.n_chunks * (size_t)g.part_len * 4);
}

template <typename T>
saf_status_t launch_fwd(const saf::FwdArgs& args, hipStream_t stream) {
    // One launch: fixed heads form their own row normalisers.
    const unsigned grid = (unsigned)((size_t)args.n_qblocks * args.B * args.H);
    hipLaunchKernelGGL(saf::fwd_kernel<T>, dim3(grid), dim3(saf::FWD_THREADS), 0, stream, args);
    return launched();
}

// Heads in order of decreasing work for slice_of: ordinary heads, then fixed.
void fill_head_order(unsigned char* order, uint64_t fixed_mask, int H) {
    int n = 0;
    for (int pass = 0; pass < 2; ++pass)
        for (int h = 0; h < H; ++h)
            if ((int)((fixed_mask >> h) & 1ull) == pass) order[n++] = (unsigned char)h;
}

size_t workspace_bytes(int B, int H, int N) {
    const size_t d_bytes = (size_t)B * H * N * sizeof(float);
    return (d_bytes + 255) & ~(size_t)255;
}

template <typename T>
saf_status_t launch_bwd_stage(saf_bwd_stage_t stage, const saf::BwdArgs& base, hipStream_t stream) {
    saf::BwdArgs args = base;
    if (stage == SAF_BWD_PREPROCESS) {
        const size_t rows = (size_t)args.B * args.H * args.N;
        const unsigned grid = (unsigned)((rows + saf::PRE_ROWS - 1) / saf::PRE_ROWS);
        hipLaunchKernelGGL(saf::bwd_pre_kernel<T>, dim3(grid), dim3(saf::PRE_THREADS), 0, stream, args);
    } else if (stage == SAF_BWD_DKDV) {
        args.n_blocks = (args.N + saf::KV_BN - 1) / saf::KV_BN;
        const unsigned grid = (unsigned)((size_t)args.n_blocks * args.B * args.H);
        hipLaunchKernelGGL(saf::bwd_kv_kernel<T>, dim3(grid), dim3(saf::KV_THREADS), 0, stream, args);
    } else {
        // SAF_BWD_DQ reads D from the workspace; SAF_BWD_DQ_WITH_D forms it
        // and writes it there for a key-block pass enqueued after it.
        args.dq_writes_dsum = stage == SAF_BWD_DQ_WITH_D ? 1 : 0;
        args.n_blocks = (args.N + saf::DQ_BM - 1) / saf::DQ_BM;
        const unsigned grid = (unsigned)((size_t)args.n_blocks * args.B * args.H);
        hipLaunchKernelGGL(saf::bwd_dq_kernel<T>, dim3(grid), dim3(saf::DQ_THREADS), 0, stream, args);
    }
    return launched();
}

saf_status_t check_bwd(saf_bwd_stage_t stage, saf_dtype_t dt, const void* Q, const void* K, const void* V,
                       const void* O, const void* dO, const float* LSE, const uint8_t* head_is_fixed,
                       const float* a, const float* r, int ld_prior, int B, int H, int N, int d, void* dQ,
                       void* dK, void* dV, void* workspace, size_t workspace_bytes_given, Problem* pr) {
    if (stage != SAF_BWD_PREPROCESS && stage != SAF_BWD_DKDV && stage != SAF_BWD_DQ && stage != SAF_BWD_DQ_WITH_D)
        return SAF_ERR_UNSUPPORTED;
    saf_status_t st = check_common(dt, head_is_fixed, a, r, ld_prior, B, H, N, d, pr);
    if (st != SAF_OK || pr->empty) return st;
    if (V == nullptr || O == nullptr || dO == nullptr || LSE == nullptr || dQ == nullptr || dK == nullptr ||
        dV == nullptr || workspace == nullptr)
        return SAF_ERR_NULL;
    if (pr->any_ordinary && (Q == nullptr || K == nullptr)) return SAF_ERR_NULL;
    if (!aligned16(V) || !aligned16(O) || !aligned16(dO) || !aligned16(dQ) || !aligned16(dK) || !aligned16(dV) ||
        !aligned16(LSE) || (Q && !aligned16(Q)) || (K && !aligned16(K)) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return SAF_ERR_ALIGNMENT;
    if (workspace_bytes_given < workspace_bytes(B, H, N)) return SAF_ERR_SHAPE;
    return SAF_OK;
}

saf::BwdArgs make_bwd_args(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                           const float* LSE, const float* a, const float* r, int ld_prior, int B, int H, int N,
                           void* dQ, void* dK, void* dV, void* workspace, const Problem& pr) {
    saf::BwdArgs args;
    args.q = Q;
    args.k = K;
    args.v = V;
    args.o = O;
    args.dO = dO;
    args.lse = LSE;
    args.a = a;
    args.r = r;
    args.dq = dQ;
    args.dk = dK;
    args.dv = dV;
    args.dsum = reinterpret_cast<float*>(workspace);
    args.fixed_mask = pr.fixed_mask;
    args.dq_writes_dsum = 0;
    fill_head_order(args.head_order, pr.fixed_mask, H);
    args.B = B;
    args.H = H;
    args.N = N;
    args.ld_prior = ld_prior;
    args.n_blocks = 0;
    args.scale = 1.0f / sqrtf((float)saf::HEAD_DIM);
    args.scale_log2 = saf::LOG2E / sqrtf((float)saf::HEAD_DIM);
    return args;
}

saf_status_t run_bwd_stage(saf_bwd_stage_t stage, saf_dtype_t dt, const saf::BwdArgs& args, hipStream_t stream) {
    return dt == SAF_DTYPE_BF16 ? launch_bwd_stage<saf::bf16>(stage, args, stream)
                                : launch_bwd_stage<float>(stage, args, stream);
}

// Calibration statistics.
constexpr int kMaxCalibT = 1 << 16;
constexpr int kMaxCalibInputs = 1 << 24;

bool aligned8(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 7u) == 0; }

unsigned fill_grid(size_t n) {
    const size_t blocks = (n + 255) / 256;
    return (unsigned)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
}

int calib_tiles(int T) { return (T + saf::CAL_TILE - 1) / saf::CAL_TILE; }
size_t calib_stats_bytes(int H, int T) {
    const size_t nt = (size_t)calib_tiles(T);
    return ((size_t)H * nt * nt * 2 * sizeof(double) + 255) & ~(size_t)255;
}
size_t calib_workspace_bytes(int H, int T) {
    const size_t nr = (size_t)((T + saf::CAL_FIN_ROWS - 1) / saf::CAL_FIN_ROWS);
    const size_t nc = (size_t)((T + saf::CAL_FIN_COLS - 1) / saf::CAL_FIN_COLS);
    return ((size_t)H * nr * nc * sizeof(double) + 255) & ~(size_t)255;
}

template <typename T>
saf_status_t launch_calib_accum(const saf::CalibArgs& args, hipStream_t stream) {
    const unsigned grid = (unsigned)((size_t)args.H * args.n_tiles * args.n_tiles);
    if (args.m2 != nullptr)
        hipLaunchKernelGGL((saf::calib_accum_kernel<T, true>), dim3(grid), dim3(saf::CAL_THREADS), 0, stream, args);
    else
        hipLaunchKernelGGL((saf::calib_accum_kernel<T, false>), dim3(grid), dim3(saf::CAL_THREADS), 0, stream, args);
    return launched();
}

}  // namespace

SAF_EXPORT saf_status_t saf_hybrid_attn_fwd(saf_dtype_t dt, const void* Q, const void* K, const void* V,
                                            const uint8_t* head_is_fixed, const float* a, const float* r,
                                            int ld_prior, int B, int H, int N, int d, void* O, float* LSE,
                                            hipStream_t stream) {
    Problem pr;
    saf_status_t st = check_common(dt, head_is_fixed, a, r, ld_prior, B, H, N, d, &pr);
    if (st != SAF_OK || pr.empty) return st;
    if (V == nullptr || O == nullptr || LSE == nullptr) return SAF_ERR_NULL;
    if (pr.any_ordinary && (Q == nullptr || K == nullptr)) return SAF_ERR_NULL;
    if (!aligned16(V) || !aligned16(O) || !aligned16(LSE) || (Q && !aligned16(Q)) || (K && !aligned16(K)))
        return SAF_ERR_ALIGNMENT;

    saf::FwdArgs args;
    args.q = Q;
    args.k = K;
    args.v = V;
    args.a = a;
    args.r = r;
    args.o = O;
    args.lse = LSE;
    args.fixed_mask = pr.fixed_mask;
    args.B = B;
    args.H = H;
    args.N = N;
    args.ld_prior = ld_prior;
    fill_head_order(args.head_order, pr.fixed_mask, H);
    args.n_qblocks = (N + saf::FWD_BM - 1) / saf::FWD_BM;
    args.scale_log2 = saf::LOG2E / sqrtf((float)saf::HEAD_DIM);
    return dt == SAF_DTYPE_BF16 ? launch_fwd<saf::bf16>(args, stream) : launch_fwd<float>(args, stream);
}

namespace {

template <typename T, int D>
void launch_gqa(const saf::GqaArgs& args, hipStream_t stream) {
    const unsigned grid = (unsigned)((size_t)args.n_qblocks * args.B * args.Hq);
    hipLaunchKernelGGL((saf::gqa_fwd_kernel<T, D>), dim3(grid), dim3(saf::GQA_THREADS), 0, stream, args);
}

}  // namespace

namespace {

struct GqaProblem {
    uint64_t mask = 0;
    bool any_ordinary = false;
    bool empty = false;
};

// Shape, flag and prior checks shared by the grouped-query entry points.
saf_status_t check_gqa(saf_dtype_t dt, const uint8_t* head_is_fixed, const float* a, const float* r, int ld_prior,
                       int B, int Hq, int Hkv, int N, int d, GqaProblem* pr) {
    if (dt != SAF_DTYPE_F32 && dt != SAF_DTYPE_BF16) return SAF_ERR_UNSUPPORTED;
    if (B < 0 || Hq < 0 || Hkv < 0 || N < 0 || d < 0) return SAF_ERR_SHAPE;
    if (d != 64 && d != 96 && d != 128) return SAF_ERR_UNSUPPORTED;
    if (Hq > 64) return SAF_ERR_UNSUPPORTED;
    // One (batch, head) slice stays below 2^31 bytes for 32-bit buffer offsets.
    if ((int64_t)N * d * (dt == SAF_DTYPE_F32 ? 4 : 2) > INT32_MAX) return SAF_ERR_SHAPE;
    if ((int64_t)B * Hq * ((N + saf::GQA_BM - 1) / saf::GQA_BM) > INT32_MAX) return SAF_ERR_SHAPE;
    if (B == 0 || Hq == 0 || N == 0) {
        pr->empty = true;
        return SAF_OK;
    }
    if (Hkv == 0 || Hq % Hkv != 0) return SAF_ERR_SHAPE;
    if (head_is_fixed == nullptr) return SAF_ERR_NULL;
    for (int h = 0; h < Hq; ++h) {
        if (head_is_fixed[h] > 1) return SAF_ERR_FLAG;
        if (head_is_fixed[h]) pr->mask |= 1ull << h;
        else pr->any_ordinary = true;
    }
    if (pr->mask && (a == nullptr || r == nullptr)) return SAF_ERR_MISSING_PRIOR;
    if (pr->mask && ld_prior < N) return SAF_ERR_SHAPE;
    return SAF_OK;
}

// Key/value heads by decreasing work (an ordinary query head weighs 2, a
// fixed one 1) for slice_of.
void fill_kv_order(unsigned char* order, uint64_t mask, int Hq, int Hkv) {
    const int group = Hq / Hkv;
    int work[64];
    for (int g = 0; g < Hkv; ++g) {
        work[g] = 0;
        for (int i = 0; i < group; ++i) work[g] += ((mask >> (g * group + i)) & 1ull) ? 1 : 2;
        order[g] = (unsigned char)g;
    }
    std::stable_sort(order, order + Hkv, [&](unsigned char x, unsigned char y) { return work[x] > work[y]; });
}

size_t gqa_workspace_bytes(int B, int Hq, int N) {
    return ((size_t)B * Hq * N * sizeof(float) + 255) & ~(size_t)255;
}

template <typename T, int D>
void launch_gqa_bwd(const saf::GqaBwdArgs& base, hipStream_t stream) {
    saf::GqaBwdArgs args = base;
    // The query-block pass runs first: it forms D of the ordinary heads'
    // rows and writes it to the workspace for the key-block pass.
    args.n_blocks = (args.N + saf::GDQ_BM - 1) / saf::GDQ_BM;
    hipLaunchKernelGGL((saf::gqa_bwd_dq_kernel<T, D>), dim3((unsigned)((size_t)args.n_blocks * args.B * args.Hq)),
                       dim3(saf::GDQ_THREADS), 0, stream, args);
    args.n_blocks = (args.N + saf::GKV_BN - 1) / saf::GKV_BN;
    const dim3 grid((unsigned)((size_t)args.n_blocks * args.B * args.Hkv));
    if constexpr (saf::gkv_split<D>()) {
        hipLaunchKernelGGL((saf::gqa_bwd_kv_kernel<T, D, saf::GKV_DK>), grid, dim3(saf::GKV_THREADS), 0, stream, args);
        hipLaunchKernelGGL((saf::gqa_bwd_kv_kernel<T, D, saf::GKV_DV>), grid, dim3(saf::GKV_THREADS), 0, stream, args);
    } else {
        hipLaunchKernelGGL((saf::gqa_bwd_kv_kernel<T, D, saf::GKV_BOTH>), grid, dim3(saf::GKV_THREADS), 0, stream,
                           args);
    }
}

}  // namespace

SAF_EXPORT saf_status_t saf_hybrid_attn_fwd_gqa(saf_dtype_t dt, const void* Q, const void* K, const void* V,
                                                const uint8_t* head_is_fixed, const float* a, const float* r,
                                                int ld_prior, int B, int Hq, int Hkv, int N, int d, void* O,
                                                float* LSE, hipStream_t stream) {
    GqaProblem pr;
    saf_status_t st = check_gqa(dt, head_is_fixed, a, r, ld_prior, B, Hq, Hkv, N, d, &pr);
    if (st != SAF_OK || pr.empty) return st;
    const uint64_t mask = pr.mask;
    if (V == nullptr || O == nullptr || LSE == nullptr) return SAF_ERR_NULL;
    if (pr.any_ordinary && (Q == nullptr || K == nullptr)) return SAF_ERR_NULL;
    if (!aligned16(V) || !aligned16(O) || !aligned16(LSE) || (Q && !aligned16(Q)) || (K && !aligned16(K)))
        return SAF_ERR_ALIGNMENT;
    saf::GqaArgs args;
    args.q = Q;
    args.k = K;
    args.v = V;
    args.a = a;
    args.r = r;
    args.o = O;
    args.lse = LSE;
    args.fixed_mask = mask;
    args.B = B;
    args.Hq = Hq;
    args.Hkv = Hkv;
    args.N = N;
    args.ld_prior = ld_prior;
    args.n_qblocks = (N + saf::GQA_BM - 1) / saf::GQA_BM;
    args.scale_log2 = saf::LOG2E / sqrtf((float)d);
    fill_kv_order(args.kv_order, mask, Hq, Hkv);
    const bool bf = dt == SAF_DTYPE_BF16;
    if (d == 64) bf ? launch_gqa<saf::bf16, 64>(args, stream) : launch_gqa<float, 64>(args, stream);
    else if (d == 96) bf ? launch_gqa<saf::bf16, 96>(args, stream) : launch_gqa<float, 96>(args, stream);
    else bf ? launch_gqa<saf::bf16, 128>(args, stream) : launch_gqa<float, 128>(args, stream);
    return launched();
}

SAF_EXPORT size_t saf_hybrid_attn_bwd_gqa_workspace_bytes(saf_dtype_t dt, int B, int Hq, int Hkv, int N, int d) {
    GqaProblem pr;
    uint8_t none[64] = {0};
    if (check_gqa(dt, none, nullptr, nullptr, N, B, Hq, Hkv, N, d, &pr) != SAF_OK || pr.empty) return 0;
    return gqa_workspace_bytes(B, Hq, N);
}

SAF_EXPORT saf_status_t saf_hybrid_attn_bwd_gqa(saf_dtype_t dt, const void* Q, const void* K, const void* V,
                                                const void* O, const void* dO, const float* LSE,
                                                const uint8_t* head_is_fixed, const float* a, const float* r,
                                                int ld_prior, int B, int Hq, int Hkv, int N, int d, void* dQ,
                                                void* dK, void* dV, void* workspace, size_t workspace_bytes_given,
                                                hipStream_t stream) {
    GqaProblem pr;
    saf_status_t st = check_gqa(dt, head_is_fixed, a, r, ld_prior, B, Hq, Hkv, N, d, &pr);
    if (st != SAF_OK || pr.empty) return st;
    if (V == nullptr || O == nullptr || dO == nullptr || LSE == nullptr || dQ == nullptr || dK == nullptr ||
        dV == nullptr || workspace == nullptr)
        return SAF_ERR_NULL;
    if (pr.any_ordinary && (Q == nullptr || K == nullptr)) return SAF_ERR_NULL;
    if (!aligned16(V) || !aligned16(O) || !aligned16(dO) || !aligned16(dQ) || !aligned16(dK) || !aligned16(dV) ||
        !aligned16(LSE) || (Q && !aligned16(Q)) || (K && !aligned16(K)) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return SAF_ERR_ALIGNMENT;
    if (workspace_bytes_given < gqa_workspace_bytes(B, Hq, N)) return SAF_ERR_SHAPE;
    saf::GqaBwdArgs args;
    args.q = Q;
    args.k = K;
    args.v = V;
    args.o = O;
    args.dO = dO;
    args.lse = LSE;
    args.a = a;
    args.r = r;
    args.dq = dQ;
    args.dk = dK;
    args.dv = dV;
    args.dsum = reinterpret_cast<float*>(workspace);
    args.fixed_mask = pr.mask;
    args.B = B;
    args.Hq = Hq;
    args.Hkv = Hkv;
    args.N = N;
    args.ld_prior = ld_prior;
    args.n_blocks = 0;
    args.scale = 1.0f / sqrtf((float)d);
    args.scale_log2 = saf::LOG2E / sqrtf((float)d);
    fill_kv_order(args.kv_order, pr.mask, Hq, Hkv);
    const bool bf = dt == SAF_DTYPE_BF16;
    if (d == 64) bf ? launch_gqa_bwd<saf::bf16, 64>(args, stream)
                    : launch_gqa_bwd<float, 64>(args, stream);
    else if (d == 96) bf ? launch_gqa_bwd<saf::bf16, 96>(args, stream)
                         : launch_gqa_bwd<float, 96>(args, stream);
    else bf ? launch_gqa_bwd<saf::bf16, 128>(args, stream)
            : launch_gqa_bwd<float, 128>(args, stream);
    return launched();
}

SAF_EXPORT size_t saf_hybrid_attn_bwd_workspace_bytes(saf_dtype_t dt, int B, int H, int N, int d) {
    if (dt != SAF_DTYPE_F32 && dt != SAF_DTYPE_BF16) return 0;
    if (B <= 0 || H <= 0 || N <= 0 || d != saf::HEAD_DIM || H > 64 || N > kMaxN) return 0;
    return workspace_bytes(B, H, N);
}

SAF_EXPORT saf_status_t saf_hybrid_attn_bwd_stage(saf_bwd_stage_t stage, saf_dtype_t dt, const void* Q,
                                                  const void* K, const void* V, const void* O, const void* dO,
                                                  const float* LSE, const uint8_t* head_is_fixed, const float* a,
                                                  const float* r, int ld_prior, int B, int H, int N, int d,
                                                  void* dQ, void* dK, void* dV, void* workspace,
                                                  size_t workspace_bytes_given, hipStream_t stream) {
    Problem pr;
    saf_status_t st = check_bwd(stage, dt, Q, K, V, O, dO, LSE, head_is_fixed, a, r, ld_prior, B, H, N, d, dQ, dK,
                                dV, workspace, workspace_bytes_given, &pr);
    if (st != SAF_OK || pr.empty) return st;
    const saf::BwdArgs args =
        make_bwd_args(Q, K, V, O, dO, LSE, a, r, ld_prior, B, H, N, dQ, dK, dV, workspace, pr);
    return run_bwd_stage(stage, dt, args, stream);
}

SAF_EXPORT saf_status_t saf_hybrid_attn_bwd(saf_dtype_t dt, const void* Q, const void* K, const void* V,
                                            const void* O, const void* dO, const float* LSE,
                                            const uint8_t* head_is_fixed, const float* a, const float* r,
                                            int ld_prior, int B, int H, int N, int d, void* dQ, void* dK,
                                            void* dV, void* workspace, size_t workspace_bytes_given,
                                            hipStream_t stream) {
    Problem pr;
    saf_status_t st = check_bwd(SAF_BWD_PREPROCESS, dt, Q, K, V, O, dO, LSE, head_is_fixed, a, r, ld_prior, B, H,
                                N, d, dQ, dK, dV, workspace, workspace_bytes_given, &pr);
    if (st != SAF_OK || pr.empty) return st;
    const saf::BwdArgs args =
        make_bwd_args(Q, K, V, O, dO, LSE, a, r, ld_prior, B, H, N, dQ, dK, dV, workspace, pr);
    // The query-block pass forms D itself and writes it for the key-block
    // pass, so no row pre-pass runs here.
    st = run_bwd_stage(SAF_BWD_DQ_WITH_D, dt, args, stream);
    if (st != SAF_OK) return st;
    return run_bwd_stage(SAF_BWD_DKDV, dt, args, stream);
}

// ---------------------------------------------------------------------------
// Backward without a caller workspace (saf_hybrid_attn_bwd_noalloc).  Its only
// scratch, the row vector D, lives in this file-scope device array: one copy
// per GPU, held until the process ends.  Host code never passes the array's
// name to a kernel (on the host it is a stand-in, not a device address); it
// uses the address hipGetSymbolAddress returns for the current device, looked
// up once per device and kept in `g_scratch_ptr`.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kNoAllocMaxRows = (size_t)1 << 22;  // B * H * N <= 4,194,304 rows: 16 MiB of float32
static __device__ __align__(256) float scratch[kNoAllocMaxRows];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
float* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device (nullptr on failure).
float* scratch_on_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
        g_scratch_ptr[dev] = reinterpret_cast<float*>(ptr);
    }
    return g_scratch_ptr[dev];
}

}  // namespace

SAF_EXPORT saf_status_t saf_hybrid_attn_bwd_noalloc(saf_dtype_t dt, const void* Q, const void* K, const void* V,
                                                    const void* O, const void* dO, const float* LSE,
                                                    const uint8_t* head_is_fixed, const float* a, const float* r,
                                                    int ld_prior, int B, int H, int N, int d, void* dQ, void* dK,
                                                    void* dV, hipStream_t stream) {
    // Validate as saf_hybrid_attn_bwd does, with a stand-in workspace of the
    // right size (the check reads only its alignment and size).
    Problem pr;
    const size_t need = (B > 0 && H > 0 && N > 0) ? workspace_bytes(B, H, N) : 0;
    void* const probe = reinterpret_cast<void*>((uintptr_t)256);
    saf_status_t st = check_bwd(SAF_BWD_PREPROCESS, dt, Q, K, V, O, dO, LSE, head_is_fixed, a, r, ld_prior, B, H,
                                N, d, dQ, dK, dV, probe, need, &pr);
    if (st != SAF_OK || pr.empty) return st;
    if ((size_t)B * H * N > kNoAllocMaxRows) return SAF_ERR_SHAPE;
    float* ws = scratch_on_current_device();
    if (ws == nullptr) return SAF_ERR_LAUNCH;
    // D is written by the query-block pass for every row the key-block pass
    // reads, so nothing needs clearing between calls.
    const saf::BwdArgs args = make_bwd_args(Q, K, V, O, dO, LSE, a, r, ld_prior, B, H, N, dQ, dK, dV, ws, pr);
    st = run_bwd_stage(SAF_BWD_DQ_WITH_D, dt, args, stream);
    if (st != SAF_OK) return st;
    return run_bwd_stage(SAF_BWD_DKDV, dt, args, stream);
}

SAF_EXPORT size_t saf_hybrid_attn_bwd_pattern_workspace_bytes(saf_dtype_t dt, int B, int H, int N, int d) {
    if (dt != SAF_DTYPE_F32 && dt != SAF_DTYPE_BF16) return 0;
    if (B <= 0 || H <= 0 || N <= 0 || d != saf::HEAD_DIM || H > 64 || N > kMaxN) return 0;
    return pattern_workspace_bytes(B, H, N);
}

SAF_EXPORT saf_status_t saf_hybrid_attn_bwd_pattern(saf_dtype_t dt, const void* V, const void* O, const void* dO,
                                                    const float* LSE, const uint8_t* head_is_fixed, const float* a,
                                                    const float* r, int ld_prior, int B, int H, int N, int d,
                                                    float* da, float* dr, void* workspace,
                                                    size_t workspace_bytes_given, hipStream_t stream) {
    Problem pr;
    saf_status_t st = check_common(dt, head_is_fixed, a, r, ld_prior, B, H, N, d, &pr);
    if (st != SAF_OK || pr.empty) return st;
    if (V == nullptr || O == nullptr || dO == nullptr || LSE == nullptr || da == nullptr || dr == nullptr ||
        workspace == nullptr)
        return SAF_ERR_NULL;
    if (!aligned16(V) || !aligned16(O) || !aligned16(dO) || !aligned16(LSE) ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return SAF_ERR_ALIGNMENT;
    if ((size_t)H * N > INT32_MAX || B > 65535 || workspace_bytes_given < pattern_workspace_bytes(B, H, N))
        return SAF_ERR_SHAPE;
    if (!pr.any_fixed) {  // every row is an ordinary head's: zeros
        const size_t n_out = (size_t)H * N;
        hipLaunchKernelGGL(saf::pat_fill_kernel, dim3(fill_grid(n_out)), dim3(256), 0, stream, da, n_out);
        hipLaunchKernelGGL(saf::pat_fill_kernel, dim3(fill_grid(n_out)), dim3(256), 0, stream, dr, n_out);
        return launched();
    }
    // D for the fixed heads: the row pre-pass with the ordinary heads masked out.
    const uint64_t all = H == 64 ? ~0ull : ((1ull << H) - 1);
    Problem inv = pr;
    inv.fixed_mask = all & ~pr.fixed_mask;
    saf::BwdArgs ba = make_bwd_args(nullptr, nullptr, V, O, dO, LSE, a, r, ld_prior, B, H, N, nullptr, nullptr,
                                    nullptr, workspace, inv);
    st = run_bwd_stage(SAF_BWD_PREPROCESS, dt, ba, stream);
    if (st != SAF_OK) return st;
    saf::PatArgs pa;
    pa.v = V;
    pa.dO = dO;
    pa.lse = LSE;
    const PatGeom geo = pattern_geometry(N);
    char* wsb = reinterpret_cast<char*>(workspace);
    const size_t bhn = align256((size_t)B * H * N * 4);
    const size_t dab = align256((size_t)B * H * geo.n_chunks * N * 4);
    pa.dsum = reinterpret_cast<const float*>(wsb);
    pa.da_part = reinterpret_cast<float*>(wsb + bhn);
    pa.dr_part = reinterpret_cast<float*>(wsb + bhn + dab);
    pa.chunk_tiles = geo.chunk_tiles;
    pa.n_chunks = geo.n_chunks;
    pa.part_len = geo.part_len;
    pa.a = a;
    pa.r = r;
    pa.da = da;
    pa.dr = dr;
    pa.B = B;
    pa.H = H;
    pa.N = N;
    pa.ld_prior = ld_prior;
    pa.n_fixed = 0;
    for (int h = 0; h < 64; ++h) pa.fixed_index[h] = 255;
    for (int h = 0; h < H; ++h)
        if ((pr.fixed_mask >> h) & 1ull) {
            pa.fixed_index[h] = (unsigned char)pa.n_fixed;
            pa.heads[pa.n_fixed++] = (unsigned char)h;
        }
    pa.n_kblocks = geo.n_kblocks;
    const dim3 grid((unsigned)((size_t)pa.n_kblocks * B * pa.n_fixed), (unsigned)geo.n_chunks);
    if (dt == SAF_DTYPE_BF16)
        hipLaunchKernelGGL(saf::bwd_pattern_kernel<saf::bf16>, grid, dim3(saf::PAT_THREADS), 0, stream, pa);
    else
        hipLaunchKernelGGL(saf::bwd_pattern_kernel<float>, grid, dim3(saf::PAT_THREADS), 0, stream, pa);
    if (launched() != SAF_OK) return SAF_ERR_LAUNCH;
    const unsigned rgrid = (unsigned)((size_t)H * ((N + saf::PRED_X - 1) / saf::PRED_X));
    hipLaunchKernelGGL(saf::pat_reduce_kernel, dim3(rgrid), dim3(256), 0, stream, pa);
    return launched();
}

SAF_EXPORT saf_status_t saf_calib_accumulate(saf_dtype_t dt, const void* Q, const void* K, const float* LSE, int B,
                                             int H, int T, int d, int n_seen, float* mean, float* m2, double* stats,
                                             hipStream_t stream) {
    if (dt != SAF_DTYPE_F32 && dt != SAF_DTYPE_BF16) return SAF_ERR_UNSUPPORTED;
    if (B < 0 || H < 0 || T < 0 || d < 0 || n_seen < 0) return SAF_ERR_SHAPE;
    if (d != saf::HEAD_DIM || H > 64) return SAF_ERR_UNSUPPORTED;
    if (T > kMaxCalibT || (int64_t)n_seen + B > kMaxCalibInputs) return SAF_ERR_SHAPE;
    if (B == 0 || H == 0 || T == 0) return SAF_OK;
    if (Q == nullptr || K == nullptr || LSE == nullptr || mean == nullptr || stats == nullptr) return SAF_ERR_NULL;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(LSE) || !aligned16(mean) || (m2 && !aligned16(m2)) ||
        !aligned8(stats))
        return SAF_ERR_ALIGNMENT;
    saf::CalibArgs args;
    args.q = Q;
    args.k = K;
    args.lse = LSE;
    args.mean = mean;
    args.m2 = m2;
    args.stats = stats;
    args.B = B;
    args.H = H;
    args.T = T;
    args.n_seen = n_seen;
    args.n_tiles = calib_tiles(T);
    args.scale = 1.0f / sqrtf((float)saf::HEAD_DIM);
    return dt == SAF_DTYPE_BF16 ? launch_calib_accum<saf::bf16>(args, stream) : launch_calib_accum<float>(args, stream);
}

SAF_EXPORT size_t saf_calib_stats_bytes(int H, int T) {
    if (H <= 0 || H > 64 || T <= 0 || T > kMaxCalibT) return 0;
    return calib_stats_bytes(H, T);
}

SAF_EXPORT size_t saf_calib_finalize_workspace_bytes(int H, int T) {
    if (H <= 0 || H > 64 || T <= 0 || T > kMaxCalibT) return 0;
    return calib_workspace_bytes(H, T);
}

SAF_EXPORT saf_status_t saf_calib_finalize(int H, int T, int n_total, const float* mean, const double* stats,
                                           float* eta_abs, float* eta_rel, float* s_var, float* s_kl,
                                           void* workspace, size_t workspace_bytes_given, hipStream_t stream) {
    if (H < 0 || T < 0 || n_total < 0) return SAF_ERR_SHAPE;
    if (H > 64) return SAF_ERR_UNSUPPORTED;
    if (T > kMaxCalibT || n_total > kMaxCalibInputs) return SAF_ERR_SHAPE;
    if (H == 0 || T == 0) return SAF_OK;
    if (n_total < 1) return SAF_ERR_SHAPE;
    if (mean == nullptr || stats == nullptr || eta_abs == nullptr || eta_rel == nullptr || s_var == nullptr ||
        s_kl == nullptr || workspace == nullptr)
        return SAF_ERR_NULL;
    if (!aligned16(mean) || !aligned8(stats) || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return SAF_ERR_ALIGNMENT;
    if (workspace_bytes_given < calib_workspace_bytes(H, T)) return SAF_ERR_SHAPE;
    saf::CalibFinalArgs args;
    args.mean = mean;
    args.stats = stats;
    args.eta_abs = eta_abs;
    args.eta_rel = eta_rel;
    args.s_var = s_var;
    args.s_kl = s_kl;
    args.part = reinterpret_cast<double*>(workspace);
    args.H = H;
    args.T = T;
    args.n_total = n_total;
    args.n_tiles = calib_tiles(T);
    args.n_cgroups = (T + saf::CAL_FIN_COLS - 1) / saf::CAL_FIN_COLS;
    args.n_rchunks = (T + saf::CAL_FIN_ROWS - 1) / saf::CAL_FIN_ROWS;
    const size_t n_eta = (size_t)H * T;
    hipLaunchKernelGGL(saf::calib_fill_kernel, dim3(fill_grid(n_eta)), dim3(256), 0, stream, eta_abs, n_eta);
    hipLaunchKernelGGL(saf::calib_fill_kernel, dim3(fill_grid(n_eta)), dim3(256), 0, stream, eta_rel, n_eta);
    if (launched() != SAF_OK) return SAF_ERR_LAUNCH;
    const unsigned grid = (unsigned)((size_t)H * args.n_rchunks * args.n_cgroups);
    hipLaunchKernelGGL(saf::calib_final_kernel, dim3(grid), dim3(saf::CAL_FIN_COLS), 0, stream, args);
    if (launched() != SAF_OK) return SAF_ERR_LAUNCH;
    hipLaunchKernelGGL(saf::calib_scores_kernel, dim3(H), dim3(256), 0, stream, args);
    return launched();
}

// ---------------------------------------------------------------------------
// Compact fit
// ---------------------------------------------------------------------------
namespace {

struct FitLayout {
    size_t rowsum, part, m, v, col, diag, logz, total;
};
FitLayout fit_layout(int H, int T) {
    const size_t ht = (size_t)H * T;
    const size_t nr = (size_t)((T + saf::FIT_ROWS - 1) / saf::FIT_ROWS);
    const size_t nc = (size_t)((T + saf::FIT_COLS - 1) / saf::FIT_COLS);
    FitLayout l;
    size_t off = 0;
    l.rowsum = off; off += align256(ht * 4);
    l.part = off;   off += align256((size_t)H * nr * nc * 8);
    l.m = off;      off += align256(2 * ht * 4);
    l.v = off;      off += align256(2 * ht * 4);
    l.col = off;    off += align256(ht * 4);
    l.diag = off;   off += align256(ht * 4);
    l.logz = off;   off += align256(ht * 4);
    l.total = off;
    return l;
}

saf::FitArgs fit_args(int H, int T, void* workspace) {
    const FitLayout l = fit_layout(H, T);
    char* w = reinterpret_cast<char*>(workspace);
    saf::FitArgs f = {};
    f.rowsum = reinterpret_cast<float*>(w + l.rowsum);
    f.part = reinterpret_cast<double*>(w + l.part);
    f.m = reinterpret_cast<float*>(w + l.m);
    f.v = reinterpret_cast<float*>(w + l.v);
    f.col = reinterpret_cast<float*>(w + l.col);
    f.diag = reinterpret_cast<float*>(w + l.diag);
    f.logz = reinterpret_cast<float*>(w + l.logz);
    f.H = H;
    f.T = T;
    f.n_cgroups = (T + saf::FIT_COLS - 1) / saf::FIT_COLS;
    f.n_rchunks = (T + saf::FIT_ROWS - 1) / saf::FIT_ROWS;
    return f;
}

saf_status_t check_fit_shape(int H, int T) {
    if (H < 0 || T < 0) return SAF_ERR_SHAPE;
    if (H > 64) return SAF_ERR_UNSUPPORTED;
    if (T > kMaxCalibT) return SAF_ERR_SHAPE;
    return SAF_OK;
}

}  // namespace

SAF_EXPORT size_t saf_fit_workspace_bytes(int H, int T) {
    if (H <= 0 || T <= 0 || check_fit_shape(H, T) != SAF_OK) return 0;
    return fit_layout(H, T).total;
}

SAF_EXPORT saf_status_t saf_fit_targets(int H, int T, const float* mean, float floor_value, float* eta_abs,
                                        float* eta_rel, double* neg_entropy, void* workspace,
                                        size_t workspace_bytes_given, hipStream_t stream) {
    saf_status_t st = check_fit_shape(H, T);
    if (st != SAF_OK) return st;
    if (H == 0 || T == 0) return SAF_OK;
    if (!(floor_value > 0.0f) || !(floor_value < 1.0f)) return SAF_ERR_SHAPE;
    if (mean == nullptr || eta_abs == nullptr || eta_rel == nullptr || neg_entropy == nullptr || workspace == nullptr)
        return SAF_ERR_NULL;
    if (!aligned16(mean) || !aligned8(neg_entropy) || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return SAF_ERR_ALIGNMENT;
    if (workspace_bytes_given < fit_layout(H, T).total) return SAF_ERR_SHAPE;
    saf::FitArgs f = fit_args(H, T, workspace);
    f.mean = mean;
    f.eta_abs = eta_abs;
    f.eta_rel = eta_rel;
    f.neg_entropy = neg_entropy;
    f.floor_value = floor_value;
    const size_t ht = (size_t)H * T;
    hipLaunchKernelGGL(saf::fit_fill_kernel, dim3(fill_grid(ht)), dim3(256), 0, stream, eta_abs, ht);
    hipLaunchKernelGGL(saf::fit_fill_kernel, dim3(fill_grid(ht)), dim3(256), 0, stream, eta_rel, ht);
    hipLaunchKernelGGL(saf::fit_rowsum_kernel, dim3((unsigned)(H * ((T + 3) / 4))), dim3(256), 0, stream, f);
    const unsigned grid = (unsigned)((size_t)H * f.n_rchunks * f.n_cgroups);
    hipLaunchKernelGGL(saf::fit_target_kernel, dim3(grid), dim3(saf::FIT_COLS), 0, stream, f);
    hipLaunchKernelGGL(saf::fit_entropy_kernel, dim3(H), dim3(256), 0, stream, f);
    return launched();
}

SAF_EXPORT saf_status_t saf_compact_fit(int H, int T, const float* eta_abs, const float* eta_rel,
                                        const double* neg_entropy, int steps, float lr, float floor_value, float* a,
                                        float* r, float* log_z, float* kl, void* workspace,
                                        size_t workspace_bytes_given, hipStream_t stream) {
    saf_status_t st = check_fit_shape(H, T);
    if (st != SAF_OK) return st;
    if (H == 0 || T == 0) return SAF_OK;
    if (steps < 0 || !(lr >= 0.0f) || !(floor_value > 0.0f) || !(floor_value < 1.0f)) return SAF_ERR_SHAPE;
    if (eta_abs == nullptr || eta_rel == nullptr || neg_entropy == nullptr || a == nullptr || r == nullptr ||
        kl == nullptr || workspace == nullptr)
        return SAF_ERR_NULL;
    if (!aligned8(neg_entropy) || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return SAF_ERR_ALIGNMENT;
    if (workspace_bytes_given < fit_layout(H, T).total) return SAF_ERR_SHAPE;
    saf::FitArgs f = fit_args(H, T, workspace);
    f.eta_abs = const_cast<float*>(eta_abs);
    f.eta_rel = const_cast<float*>(eta_rel);
    f.neg_entropy = const_cast<double*>(neg_entropy);
    f.alpha = a;
    f.rho = r;
    f.kl = kl;
    f.floor_value = floor_value;
    f.lr = lr;
    if (log_z != nullptr) f.logz = log_z;
    saf::NormArgs na = {};
    na.a = a;
    na.r = r;
    na.lse = f.logz;
    na.B = 1;
    na.H = H;
    na.N = T;
    na.ld_prior = T;
    na.n_rblocks = (T + saf::NORM_ROWS - 1) / saf::NORM_ROWS;
    na.n_fixed = H;
    for (int h = 0; h < H; ++h) na.heads[h] = (unsigned char)h;
    const size_t ht = (size_t)H * T;
    const unsigned elem_grid = fill_grid(ht);
    const unsigned lse_grid = (unsigned)((size_t)na.n_rblocks * H);
    const unsigned marg_grid = (unsigned)((size_t)H * f.n_rchunks * f.n_cgroups);
    hipLaunchKernelGGL(saf::fit_init_kernel, dim3(elem_grid), dim3(256), 0, stream, f);
    if (launched() != SAF_OK) return SAF_ERR_LAUNCH;
    double p1 = 1.0, p2 = 1.0;
    for (int t = 1; t <= steps; ++t) {
        p1 *= (double)saf::FIT_ADAM_BETA1;
        p2 *= (double)saf::FIT_ADAM_BETA2;
        f.bc1 = (float)(1.0 - p1);
        f.bc2 = (float)(1.0 - p2);
        hipLaunchKernelGGL(saf::fixed_lse_kernel, dim3(lse_grid), dim3(saf::NORM_THREADS), 0, stream, na);
        hipLaunchKernelGGL(saf::fit_marginals_kernel, dim3(marg_grid), dim3(saf::FIT_COLS), 0, stream, f);
        hipLaunchKernelGGL(saf::fit_adam_kernel, dim3(elem_grid), dim3(256), 0, stream, f);
        if (launched() != SAF_OK) return SAF_ERR_LAUNCH;
    }
    hipLaunchKernelGGL(saf::fixed_lse_kernel, dim3(lse_grid), dim3(saf::NORM_THREADS), 0, stream, na);
    hipLaunchKernelGGL(saf::fit_kl_kernel, dim3(H), dim3(256), 0, stream, f);
    return launched();
}

// Measurement aids.
SAF_EXPORT saf_status_t saf_clock_probe(uint64_t* out, int duration_us, hipStream_t stream) {
    if (out == nullptr) return SAF_ERR_NULL;
    if (duration_us < 1 || duration_us > 1000000) return SAF_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(out) & 7u) != 0) return SAF_ERR_ALIGNMENT;
    const uint64_t ticks = (uint64_t)duration_us * 100u;  // reference clock: 100 MHz
    hipLaunchKernelGGL(saf::clock_probe_kernel, dim3(1), dim3(64), 0, stream, out, ticks);
    return launched();
}

SAF_EXPORT saf_status_t saf_lds_read_probe(const void* src, size_t bytes, float* sink, hipStream_t stream) {
    if (src == nullptr || sink == nullptr) return SAF_ERR_NULL;
    if (bytes < (size_t)saf::PROBE_UNIT || bytes % saf::PROBE_UNIT != 0 || bytes > ((size_t)1 << 40))
        return SAF_ERR_SHAPE;
    if (!aligned16(src) || (reinterpret_cast<uintptr_t>(sink) & 3u) != 0) return SAF_ERR_ALIGNMENT;
    const unsigned long long units = bytes / saf::PROBE_UNIT;
    const unsigned grid = (unsigned)((units + saf::PROBE_UNITS_PER_WG - 1) / saf::PROBE_UNITS_PER_WG);
    hipLaunchKernelGGL(saf::lds_read_probe_kernel, dim3(grid), dim3(saf::PROBE_THREADS), 0, stream,
                       reinterpret_cast<const char*>(src), units, sink);
    return launched();
}

SAF_EXPORT saf_status_t saf_lds_pattern_probe(int pattern, int iters, uint32_t* sink, hipStream_t stream) {
    if (sink == nullptr) return SAF_ERR_NULL;
    if (pattern < 0 || pattern >= saf::LDS_PATTERN_COUNT || iters < 1 || iters > (1 << 20)) return SAF_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(sink) & 3u) != 0) return SAF_ERR_ALIGNMENT;
    const dim3 grid(saf::LDS_PATTERN_BLOCKS), block(saf::LDS_PATTERN_THREADS);
    switch (pattern) {
        case 0: hipLaunchKernelGGL(saf::lds_pattern_kernel<0>, grid, block, 0, stream, sink, iters); break;
        case 1: hipLaunchKernelGGL(saf::lds_pattern_kernel<1>, grid, block, 0, stream, sink, iters); break;
        case 2: hipLaunchKernelGGL(saf::lds_pattern_kernel<2>, grid, block, 0, stream, sink, iters); break;
        case 3: hipLaunchKernelGGL(saf::lds_pattern_kernel<3>, grid, block, 0, stream, sink, iters); break;
        case 4: hipLaunchKernelGGL(saf::lds_pattern_kernel<4>, grid, block, 0, stream, sink, iters); break;
        case 5: hipLaunchKernelGGL(saf::lds_pattern_kernel<5>, grid, block, 0, stream, sink, iters); break;
        default: hipLaunchKernelGGL(saf::lds_pattern_kernel<6>, grid, block, 0, stream, sink, iters); break;
    }
    return launched();
}

SAF_EXPORT saf_status_t saf_mfma_rate_probe(int shape, int waves_per_simd, int iters, uint64_t* clk, float* sink,
                                            hipStream_t stream) {
    if (clk == nullptr || sink == nullptr) return SAF_ERR_NULL;
    if (shape < 0 || shape > 1 || waves_per_simd < 1 || waves_per_simd > 2 || iters < 1 || iters > (1 << 20))
        return SAF_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(clk) & 7u) != 0 || (reinterpret_cast<uintptr_t>(sink) & 3u) != 0)
        return SAF_ERR_ALIGNMENT;
    const dim3 grid(saf::MFMA_PROBE_BLOCKS), block(256 * waves_per_simd);
    if (shape == 0)
        hipLaunchKernelGGL(saf::mfma_rate_kernel<0>, grid, block, 0, stream, clk, sink, iters);
    else
        hipLaunchKernelGGL(saf::mfma_rate_kernel<1>, grid, block, 0, stream, clk, sink, iters);
    return launched();
}

SAF_EXPORT const char* saf_status_str(saf_status_t s) {
    switch (s) {
        case SAF_OK: return "ok";
        case SAF_ERR_NULL: return "a required pointer is NULL";
        case SAF_ERR_SHAPE: return "invalid size (negative, N above the limit, grid too large, ld_prior < N, or workspace too small)";
        case SAF_ERR_UNSUPPORTED: return "unsupported dtype, head dimension (d must be 64) or head count (H <= 64)";
        case SAF_ERR_MISSING_PRIOR: return "a head is fixed but a or r is NULL";
        case SAF_ERR_LAUNCH: return "kernel launch failed";
        case SAF_ERR_ALIGNMENT: return "a tensor pointer is not 16-byte aligned (workspace: 256-byte)";
        case SAF_ERR_FLAG: return "head_is_fixed holds a byte other than 0 or 1";
    }
    return "unknown status";
}
