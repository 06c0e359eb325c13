/*
 * saf.h -- C ABI of libsaf.so: the fused hybrid causal-attention layer of
 * Selective Attention Freezing ("When Can Attention Heads Be Statically
 * Defined?"), forward and backward, for AMD Instinct MI355X (gfx950).
 *
 * One layer has H heads.  An ordinary head computes causal softmax attention
 * (Appendix "Attention notation and calibration", Eqs. standard-head):
 *     S = Q K^T / sqrt(d),  A = softmax_causal(S),  O = A V.
 * A fixed ("replaced") head mixes values with a fixed causal row-stochastic
 * pattern built from two length-N preference vectors (Section
 * "Fixed-pattern construction and fitting", Eq. compact-prior), with 0-based
 * storage a[j] = alpha(j+1) and r[delta] = rho(delta):
 *     P(i, j) = exp(a[j] + r[i - j]) / Z(i)  for j <= i,  0 for j > i,
 *     Z(i)    = sum_{j <= i} exp(a[j] + r[i - j]),         O = P V.
 * Fixed heads never read Q or K, take no 1/sqrt(d), and the pattern takes no
 * gradient: the backward gives a fixed head only dV = P^T dO and writes exact
 * zeros into its dQ and dK slices (Section "Replacement schedules and fused
 * execution", paragraph "Fused computation"; Appendix "Mixed-head execution
 * and numerical checks").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensors Q, K, V, O, dO, dQ, dK, dV are DEVICE pointers to contiguous
 *   [B, H, N, d] arrays of the element type `dt` (row-major, d fastest), each
 *   16-byte aligned.  LSE is a DEVICE pointer to contiguous [B, H, N] float32.
 * - a and r are DEVICE pointers to float32 [H, ld_prior] arrays (ld_prior >=
 *   N; only the first N entries of each row are read; rows of ordinary heads
 *   are never read).  They are shared by every batch element.  Entries must be
 *   finite.
 * - head_is_fixed is a HOST pointer to H bytes: 0 = ordinary, 1 = fixed.
 * - The caller owns every buffer.  The library never allocates or frees
 *   device memory, keeps no mutable global state, never synchronises the
 *   stream, and only enqueues kernels on `stream` (0 = the null stream).
 *   Outputs are overwritten, never accumulated into.
 * - Arguments are checked before anything is enqueued; on any error nothing
 *   is launched and nothing is written.  A kernel fault surfaces at the
 *   caller's next synchronisation, not here.
 * - Limits of this entry point: d == 64, 1 <= H <= 64, N <= 2^24 for bf16 and
 *   N <= 2^23 for float32 (one (batch, head) slice stays below 2^31 bytes),
 *   and B * H * ceil(N / 32) <= 2^31 - 1.  B, H or N equal to 0 is an empty
 *   problem: SAF_OK, nothing launched.
 * - Numerics: products on MFMA in the element type with float32 accumulation;
 *   softmax statistics, LSE and the fixed-head normalisers in float32.  Results
 *   are rounded once to the element type (nearest even for bf16).
 */
#ifndef SAF_H
#define SAF_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SAF_DTYPE_F32 = 0,  /* float32 activations, float32 MFMA (v_mfma_f32_32x32x2_f32) */
    SAF_DTYPE_BF16 = 1  /* bfloat16 activations, bf16 MFMA with float32 accumulation */
} saf_dtype_t;

typedef enum {
    SAF_OK = 0,
    SAF_ERR_NULL = 1,          /* a required pointer is NULL */
    SAF_ERR_SHAPE = 2,         /* negative size, N or B*H*N above the limits, ld_prior < N, or workspace too small */
    SAF_ERR_UNSUPPORTED = 3,   /* unknown dtype, d != 64, H > 64 */
    SAF_ERR_MISSING_PRIOR = 4, /* a head is fixed but a or r is NULL */
    SAF_ERR_LAUNCH = 5,        /* the HIP runtime rejected a kernel launch */
    SAF_ERR_ALIGNMENT = 6,     /* a tensor pointer is not 16-byte aligned */
    SAF_ERR_FLAG = 7           /* head_is_fixed holds a byte other than 0 or 1 */
} saf_status_t;

/*
 * Forward of the hybrid layer (Section "Replacement schedules and fused
 * execution"; Appendix "Mixed-head execution and numerical checks"): one
 * launch of the attention kernel for all heads, in which every workgroup
 * takes one (batch, head, block of queries) and the head's flag selects its
 * path; outputs land in the original head order.  A fixed head's workgroup
 * sums its row normalisers Z(i) from a and r as it forms the weights (the
 * paper precomputes these normalisers; here they are recomputed on every
 * call, in float32) and writes log Z(i) into LSE.
 *   Q, K : [B,H,N,d] `dt`; read for ordinary heads only (fixed-head slices may
 *          hold anything, NaN included).  May be NULL if every head is fixed.
 *   V    : [B,H,N,d] `dt`.
 *   O    : [B,H,N,d] `dt`, written.
 *   LSE  : [B,H,N] float32, written: natural-log row normaliser,
 *          log sum_{j<=i} exp(S[i,j]) for ordinary heads, log Z(i) for fixed.
 */
saf_status_t saf_hybrid_attn_fwd(saf_dtype_t dt,
                                 const void* Q, const void* K, const void* V,
                                 const uint8_t* head_is_fixed,
                                 const float* a, const float* r, int ld_prior,
                                 int B, int H, int N, int d,
                                 void* O, float* LSE,
                                 hipStream_t stream);

/*
 * Forward of the hybrid layer with grouped-query attention and head
 * dimension 64, 96 or 128 (the paper's grouped-query prefill layout --
 * Appendix "Replacement in pretrained models", subsection "GQA prefill
 * measurements": 32 query heads sharing 8 key/value heads at d = 128 -- and
 * its 1B model's head width, Appendix "1B training and evaluation").  Query head h uses key/value head h / (Hq / Hkv); a fixed query
 * head reads only V of its group (the grouped-query implementation keeps the
 * shared key and value heads, Appendix "Mixed-head execution and numerical
 * checks").  Same conventions and outputs as saf_hybrid_attn_fwd, with
 *   Q, O : [B, Hq, N, d] `dt`;  K, V : [B, Hkv, N, d] `dt`;
 *   LSE  : [B, Hq, N] float32;  head_is_fixed, a, r : per query head (Hq).
 * Limits: d in {64, 96, 128}, Hq <= 64, Hq a multiple of Hkv, one slice
 * N * d * sizeof(dt) < 2^31 bytes.  With Hkv == Hq and d == 64 it computes
 * what saf_hybrid_attn_fwd computes (a separate, simpler kernel: one 32-query
 * block per wavefront; one launch, in which a fixed head's workgroup sums its
 * row normalisers from the weights it forms, as in saf_hybrid_attn_fwd).
 * Its backward is saf_hybrid_attn_bwd_gqa.
 */
saf_status_t saf_hybrid_attn_fwd_gqa(saf_dtype_t dt,
                                     const void* Q, const void* K, const void* V,
                                     const uint8_t* head_is_fixed,
                                     const float* a, const float* r, int ld_prior,
                                     int B, int Hq, int Hkv, int N, int d,
                                     void* O, float* LSE,
                                     hipStream_t stream);

/* Bytes of device workspace saf_hybrid_attn_bwd_gqa needs (a multiple of
 * 256).  Returns 0 for an empty or invalid problem. */
size_t saf_hybrid_attn_bwd_gqa_workspace_bytes(saf_dtype_t dt, int B, int Hq, int Hkv, int N, int d);

/*
 * Backward of the grouped-query hybrid layer (head dimension 64, 96 or 128)
 * for the loss sum(O * dO).  A shared key/value head receives the sum over
 * the query heads of its group: ordinary query heads add to dK and dV as in
 * saf_hybrid_attn_bwd, fixed query heads add P^T dO to dV only and get exact
 * zeros in dQ (the grouped-query path keeps every shared key/value head and
 * maps each ordinary query head to its group, Appendix "Mixed-head execution
 * and numerical checks").  Two launches (three at d = 128): the query-block
 * pass, which also forms D = rowsum(dO * O) of the ordinary heads and writes
 * it to the workspace, then the key-block pass (one workgroup per batch
 * element, key/value head and 128 keys, looping over the group); at d = 128
 * the key-block pass runs once for dK and once for dV.
 *   Q, O, dO : [B, Hq, N, d] `dt` (O and LSE as written by
 *              saf_hybrid_attn_fwd_gqa);  LSE : [B, Hq, N] float32;
 *   K, V     : [B, Hkv, N, d] `dt`;
 *   dQ       : [B, Hq, N, d] `dt`, written (zeros for fixed heads);
 *   dK, dV   : [B, Hkv, N, d] `dt`, written (dK is zero for a key/value head
 *              whose query heads are all fixed);
 *   workspace: DEVICE, >= saf_hybrid_attn_bwd_gqa_workspace_bytes(), owned
 *              by the caller, 256-byte aligned; contents on entry ignored.
 * Limits and errors as saf_hybrid_attn_fwd_gqa; SAF_ERR_SHAPE also when the
 * workspace is too small.
 */
saf_status_t saf_hybrid_attn_bwd_gqa(saf_dtype_t dt,
                                     const void* Q, const void* K, const void* V,
                                     const void* O, const void* dO, const float* LSE,
                                     const uint8_t* head_is_fixed,
                                     const float* a, const float* r, int ld_prior,
                                     int B, int Hq, int Hkv, int N, int d,
                                     void* dQ, void* dK, void* dV,
                                     void* workspace, size_t workspace_bytes,
                                     hipStream_t stream);

/* Bytes of device workspace saf_hybrid_attn_bwd needs (a multiple of 256).
 * Returns 0 for an empty or invalid problem. */
size_t saf_hybrid_attn_bwd_workspace_bytes(saf_dtype_t dt, int B, int H, int N, int d);

/*
 * Backward of the hybrid layer for the loss sum(O * dO) (Appendix "Mixed-head
 * execution and numerical checks": key-block programs produce dV for every
 * head and dK for ordinary heads; a separate query-block pass produces dQ for
 * ordinary heads only).  Two launches: the query-block pass, which also forms
 * D_i = sum_c dO*O for ordinary heads and leaves it in the workspace, then the
 * key-block pass, which reads it.
 *   Q, K, V, O, dO : [B,H,N,d] `dt` (O and LSE as written by the forward).
 *   LSE            : [B,H,N] float32 from the forward.
 *   dQ, dK, dV     : [B,H,N,d] `dt`, written; fixed heads get exact zeros in
 *                    dQ and dK.
 *   workspace      : DEVICE, >= saf_hybrid_attn_bwd_workspace_bytes(), owned
 *                    by the caller, 256-byte aligned; its contents on entry
 *                    are ignored.
 */
saf_status_t saf_hybrid_attn_bwd(saf_dtype_t dt,
                                 const void* Q, const void* K, const void* V,
                                 const void* O, const void* dO, const float* LSE,
                                 const uint8_t* head_is_fixed,
                                 const float* a, const float* r, int ld_prior,
                                 int B, int H, int N, int d,
                                 void* dQ, void* dK, void* dV,
                                 void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/*
 * Backward of the hybrid layer that allocates nothing and takes no workspace,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  Same
 * arguments (minus the workspace), launches, results and errors as
 * saf_hybrid_attn_bwd; its one scratch buffer, the row vector D, is a
 * file-scope device array of the library holding 2^22 float32 (16 MiB), one
 * copy per GPU, kept until the process ends.
 *   Limit: B * H * N <= 4,194,304; larger problems return SAF_ERR_SHAPE
 *          before anything is launched.
 *   The current HIP device must be the device `stream` belongs to (the
 *   array's address is looked up for the current device on its first call
 *   there).  SAF_ERR_LAUNCH if that lookup fails.
 *   Every call on one GPU shares that GPU's array: calls that overlap in
 *   time on one GPU (two streams, or two threads) race and must not be
 *   issued.  Calls in order on one stream are safe: each call writes every
 *   entry of D it reads before reading it.
 */
saf_status_t saf_hybrid_attn_bwd_noalloc(saf_dtype_t dt,
                                         const void* Q, const void* K, const void* V,
                                         const void* O, const void* dO, const float* LSE,
                                         const uint8_t* head_is_fixed,
                                         const float* a, const float* r, int ld_prior,
                                         int B, int H, int N, int d,
                                         void* dQ, void* dK, void* dV,
                                         hipStream_t stream);

/* The backward's launches, enqueued one at a time (same arguments and
 * contract).  Two sequences give the gradients, on one stream with one
 * workspace:
 *   SAF_BWD_DQ_WITH_D, then SAF_BWD_DKDV: exactly the launches of
 *     saf_hybrid_attn_bwd (the query-block pass forms D = rowsum(dO * O)
 *     from the dO fragments it holds and writes it into the workspace);
 *   SAF_BWD_PREPROCESS (a row pre-pass that writes D), then SAF_BWD_DKDV
 *     and SAF_BWD_DQ in either order (both read D): the same gradients up
 *     to the float32 rounding order of D.
 * DKDV writes dK and dV; DQ and DQ_WITH_D write dQ.  Any other value is
 * SAF_ERR_UNSUPPORTED. */
typedef enum {
    SAF_BWD_PREPROCESS = 0,
    SAF_BWD_DKDV = 1,
    SAF_BWD_DQ = 2,
    SAF_BWD_DQ_WITH_D = 3
} saf_bwd_stage_t;

saf_status_t saf_hybrid_attn_bwd_stage(saf_bwd_stage_t stage, saf_dtype_t dt,
                                       const void* Q, const void* K, const void* V,
                                       const void* O, const void* dO, const float* LSE,
                                       const uint8_t* head_is_fixed,
                                       const float* a, const float* r, int ld_prior,
                                       int B, int H, int N, int d,
                                       void* dQ, void* dK, void* dV,
                                       void* workspace, size_t workspace_bytes,
                                       hipStream_t stream);

/*
 * Gradients of trainable fixed patterns (Appendix "Pattern content and
 * trainability": the variant that keeps optimising alpha and rho after
 * replacement).  For every fixed head, with L(i, j) = a[j] + r[i - j],
 * P = softmax_causal(L) and the loss sum(O * dO):
 *     dP = dO V^T,  D_i = rowsum(dO * O)_i,  dL = P * (dP - D),
 *     da[h][j] = sum_b sum_i dL(i, j),   dr[h][delta] = sum_b sum_{i-j=delta} dL(i, j).
 * The frozen layer never needs this call; it adds one N x N x d product per
 * fixed head and batch element.  Call it beside saf_hybrid_attn_bwd (which
 * still gives dV, and zeros in the fixed heads' dQ and dK).
 *   V, O, dO  : [B,H,N,d] `dt` (O and LSE as written by the forward).
 *   LSE       : [B,H,N] float32 from the forward (log Z for fixed heads).
 *   da, dr    : DEVICE [H, N] float32, written; rows of ordinary heads are 0.
 *               Partial sums per batch element and block of 128 keys go to
 *               the workspace and are added in a fixed order: the result does
 *               not depend on scheduling.
 *   workspace : DEVICE, >= saf_hybrid_attn_bwd_pattern_workspace_bytes(),
 *               256-byte aligned, contents on entry ignored (about
 *               B * H * N^2 / 64 bytes: 25 MB at B = 8, H = 12, N = 4096).
 * Three launches: the row pre-pass D for the fixed heads, one workgroup per
 * (batch element, fixed head, block of 128 keys, chunk of query tiles), and
 * the reduction of the partial sums, which also writes the ordinary heads'
 * zeros (with no fixed head: two zero fills only).
 */
size_t saf_hybrid_attn_bwd_pattern_workspace_bytes(saf_dtype_t dt, int B, int H, int N, int d);

saf_status_t saf_hybrid_attn_bwd_pattern(saf_dtype_t dt,
                                         const void* V, const void* O, const void* dO,
                                         const float* LSE,
                                         const uint8_t* head_is_fixed,
                                         const float* a, const float* r, int ld_prior,
                                         int B, int H, int N, int d,
                                         float* da, float* dr,
                                         void* workspace, size_t workspace_bytes,
                                         hipStream_t stream);

/* Static text for a status code ("unknown status" for anything else). */
const char* saf_status_str(saf_status_t s);

#ifdef __cplusplus
}
#endif

#endif /* SAF_H */
