/*
 * saf_calib.h -- C ABI of libsaf.so for the calibration statistics of
 * Selective Attention Freezing ("When Can Attention Heads Be Statically
 * Defined?"), for AMD Instinct MI355X (gfx950).
 *
 * Before replacing heads, the method runs the model on N calibration inputs
 * and measures, for every head of a layer (Section "Calibration and head
 * selection"; Algorithm "calibration", its measuring step):
 *   - the empirical mean attention  A_hat = (1/N) sum_n A^(n),  where
 *     A^(n) = softmax_causal(Q_n K_n^T / sqrt(d)) is the head's causal
 *     attention matrix on input n (diagonal visible);
 *   - the attention-variance score (Eq. variance-score)
 *       s_var = sum_n ||A^(n) - A_hat||_F^2 / ((N - 1) T^2);
 *   - the forward-KL score (Eq. forward-kl-score)
 *       s_KL = (1 / (N T)) sum_n sum_i KL(A^(n)[i, 0..i] || A_hat[i, 0..i]);
 *   - the marginals of the target pattern A_hat, the sufficient statistics
 *     of the compact fit (Eq. fit-objective):
 *       eta_abs(j) = sum_{i >= j} A_hat(i, j),
 *       eta_rel(delta) = sum_{i - j = delta} A_hat(i, j).
 * The calibration inputs arrive in micro-batches.  saf_calib_accumulate folds
 * one micro-batch into a running state without ever writing a per-input
 * T x T matrix; saf_calib_finalize turns the state into the scores and
 * marginals.  The state after the last micro-batch holds A_hat itself.
 *
 * Conventions are those of saf.h (caller-owned DEVICE buffers, no
 * allocation, no synchronisation, arguments checked before anything is
 * enqueued, status codes from saf_status_t).  Indices are 0-based: query i,
 * key j, offset delta = i - j.
 *
 * Running state of one layer (caller-owned DEVICE buffers):
 *   mean  : [H, T, T] float32, row-major (query, key): the mean of A over the
 *           inputs folded in so far; entries above the diagonal are 0.
 *   m2    : optional [H, T, T] float32: per entry, the sum over those inputs
 *           of the squared deviation from their mean (the per-entry sample
 *           variance is m2 / (n - 1)).  Pass NULL to skip it: the scores do
 *           not need it, and keeping it doubles the memory traffic.
 *   stats : saf_calib_stats_bytes(H, T) bytes of float64 partial sums, per
 *           head and 128 x 128 tile of the attention matrix: the sum over
 *           those inputs of A ln A over the tile (0 ln 0 = 0) and the tile's
 *           sum of squared deviations.  Its layout is private to the library;
 *           saf_calib_finalize reads it.
 * Limits: d == 64, 1 <= H <= 64, T <= 65536, n_seen + B <= 2^24.
 */
#ifndef SAF_CALIB_H
#define SAF_CALIB_H

#include "saf.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Fold one micro-batch of B calibration inputs into the running state.
 *   Q, K  : DEVICE [B, H, T, d] `dt`, 16-byte aligned: the layer's queries and
 *           keys on these inputs (every head ordinary, as before replacement).
 *   LSE   : DEVICE [B, H, T] float32: the natural-log row normalisers of the
 *           same attention, as saf_hybrid_attn_fwd writes them with every head
 *           ordinary.  The weights are recomputed as exp(S - LSE).
 *   n_seen: inputs already folded into the state.  0 starts a new state:
 *           mean, m2 (if kept) and stats are then written in full and their
 *           previous contents ignored.
 *   mean, m2 (16-byte aligned; m2 may be NULL), stats (8-byte aligned): the
 *           state, updated.  Whether m2 is kept must not change between the
 *           calls of one state.
 * Per entry the mean follows Welford's recurrence over the inputs in order,
 * so the mean after several calls is bitwise the mean after one call over the
 * same inputs.  One launch per micro-batch; no atomics, so the state does not
 * depend on the order in which workgroups run.
 */
saf_status_t saf_calib_accumulate(saf_dtype_t dt,
                                  const void* Q, const void* K, const float* LSE,
                                  int B, int H, int T, int d, int n_seen,
                                  float* mean, float* m2, double* stats,
                                  hipStream_t stream);

/* Bytes of the stats buffer of a state (a multiple of 256); 0 for an invalid
 * problem. */
size_t saf_calib_stats_bytes(int H, int T);

/* Bytes of device workspace saf_calib_finalize needs (a multiple of 256);
 * 0 for an invalid problem. */
size_t saf_calib_finalize_workspace_bytes(int H, int T);

/*
 * Scores and marginals from the state after n_total inputs (n_total >= 1).
 *   eta_abs, eta_rel : DEVICE [H, T] float32, written.
 *   s_var, s_kl      : DEVICE [H] float32, written; s_var is NaN when
 *                      n_total == 1 (the sample variance needs two inputs).
 *   workspace        : DEVICE, >= saf_calib_finalize_workspace_bytes(),
 *                      256-byte aligned, contents on entry ignored.
 * Four launches: two zero fills, one pass over the lower triangle of the
 * mean, and a per-head reduction.  The marginals gather partial sums over
 * 256-row chunks with float32 atomic adds, so their last bits may depend on
 * the order in which workgroups finish; the scores are reduced in float64
 * without atomics.
 */
saf_status_t saf_calib_finalize(int H, int T, int n_total,
                                const float* mean, const double* stats,
                                float* eta_abs, float* eta_rel, float* s_var, float* s_kl,
                                void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SAF_CALIB_H */
