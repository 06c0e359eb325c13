/*
 * saf_fit.h -- C ABI of libsaf.so for the compact fit of Selective Attention
 * Freezing ("When Can Attention Heads Be Statically Defined?"), for AMD
 * Instinct MI355X (gfx950).
 *
 * A replaced head's pattern is the compact form of Eq. compact-prior,
 *     P(i, j) = exp(a[j] + r[i - j]) / Z(i),  j <= i,
 * fitted to a target pattern Pi by minimising the row-averaged
 * cross-entropy of Eq. fit-objective,
 *     L(a, r) = (1/T) [ sum_i log Z(i) - sum_j eta_abs(j) a[j] - sum_d eta_rel(d) r[d] ],
 * whose sufficient statistics are the target's marginals eta_abs(j) =
 * sum_{i >= j} Pi(i, j) and eta_rel(d) = sum_{i - j = d} Pi(i, j) (Section
 * "Fixed-pattern construction and fitting").  The fitter follows the paper's
 * recipe (Algorithm "calibration" and the paragraph after it): the target is
 * the calibration mean with its causal entries floored at 1e-9 and its rows
 * renormalised; a = 0 and r[d] = log max(eta_rel(d) / (T - d), 1e-9) to start;
 * then J = 400 Adam steps at learning rate 0.05, no early stopping (Adam's
 * other constants: beta1 = 0.9, beta2 = 0.999, epsilon = 1e-8); a fit is
 * accepted when the row-averaged KL of the target from the fit is at most
 * 0.2 nats.  The gradient is (column sums of P - eta_abs) / T for a and
 * (diagonal sums of P - eta_rel) / T for r (Appendix "Compact fitting and
 * storage").  Indices are 0-based: a[j] = alpha(j+1), r[d] = rho(d).
 *
 * Conventions are those of saf.h (caller-owned DEVICE buffers, no
 * allocation, no synchronisation, arguments checked before anything is
 * enqueued, status codes from saf_status_t).  All heads of a layer are
 * fitted together.  Limits: 1 <= H <= 64, T <= 65536.
 */
#ifndef SAF_FIT_H
#define SAF_FIT_H

#include "saf.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Bytes of device workspace saf_fit_targets and saf_compact_fit need (a
 * multiple of 256); 0 for an invalid problem. */
size_t saf_fit_workspace_bytes(int H, int T);

/*
 * Targets from the calibration mean.
 *   mean        : DEVICE [H, T, T] float32, row-major (query, key), as
 *                 saf_calib_accumulate leaves it; only j <= i is read.
 *   floor_value : the floor of the causal entries (the paper's 1e-9).
 *   eta_abs, eta_rel : DEVICE [H, T] float32, written.
 *   neg_entropy : DEVICE [H] float64, written: sum_ij Pi ln Pi.
 * Four launches.  The marginals gather 256-row partial sums with float32
 * atomic adds (their last bits may depend on scheduling).
 */
saf_status_t saf_fit_targets(int H, int T, const float* mean, float floor_value,
                             float* eta_abs, float* eta_rel, double* neg_entropy,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * The fitter: initialisation and `steps` Adam steps at learning rate `lr`,
 * then the acceptance KL.
 *   eta_abs, eta_rel, neg_entropy : as saf_fit_targets writes them.
 *   floor_value : the floor of the initial r (the paper's 1e-9).
 *   a, r        : DEVICE [H, T] float32, written: the fitted preference
 *                 vectors, ready for saf_hybrid_attn_fwd (ld_prior = T).
 *   log_z       : DEVICE [H, T] float32, written: log Z(i) of the fit; may
 *                 be NULL.
 *   kl          : DEVICE [H] float32, written: the row-averaged KL (nats) of
 *                 the target from the fit.
 * Three launches per step plus four; float32 arithmetic (the sums behind the
 * KL in float64).
 */
saf_status_t saf_compact_fit(int H, int T, const float* eta_abs, const float* eta_rel,
                             const double* neg_entropy, int steps, float lr, float floor_value,
                             float* a, float* r, float* log_z, float* kl,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SAF_FIT_H */
