"""Plain fp64 CPU oracle for the compact fit of Selective Attention Freezing
("When Can Attention Heads Be Statically Defined?").

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import or call this module.
The GPU product path never imports it, and this module imports nothing from
the product package.

The method fits the compact pattern of Eq. compact-prior,
``P_hat(i, j) = exp(alpha(j) + rho(i - j)) / Z(i)`` for ``j <= i``, to a target
causal row-stochastic pattern ``Pi`` (Section "Fixed-pattern construction and
fitting"; Algorithm "calibration"; Appendix "Compact fitting and storage"):

* target: the mean attention with its causal entries floored at ``1e-9`` and
  each row renormalised;
* sufficient statistics: ``eta_abs(j) = sum_{i >= j} Pi(i, j)`` and
  ``eta_rel(delta) = sum_{i - j = delta} Pi(i, j)``;
* objective (Eq. fit-objective), row-averaged cross-entropy:
  ``L = (1/T) [sum_i log Z(i) - sum_j eta_abs(j) alpha(j) - sum_delta eta_rel(delta) rho(delta)]``,
  with gradient ``(column sums of P_hat - eta_abs) / T`` for alpha and
  ``(diagonal sums of P_hat - eta_rel) / T`` for rho;
* fitter: ``alpha = 0``, ``rho(delta) = log max(eta_rel(delta) / (T - delta), 1e-9)``,
  then ``J = 400`` Adam steps at learning rate ``0.05``, no early stopping;
* acceptance: the row-averaged KL ``(1/T) sum_i KL(Pi[i] || P_hat[i])``
  must not exceed ``0.2`` nats; since every row of ``Pi`` sums to one it equals
  ``L + (1/T) sum_ij Pi log Pi``.

Everything is the dense definition in float64 (``P_hat`` materialised each
step).  Indices are 0-based: ``alpha(j)`` is ``a[j]``, ``rho(delta)`` is
``r[delta]``.

Readings of points the paper leaves open:

* Adam's other constants are the common defaults (Kingma and Ba):
  ``beta1 = 0.9``, ``beta2 = 0.999``, ``epsilon = 1e-8``, bias-corrected
  moments, the update ``theta -= lr * m_hat / (sqrt(v_hat) + epsilon)``.
* ``0 log 0 = 0`` in the target's entropy (floored targets have no zeros in
  the causal triangle).
"""

from __future__ import annotations

from typing import Dict, Tuple

import numpy as np
from scipy.special import xlogy

__all__ = ["fit_targets", "compact_logits", "fit_objective", "fit", "fit_kl", "FIT_STEPS", "FIT_LR",
           "FIT_FLOOR"]

FIT_STEPS = 400
FIT_LR = 0.05
FIT_FLOOR = 1e-9
ADAM_BETA1 = 0.9
ADAM_BETA2 = 0.999
ADAM_EPS = 1e-8


def _causal(T: int) -> np.ndarray:
    i = np.arange(T)
    return i[None, :] <= i[:, None]


def fit_targets(mean, floor: float = FIT_FLOOR) -> Dict[str, np.ndarray]:
    """Target pattern and its statistics from one head's mean attention
    ``[T, T]``: ``Pi`` (floored, row-renormalised), ``eta_abs``, ``eta_rel``
    and ``neg_entropy = sum_ij Pi log Pi``."""
    mean = np.asarray(mean, dtype=np.float64)
    T = mean.shape[0]
    mask = _causal(T)
    pi = np.where(mask, np.maximum(mean, floor), 0.0)
    pi /= pi.sum(axis=1, keepdims=True)
    eta_abs = pi.sum(axis=0)
    eta_rel = np.array([np.trace(pi, offset=-delta) for delta in range(T)])
    return {"Pi": pi, "eta_abs": eta_abs, "eta_rel": eta_rel, "neg_entropy": float(np.sum(xlogy(pi, pi)))}


def compact_logits(alpha, rho) -> np.ndarray:
    """``L(i, j) = alpha(j) + rho(i - j)`` for ``j <= i``, ``-inf`` above."""
    alpha = np.asarray(alpha, dtype=np.float64)
    rho = np.asarray(rho, dtype=np.float64)
    T = alpha.shape[0]
    i = np.arange(T)
    off = i[:, None] - i[None, :]
    L = alpha[None, :] + rho[np.clip(off, 0, None)]
    L[off < 0] = -np.inf
    return L


def fit_objective(alpha, rho, eta_abs, eta_rel) -> Tuple[float, np.ndarray, np.ndarray, np.ndarray]:
    """``(L, dL/dalpha, dL/drho, log Z)`` of Eq. fit-objective."""
    alpha = np.asarray(alpha, dtype=np.float64)
    rho = np.asarray(rho, dtype=np.float64)
    T = alpha.shape[0]
    L = compact_logits(alpha, rho)
    m = L.max(axis=1)
    logz = m + np.log(np.exp(L - m[:, None]).sum(axis=1))
    obj = (logz.sum() - np.dot(eta_abs, alpha) - np.dot(eta_rel, rho)) / T
    P = np.exp(L - logz[:, None])
    g_alpha = (P.sum(axis=0) - eta_abs) / T
    g_rho = (np.array([np.trace(P, offset=-delta) for delta in range(T)]) - eta_rel) / T
    return float(obj), g_alpha, g_rho, logz


def fit(eta_abs, eta_rel, steps: int = FIT_STEPS, lr: float = FIT_LR) -> Tuple[np.ndarray, np.ndarray]:
    """The fitter: initialisation, then ``steps`` Adam steps on Eq.
    fit-objective.  Returns ``(alpha, rho)``."""
    eta_abs = np.asarray(eta_abs, dtype=np.float64)
    eta_rel = np.asarray(eta_rel, dtype=np.float64)
    T = eta_abs.shape[0]
    alpha = np.zeros(T)
    rho = np.log(np.maximum(eta_rel / (T - np.arange(T)), FIT_FLOOR))
    theta = [alpha, rho]
    m = [np.zeros(T), np.zeros(T)]
    v = [np.zeros(T), np.zeros(T)]
    for t in range(1, steps + 1):
        _, ga, gr, _ = fit_objective(theta[0], theta[1], eta_abs, eta_rel)
        for k, g in enumerate((ga, gr)):
            m[k] = ADAM_BETA1 * m[k] + (1.0 - ADAM_BETA1) * g
            v[k] = ADAM_BETA2 * v[k] + (1.0 - ADAM_BETA2) * g * g
            m_hat = m[k] / (1.0 - ADAM_BETA1 ** t)
            v_hat = v[k] / (1.0 - ADAM_BETA2 ** t)
            theta[k] = theta[k] - lr * m_hat / (np.sqrt(v_hat) + ADAM_EPS)
    return theta[0], theta[1]


def fit_kl(alpha, rho, eta_abs, eta_rel, neg_entropy: float) -> float:
    """Row-averaged KL of the target from the fitted pattern:
    ``L + neg_entropy / T``."""
    T = np.asarray(alpha).shape[0]
    obj, _, _, _ = fit_objective(alpha, rho, eta_abs, eta_rel)
    return obj + neg_entropy / T
