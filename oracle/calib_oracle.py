"""Plain fp64 CPU oracle for the calibration statistics of Selective Attention
Freezing ("When Can Attention Heads Be Statically Defined?").

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import or call this module.
The GPU product path never imports it, and this module imports nothing from
the product package.

At the replacement checkpoint the method runs the model on ``N`` calibration
sequences and, for every head, measures (Section "Calibration and head
selection"; Algorithm "calibration", its measuring step):

* the empirical mean attention ``A_hat = (1/N) sum_n A^(n)``, where
  ``A^(n) = softmax_causal(Q_n K_n^T / sqrt(d_h))`` is the head's causal
  attention matrix on input ``n`` (diagonal visible);
* the attention-variance score (Eq. variance-score)
  ``s_var = 1 / ((N - 1) T^2) * sum_n ||A^(n) - A_hat||_F^2``;
* the forward-KL score (Eq. forward-kl-score)
  ``s_KL = 1 / (N T) * sum_n sum_i KL(A^(n)[i, :i+1] || A_hat[i, :i+1])``;
* the marginals of the target pattern ``A_hat`` that are the sufficient
  statistics of the compact fit (Section "Fixed-pattern construction and
  fitting", Eq. fit-objective): ``eta_abs(j) = sum_{i >= j} A_hat(i, j)`` and
  ``eta_rel(delta) = sum_{i - j = delta} A_hat(i, j)``.

Everything is the dense definition in float64, materialising every
``A^(n)``.  Query rows are independent, so each function may evaluate rows in
blocks (``row_block``) or only a listed subset of rows (``rows``): every
statistic is a sum over rows, and a subset gives that subset's share exactly.

Readings of points the paper leaves open:

* Indices are 0-based: query ``i`` and key ``j`` in ``0..T-1``, offset
  ``delta = i - j`` in ``0..T-1``.
* ``0 log 0 = 0`` in the KL sums (entries that underflow to zero or are
  masked contribute nothing).
* With a single calibration input ``s_var`` is 0/0 and is returned as NaN.
"""

from __future__ import annotations

import math
from typing import Dict, Optional

import numpy as np
from scipy.special import xlogy

__all__ = ["attention_matrix", "calibration_stats"]

_F64 = np.float64


def attention_matrix(q, k, rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Causal attention weights ``softmax(q_i . k_j / sqrt(d))`` over
    ``j <= i`` for the query rows ``rows`` (all rows by default); zeros above
    the diagonal (Eqs. standard-head)."""
    q = np.asarray(q, dtype=_F64)
    k = np.asarray(k, dtype=_F64)
    T, d = k.shape
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    s = (q[rows] @ k.T) / math.sqrt(d)
    s[np.arange(T)[None, :] > rows[:, None]] = -np.inf
    m = np.max(s, axis=1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=1, keepdims=True)


def calibration_stats(Q, K, rows: Optional[np.ndarray] = None,
                      row_block: int = 256) -> Dict[str, np.ndarray]:
    """Calibration statistics of every head from ``Q, K`` ``[N, H, T, d]``
    (calibration input, head, position, channel).

    Returns a dict of float64 arrays:

    * ``A_mean`` ``[H, R, T]``: rows ``rows`` of ``A_hat`` (``R = T`` rows by
      default);
    * ``sq_dev`` ``[H, R, T]``: per entry, ``sum_n (A^(n) - A_hat)^2`` (the
      sample variance of the entry times ``N - 1``);
    * ``s_var`` ``[H]``, ``s_kl`` ``[H]``: the two scores, summed over the
      evaluated rows only (the full scores when every row is evaluated);
    * ``eta_abs`` ``[H, T]``, ``eta_rel`` ``[H, T]``: the marginals, summed over
      the evaluated rows only.
    """
    Q = np.asarray(Q)
    K = np.asarray(K)
    N, H, T, _ = Q.shape
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64).reshape(-1)
    R = rows.shape[0]
    A_mean = np.zeros((H, R, T))
    sq_ent = np.zeros((H, R, T))
    sq_dev = np.zeros(H)       # sum_n ||A^(n) - A_hat||^2 over the rows
    kl_sum = np.zeros(H)       # sum_n sum_i KL(A^(n)[i] || A_hat[i]) over the rows
    eta_abs = np.zeros((H, T))
    eta_rel = np.zeros((H, T))
    for h in range(H):
        for start in range(0, R, row_block):
            sel = slice(start, min(R, start + row_block))
            r_blk = rows[sel]
            A = np.stack([attention_matrix(Q[n, h], K[n, h], r_blk) for n in range(N)])  # [N, rb, T]
            mean = A.mean(axis=0)
            A_mean[h, sel] = mean
            sq_ent[h, sel] = np.sum((A - mean[None]) ** 2, axis=0)
            sq_dev[h] += np.sum(sq_ent[h, sel])
            # KL(p || q) = sum p log p - sum p log q, with 0 log 0 = 0.
            kl_sum[h] += np.sum(xlogy(A, A)) - np.sum(xlogy(A, np.broadcast_to(mean, A.shape)))
            eta_abs[h] += mean.sum(axis=0)
            for li, i in enumerate(r_blk):
                # Row i holds offsets delta = i - j for j = 0..i.
                eta_rel[h, : i + 1] += mean[li, i::-1]
    s_var = sq_dev / ((N - 1) * T * T) if N > 1 else np.full(H, np.nan)
    s_kl = kl_sum / (N * T)
    return {"A_mean": A_mean, "sq_dev": sq_ent, "s_var": s_var, "s_kl": s_kl, "eta_abs": eta_abs,
            "eta_rel": eta_rel}
