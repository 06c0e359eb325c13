"""Pins for the calibration-statistics oracle.

The oracle's mean attention, variance score, forward-KL score and marginals
are checked against things other than itself: a scalar-loop softmax on tiny
inputs, numpy's per-entry sample variance (``ddof=1``) and scipy's relative
entropy (library special cases of Eqs. variance-score and forward-kl-score),
``numpy.trace`` for the relative-distance marginal, closed forms for uniform
attention (``Q = 0``) and for identical inputs, the two-input closed form of
the variance score, and the row-stochastic invariants the paper relies on
(every row of the target sums to one, so both marginals sum to ``T``).
"""

import math

import numpy as np
import pytest
from scipy.stats import entropy

from oracle import calib_oracle as co

RNG = np.random.default_rng(20261202)


def _inputs(N, H, T, d, scale=1.0):
    return RNG.standard_normal((N, H, T, d)) * scale, RNG.standard_normal((N, H, T, d)) * scale


def _loop_attention(q, k):
    """Scalar-loop causal softmax with the 1/sqrt(d) temperature."""
    T, d = k.shape
    A = np.zeros((T, T))
    for i in range(T):
        s = [sum(q[i, c] * k[j, c] for c in range(d)) / math.sqrt(d) for j in range(i + 1)]
        m = max(s)
        z = sum(math.exp(x - m) for x in s)
        for j in range(i + 1):
            A[i, j] = math.exp(s[j] - m) / z
    return A


def test_attention_matrix_matches_scalar_loops():
    Q, K = _inputs(1, 1, 7, 3, scale=1.5)
    np.testing.assert_allclose(co.attention_matrix(Q[0, 0], K[0, 0]), _loop_attention(Q[0, 0], K[0, 0]),
                               rtol=1e-13, atol=1e-15)


def test_scores_and_mean_against_library_routines():
    N, H, T, d = 4, 2, 9, 3
    Q, K = _inputs(N, H, T, d, scale=1.5)
    st = co.calibration_stats(Q, K, row_block=4)
    for h in range(H):
        A = np.stack([_loop_attention(Q[n, h], K[n, h]) for n in range(N)])
        np.testing.assert_allclose(st["A_mean"][h], A.mean(axis=0), rtol=1e-12, atol=1e-15)
        # Eq. variance-score: (1/T^2) * sum over entries of the sample variance.
        s_var = np.var(A, axis=0, ddof=1).sum() / (T * T)
        np.testing.assert_allclose(st["s_var"][h], s_var, rtol=1e-10)
        np.testing.assert_allclose(st["sq_dev"][h], np.var(A, axis=0, ddof=0) * N, rtol=1e-10, atol=1e-18)
        # Eq. forward-kl-score with scipy's KL of each causal row.
        Ahat = A.mean(axis=0)
        kl = sum(entropy(A[n, i, : i + 1], Ahat[i, : i + 1]) for n in range(N) for i in range(T))
        np.testing.assert_allclose(st["s_kl"][h], kl / (N * T), rtol=1e-10)
        np.testing.assert_allclose(st["eta_abs"][h], Ahat.sum(axis=0), rtol=1e-12)
        rel = np.array([np.trace(Ahat, offset=-delta) for delta in range(T)])
        np.testing.assert_allclose(st["eta_rel"][h], rel, rtol=1e-12)


def test_two_inputs_closed_form():
    """With N = 2 the deviations are +-(A1 - A2)/2, so
    s_var = ||A1 - A2||_F^2 / (2 T^2)."""
    N, H, T, d = 2, 1, 8, 4
    Q, K = _inputs(N, H, T, d, scale=2.0)
    st = co.calibration_stats(Q, K)
    A1, A2 = (_loop_attention(Q[n, 0], K[n, 0]) for n in range(2))
    np.testing.assert_allclose(st["s_var"][0], np.sum((A1 - A2) ** 2) / (2 * T * T), rtol=1e-10)


def test_uniform_attention_closed_form():
    """Q = 0 gives A(i, j) = 1/(i+1) for every input: no variance, no KL, and
    harmonic-number marginals eta_abs(j) = H_T - H_j, eta_rel(delta) = H_T - H_delta
    (H_m = 1 + 1/2 + ... + 1/m)."""
    N, H, T, d = 3, 2, 11, 4
    _, K = _inputs(N, H, T, d)
    Q = np.zeros_like(K)
    st = co.calibration_stats(Q, K, row_block=3)
    harm = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, T + 1))])
    i = np.arange(T)
    uniform = np.where(i[None, :] <= i[:, None], 1.0 / (i[:, None] + 1.0), 0.0)
    for h in range(H):
        np.testing.assert_allclose(st["A_mean"][h], uniform, rtol=1e-14, atol=0)
        np.testing.assert_allclose(st["eta_abs"][h], harm[T] - harm[:T], rtol=1e-13)
        np.testing.assert_allclose(st["eta_rel"][h], harm[T] - harm[:T], rtol=1e-13)
    np.testing.assert_allclose(st["s_var"], 0.0, atol=1e-30)
    np.testing.assert_allclose(st["s_kl"], 0.0, atol=1e-15)


def test_identical_inputs_have_zero_scores():
    N, H, T, d = 5, 2, 10, 4
    Q1, K1 = _inputs(1, H, T, d, scale=2.0)
    Q, K = np.repeat(Q1, N, axis=0), np.repeat(K1, N, axis=0)
    st = co.calibration_stats(Q, K)
    np.testing.assert_allclose(st["s_var"], 0.0, atol=1e-30)
    np.testing.assert_allclose(st["s_kl"], 0.0, atol=1e-15)
    for h in range(H):
        np.testing.assert_allclose(st["A_mean"][h], _loop_attention(Q1[0, h], K1[0, h]), rtol=1e-12, atol=1e-15)


def test_marginals_sum_to_sequence_length_and_rows_are_stochastic():
    N, H, T, d = 3, 2, 33, 8
    Q, K = _inputs(N, H, T, d, scale=1.5)
    st = co.calibration_stats(Q, K, row_block=10)
    np.testing.assert_allclose(st["A_mean"].sum(axis=2), 1.0, rtol=0, atol=1e-12)
    assert np.all(np.triu(st["A_mean"], 1) == 0)
    np.testing.assert_allclose(st["eta_abs"].sum(axis=1), T, rtol=1e-12)
    np.testing.assert_allclose(st["eta_rel"].sum(axis=1), T, rtol=1e-12)
    assert np.all(st["s_var"] > 0) and np.all(st["s_kl"] > 0)


def test_row_subsets_add_up():
    """Every statistic is a sum over query rows: two disjoint row subsets give
    the full result."""
    N, H, T, d = 3, 1, 17, 4
    Q, K = _inputs(N, H, T, d, scale=1.5)
    full = co.calibration_stats(Q, K)
    even, odd = np.arange(0, T, 2), np.arange(1, T, 2)
    a, b = co.calibration_stats(Q, K, rows=even), co.calibration_stats(Q, K, rows=odd)
    for key in ("s_var", "s_kl", "eta_abs", "eta_rel"):
        np.testing.assert_allclose(a[key] + b[key], full[key], rtol=1e-12, atol=1e-16)
    for key in ("A_mean", "sq_dev"):
        np.testing.assert_allclose(a[key][0], full[key][0][even], rtol=0, atol=0)
        np.testing.assert_allclose(b[key][0], full[key][0][odd], rtol=0, atol=0)


def test_single_input_variance_is_undefined():
    Q, K = _inputs(1, 1, 5, 2)
    st = co.calibration_stats(Q, K)
    assert np.isnan(st["s_var"][0])
    assert st["s_kl"][0] == 0.0


def test_calib_golden_file_invariants():
    """tests/golden/calib124m_4k_head0.npz (written by
    make_calib124m_head0.py from the oracle) is self-consistent: both
    marginals of the mean attention total T, the stored mean rows are
    row-stochastic and causal, and both scores are positive."""
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "calib124m_4k_head0.npz")
    ref = np.load(path)
    T = ref["eta_abs"].shape[0]
    assert T == 4096
    np.testing.assert_allclose(ref["eta_abs"].sum(), T, rtol=1e-12)
    np.testing.assert_allclose(ref["eta_rel"].sum(), T, rtol=1e-12)
    rows = ref["rows"]
    np.testing.assert_allclose(ref["A_mean_rows"].sum(axis=1), 1.0, atol=1e-12)
    for li, i in enumerate(rows):
        assert not ref["A_mean_rows"][li, i + 1:].any()
    assert float(ref["s_var"]) > 0 and float(ref["s_kl"]) > 0
