"""Pins for the compact-fit oracle (``oracle.fit_oracle``).

Checked against: central finite differences of Eq. fit-objective; torch
autograd of the same objective and torch.optim.Adam (a library special case of
the fitter's update); scipy's relative entropy for the acceptance KL; the
optimality property the paper states (at an optimum the fitted pattern
reproduces both target marginals) and the exact recovery of a target that is
itself a compact pattern; the closed form of the initialisation; and the
floor-and-renormalise construction of the target.
"""

import math

import numpy as np
import pytest
from scipy.stats import entropy

from oracle import fit_oracle as fo

RNG = np.random.default_rng(20261203)


def _compact(alpha, rho):
    L = fo.compact_logits(alpha, rho)
    L = L - L.max(axis=1, keepdims=True)
    P = np.exp(L)
    return P / P.sum(axis=1, keepdims=True)


def _random_target(T, sharp=2.0):
    """A causal row-stochastic pattern that is not compact."""
    S = RNG.standard_normal((T, T)) * sharp
    S[np.triu_indices(T, 1)] = -np.inf
    P = np.exp(S - S.max(axis=1, keepdims=True))
    return P / P.sum(axis=1, keepdims=True)


def test_targets_floor_and_renormalise():
    T = 12
    A = _random_target(T)
    A[5, 2] = 0.0  # an empty causal entry gets the floor
    t = fo.fit_targets(A)
    pi = t["Pi"]
    np.testing.assert_allclose(pi.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert pi[5, 2] > 0 and np.all(np.triu(pi, 1) == 0)
    np.testing.assert_allclose(pi[5, 2], 1e-9 / (A[5].sum() + 1e-9), rtol=1e-12)
    np.testing.assert_allclose(t["eta_abs"].sum(), T, rtol=1e-13)
    np.testing.assert_allclose(t["eta_rel"].sum(), T, rtol=1e-13)
    np.testing.assert_allclose(t["neg_entropy"], sum(-entropy(pi[i, : i + 1]) for i in range(T)), rtol=1e-12)


def test_objective_gradient_matches_finite_differences():
    T = 9
    t = fo.fit_targets(_random_target(T))
    a, r = RNG.standard_normal(T), RNG.standard_normal(T)
    _, ga, gr, _ = fo.fit_objective(a, r, t["eta_abs"], t["eta_rel"])
    eps = 1e-6
    for x, g in ((a, ga), (r, gr)):
        num = np.zeros(T)
        for k in range(T):
            old = x[k]
            x[k] = old + eps
            fp = fo.fit_objective(a, r, t["eta_abs"], t["eta_rel"])[0]
            x[k] = old - eps
            fm = fo.fit_objective(a, r, t["eta_abs"], t["eta_rel"])[0]
            x[k] = old
            num[k] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-10)
    # Shift invariance (a common constant absorbed by every row): the
    # gradients sum to zero.
    assert abs(ga.sum()) < 1e-14 and abs(gr.sum()) < 1e-14


def test_fitter_matches_torch_adam():
    """The fitter's steps equal torch.optim.Adam on the same objective (torch
    autograd through a dense float64 build of Eq. fit-objective)."""
    torch = pytest.importorskip("torch")
    T, steps = 10, 25
    t = fo.fit_targets(_random_target(T))
    a0 = np.zeros(T)
    r0 = np.log(np.maximum(t["eta_rel"] / (T - np.arange(T)), 1e-9))
    a = torch.tensor(a0, requires_grad=True)
    r = torch.tensor(r0, requires_grad=True)
    ea, er = torch.tensor(t["eta_abs"]), torch.tensor(t["eta_rel"])
    i = torch.arange(T)
    off = i[:, None] - i[None, :]
    opt = torch.optim.Adam([a, r], lr=fo.FIT_LR)
    for _ in range(steps):
        opt.zero_grad()
        L = (a[None, :] + r[off.clamp(min=0)]).masked_fill(off < 0, float("-inf"))
        obj = (torch.logsumexp(L, dim=1).sum() - (ea * a).sum() - (er * r).sum()) / T
        obj.backward()
        opt.step()
    fa, fr = fo.fit(t["eta_abs"], t["eta_rel"], steps=steps)
    np.testing.assert_allclose(fa, a.detach().numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(fr, r.detach().numpy(), rtol=1e-10, atol=1e-12)


def test_fit_reproduces_marginals_and_recovers_compact_targets():
    """The optimality condition of Appendix "Compact fitting and storage": at
    an optimum the fitted pattern has the target's marginals.  A target that
    is itself compact is recovered (KL to 0)."""
    T = 24
    a_true, r_true = RNG.standard_normal(T), -0.3 * np.arange(T) + 0.5 * RNG.standard_normal(T)
    t = fo.fit_targets(_compact(a_true, r_true), floor=0.0)
    a, r = fo.fit(t["eta_abs"], t["eta_rel"], steps=3000)
    P = _compact(a, r)
    np.testing.assert_allclose(P, t["Pi"], rtol=0, atol=2e-4)
    np.testing.assert_allclose(P.sum(axis=0), t["eta_abs"], rtol=0, atol=2e-3)
    assert fo.fit_kl(a, r, t["eta_abs"], t["eta_rel"], t["neg_entropy"]) < 1e-5


def test_acceptance_kl_equals_row_kl():
    T = 15
    t = fo.fit_targets(_random_target(T))
    a, r = fo.fit(t["eta_abs"], t["eta_rel"], steps=60)
    P = _compact(a, r)
    kl = sum(entropy(t["Pi"][i, : i + 1], P[i, : i + 1]) for i in range(T)) / T
    np.testing.assert_allclose(fo.fit_kl(a, r, t["eta_abs"], t["eta_rel"], t["neg_entropy"]), kl, rtol=1e-10)
    # More steps never make a convex fit worse at this learning rate here.
    a2, r2 = fo.fit(t["eta_abs"], t["eta_rel"], steps=400)
    assert fo.fit_kl(a2, r2, t["eta_abs"], t["eta_rel"], t["neg_entropy"]) <= kl + 1e-12


def test_initialisation_closed_form():
    """No step: alpha = 0, rho = log max(eta_rel / (T - delta), 1e-9).  For the
    uniform target Pi(i, j) = 1/(i+1), eta_rel(delta) = H_T - H_delta."""
    T = 8
    i = np.arange(T)
    U = np.where(i[None, :] <= i[:, None], 1.0 / (i[:, None] + 1.0), 0.0)
    t = fo.fit_targets(U, floor=0.0)
    harm = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, T + 1))])
    np.testing.assert_allclose(t["eta_rel"], harm[T] - harm[:T], rtol=1e-14)
    a, r = fo.fit(t["eta_abs"], t["eta_rel"], steps=0)
    assert not a.any()
    np.testing.assert_allclose(r, [math.log((harm[T] - harm[d]) / (T - d)) for d in range(T)], rtol=1e-14)


def test_fit_golden_file_invariants():
    """tests/golden/fit_golden.npz (written by make_fit_golden.py from the
    oracle) is self-consistent: each stored pattern row sums to one, the
    column and diagonal sums each total T, the stored log Z is the oracle's
    normaliser of the stored alpha and rho, and the KL is non-negative."""
    import os
    from oracle import fit_oracle as fo
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "fit_golden.npz")
    ref = np.load(path)
    keys = sorted({k.rsplit("_", 1)[0] for k in ref.files if k.endswith("_kl")})
    assert keys == ["t1024_h0", "t1024_h1", "t4096_h0"]
    for key in keys:
        T = ref[key + "_a"].shape[0]
        np.testing.assert_allclose(ref[key + "_P_rows"].sum(axis=1), 1.0, atol=1e-12)
        np.testing.assert_allclose(ref[key + "_col"].sum(), T, rtol=1e-12)
        np.testing.assert_allclose(ref[key + "_diag"].sum(), T, rtol=1e-12)
        assert float(ref[key + "_kl"]) >= 0.0
        if T <= 1024:
            rows = ref[key + "_rows"]
            L = fo.compact_logits(ref[key + "_a"], ref[key + "_r"])[rows]
            m = L.max(axis=1)
            lz = m + np.log(np.exp(L - m[:, None]).sum(axis=1))
            np.testing.assert_allclose(ref[key + "_logz"][rows], lz, rtol=0, atol=1e-12)
            np.testing.assert_allclose(ref[key + "_P_rows"], np.exp(L - lz[:, None]), rtol=0, atol=1e-15)
