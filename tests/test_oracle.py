"""Pins for the fp64 CPU oracle.

The oracle is the reference the GPU kernels are held to, so it is checked
here against things other than itself: closed forms that Eq. compact-prior
reduces to, a 1-based brute-force evaluation of that equation on tiny inputs,
PyTorch's own causal attention and autograd (a library special case for
ordinary heads), central finite differences of the loss ``sum(O * dO)``, and
invariants the paper states (row normalisation absorbs additive shifts;
fixed heads read neither queries nor keys).
"""

import math

import numpy as np
import pytest

from oracle import saf_oracle as orc

RNG = np.random.default_rng(20260101)


def _rand(*shape):
    return RNG.standard_normal(shape)


# ---------------------------------------------------------------------------
# Fixed-head pattern (Eq. compact-prior)
# ---------------------------------------------------------------------------

def test_pattern_is_causal_and_row_stochastic():
    n = 40
    a, r = _rand(n) * 3, _rand(n) * 3
    P = orc.fixed_pattern(a, r)
    assert np.all(P >= 0)
    assert np.all(np.triu(P, 1) == 0)
    np.testing.assert_allclose(P.sum(axis=1), 1.0, rtol=0, atol=1e-12)
    assert np.all(np.diag(P) > 0)


def test_brute_force_one_based_definition():
    """Eq. compact-prior written with the paper's 1-based alpha(1..T) and
    rho(0..T-1), evaluated with scalar loops, against the oracle's 0-based
    storage a[j] = alpha(j+1), r[delta] = rho(delta)."""
    T, d = 9, 3
    alpha = {k: float(x) for k, x in zip(range(1, T + 1), _rand(T))}
    rho = {k: float(x) for k, x in zip(range(0, T), _rand(T))}
    V = _rand(T, d)
    P_ref = np.zeros((T, T))
    for i in range(1, T + 1):
        Z = sum(math.exp(alpha[k] + rho[i - k]) for k in range(1, i + 1))
        for j in range(1, i + 1):
            P_ref[i - 1, j - 1] = math.exp(alpha[j] + rho[i - j]) / Z
    a = np.array([alpha[j] for j in range(1, T + 1)])
    r = np.array([rho[k] for k in range(T)])
    np.testing.assert_allclose(orc.fixed_pattern(a, r), P_ref, rtol=1e-13, atol=1e-15)
    o, lse = orc.head_forward(None, None, V, True, a, r)
    o_ref = np.array([[sum(P_ref[i, j] * V[j, c] for j in range(T)) for c in range(d)]
                      for i in range(T)])
    np.testing.assert_allclose(o, o_ref, rtol=1e-12, atol=1e-14)
    lse_ref = [math.log(sum(math.exp(alpha[k] + rho[i - k]) for k in range(1, i + 1)))
               for i in range(1, T + 1)]
    np.testing.assert_allclose(lse, lse_ref, rtol=1e-13)


def test_uniform_closed_form():
    """a = c1, r = c2: every visible key gets weight 1/(i+1)."""
    n, d = 33, 5
    c1, c2 = 0.7, -1.9
    a, r = np.full(n, c1), np.full(n, c2)
    V, dO = _rand(n, d), _rand(n, d)
    o, lse = orc.head_forward(None, None, V, True, a, r)
    counts = np.arange(1, n + 1)[:, None]
    np.testing.assert_allclose(o, np.cumsum(V, axis=0) / counts, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(lse, np.log(np.arange(1, n + 1)) + c1 + c2, rtol=1e-13)
    dq, dk, dv = orc.head_backward(None, None, V, dO, True, a, r)
    w = dO / counts                                  # dO_i / (i + 1)
    dv_ref = np.cumsum(w[::-1], axis=0)[::-1]         # sum over i >= j
    np.testing.assert_allclose(dv, dv_ref, rtol=1e-12, atol=1e-14)
    assert not dq.any() and not dk.any()


def test_identity_closed_form():
    n, d = 20, 4
    a = _rand(n)
    r = np.full(n, -1e4)
    r[0] = 0.0
    V, dO = _rand(n, d), _rand(n, d)
    o, lse = orc.head_forward(None, None, V, True, a, r)
    np.testing.assert_allclose(o, V, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(lse, a, rtol=1e-13, atol=1e-15)
    _, _, dv = orc.head_backward(None, None, V, dO, True, a, r)
    np.testing.assert_allclose(dv, dO, rtol=1e-13, atol=1e-15)


def test_geometric_normaliser_closed_form():
    n, lam = 64, 0.3
    a = np.zeros(n)
    r = -lam * np.arange(n)
    i = np.arange(n)
    Z = (1 - np.exp(-lam * (i + 1))) / (1 - np.exp(-lam))
    np.testing.assert_allclose(orc.fixed_log_normaliser(a, r), np.log(Z), rtol=1e-13)


def test_absolute_only_is_prefix_softmax():
    """r constant: P(i, j) = exp(a_j) / sum_{k<=i} exp(a_k), so O is a ratio of
    running sums."""
    n, d = 50, 6
    a, r = _rand(n) * 2, np.full(n, 0.4)
    V = _rand(n, d)
    ea = np.exp(a)
    o_ref = np.cumsum(ea[:, None] * V, axis=0) / np.cumsum(ea)[:, None]
    o, lse = orc.head_forward(None, None, V, True, a, r)
    np.testing.assert_allclose(o, o_ref, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(lse, np.log(np.cumsum(ea)) + 0.4, rtol=1e-13)


def test_relative_only_is_causal_convolution():
    """a constant: P(i, j) = exp(r_{i-j}) / sum_{delta<=i} exp(r_delta), i.e. a
    normalised causal convolution of V with exp(r)."""
    n, d = 45, 3
    a, r = np.full(n, -0.8), _rand(n) * 2
    V = _rand(n, d)
    er = np.exp(r)
    num = np.stack([np.convolve(er, V[:, c])[:n] for c in range(d)], axis=1)
    o_ref = num / np.cumsum(er)[:, None]
    o, _ = orc.head_forward(None, None, V, True, a, r)
    np.testing.assert_allclose(o, o_ref, rtol=1e-12, atol=1e-14)


def test_shift_invariance_of_pattern():
    """Additive shifts of a and r are absorbed by row normalisation: O and dV
    are unchanged and LSE moves by c1 + c2.  c1 = 100 would overflow a naive
    float32 exp."""
    n, d = 37, 4
    a, r = _rand(n), _rand(n)
    V, dO = _rand(n, d), _rand(n, d)
    o0, l0 = orc.head_forward(None, None, V, True, a, r)
    o1, l1 = orc.head_forward(None, None, V, True, a + 100.0, r - 3.0)
    np.testing.assert_allclose(o1, o0, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l1, l0 + 97.0, rtol=1e-13)
    dv0 = orc.head_backward(None, None, V, dO, True, a, r)[2]
    dv1 = orc.head_backward(None, None, V, dO, True, a + 100.0, r - 3.0)[2]
    np.testing.assert_allclose(dv1, dv0, rtol=1e-12, atol=1e-13)


def test_prior_prefix_is_used_when_longer():
    n, L, d = 17, 30, 3
    a, r = _rand(L), _rand(L)
    V = _rand(n, d)
    o_long, _ = orc.head_forward(None, None, V, True, a, r)
    o_cut, _ = orc.head_forward(None, None, V, True, a[:n], r[:n])
    np.testing.assert_array_equal(o_long, o_cut)


# ---------------------------------------------------------------------------
# Ordinary head: library special case and cross-path identity
# ---------------------------------------------------------------------------

def test_ordinary_matches_torch_causal_attention_and_autograd():
    torch = pytest.importorskip("torch")
    import torch.nn.functional as F
    B, H, N, d = 2, 3, 29, 8
    Q, K, V, dO = (_rand(B, H, N, d) for _ in range(4))
    is_fixed = np.zeros(H, dtype=np.uint8)
    O, LSE = orc.layer_forward(Q, K, V, is_fixed)
    dQ, dK, dV = orc.layer_backward(Q, K, V, dO, is_fixed)
    q, k, v = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (Q, K, V))
    o = F.scaled_dot_product_attention(q, k, v, is_causal=True)
    o.backward(torch.tensor(dO))
    np.testing.assert_allclose(O, o.detach().numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dQ, q.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dK, k.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dV, v.grad.numpy(), rtol=1e-10, atol=1e-11)
    # Row 0 sees only key 0: LSE_0 = q0.k0/sqrt(d) and O_0 = V_0.
    np.testing.assert_allclose(LSE[..., 0], np.sum(Q[..., 0, :] * K[..., 0, :], -1) / math.sqrt(d),
                               rtol=1e-13)
    np.testing.assert_allclose(O[..., 0, :], V[..., 0, :], rtol=1e-13)


def test_zero_query_ordinary_equals_uniform_fixed():
    """An ordinary head with Q = 0 has all scores 0 (uniform causal average),
    as does a fixed head with a = r = 0; LSE is log(i+1) for both."""
    n, d = 31, 8
    K, V, dO = _rand(n, d), _rand(n, d), _rand(n, d)
    o_ord, l_ord = orc.head_forward(np.zeros((n, d)), K, V, False)
    o_fix, l_fix = orc.head_forward(None, None, V, True, np.zeros(n), np.zeros(n))
    np.testing.assert_allclose(o_ord, o_fix, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l_ord, np.log(np.arange(1, n + 1)), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(l_fix, l_ord, rtol=1e-13, atol=1e-15)
    dv_ord = orc.head_backward(np.zeros((n, d)), K, V, dO, False)[2]
    dv_fix = orc.head_backward(None, None, V, dO, True, np.zeros(n), np.zeros(n))[2]
    np.testing.assert_allclose(dv_ord, dv_fix, rtol=1e-12, atol=1e-14)


def test_cross_path_identity():
    """A fixed head with (a, r[delta] = -lam*delta) equals an ordinary head with
    q_i = (sqrt(d), 0, ...) and k_j = (a_j + lam*j, 0, ...): scores differ by
    the row constant -lam*i, so O and dV agree and LSE_ord = LSE_fix + lam*i."""
    n, d, lam = 26, 4, 0.35
    a = _rand(n)
    r = -lam * np.arange(n)
    q = np.zeros((n, d))
    q[:, 0] = math.sqrt(d)
    k = np.zeros((n, d))
    k[:, 0] = a + lam * np.arange(n)
    V, dO = _rand(n, d), _rand(n, d)
    o_f, l_f = orc.head_forward(None, None, V, True, a, r)
    o_o, l_o = orc.head_forward(q, k, V, False)
    np.testing.assert_allclose(o_o, o_f, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(l_o, l_f + lam * np.arange(n), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(orc.head_backward(q, k, V, dO, False)[2],
                               orc.head_backward(None, None, V, dO, True, a, r)[2],
                               rtol=1e-11, atol=1e-13)


# ---------------------------------------------------------------------------
# Backward: finite differences, autograd for fixed heads, identities
# ---------------------------------------------------------------------------

def _loss(Q, K, V, dO, is_fixed, a, r):
    O, _ = orc.layer_forward(Q, K, V, is_fixed, a, r)
    return float(np.sum(O * dO))


def test_backward_matches_central_finite_differences():
    B, H, N, d = 1, 2, 7, 3
    Q, K, V, dO = (_rand(B, H, N, d) for _ in range(4))
    a, r = _rand(H, N), _rand(H, N)
    is_fixed = np.array([0, 1], dtype=np.uint8)
    dQ, dK, dV = orc.layer_backward(Q, K, V, dO, is_fixed, a, r)
    eps = 1e-6
    for X, G in ((Q, dQ), (K, dK), (V, dV)):
        num = np.zeros_like(X)
        for idx in np.ndindex(X.shape):
            old = X[idx]
            X[idx] = old + eps
            fp = _loss(Q, K, V, dO, is_fixed, a, r)
            X[idx] = old - eps
            fm = _loss(Q, K, V, dO, is_fixed, a, r)
            X[idx] = old
            num[idx] = (fp - fm) / (2 * eps)
        err = np.linalg.norm(G - num) / np.linalg.norm(num)
        assert err < 1e-7, err
    # The fixed head's query/key gradients are exactly zero.
    assert not dQ[:, 1].any() and not dK[:, 1].any()
    assert np.abs(dQ[:, 0]).max() > 0 and np.abs(dK[:, 0]).max() > 0


def test_fixed_value_gradient_matches_autograd():
    torch = pytest.importorskip("torch")
    n, d = 23, 5
    a, r = _rand(n), _rand(n)
    V, dO = _rand(n, d), _rand(n, d)
    P = torch.tensor(orc.fixed_pattern(a, r))
    v = torch.tensor(V, requires_grad=True)
    (P @ v).backward(torch.tensor(dO))
    dv = orc.head_backward(None, None, V, dO, True, a, r)[2]
    np.testing.assert_allclose(dv, v.grad.numpy(), rtol=1e-12, atol=1e-14)


def test_delta_identity():
    """sum_j P_ij dP_ij (the oracle's D) equals rowsum(dO * O)."""
    n, d = 19, 6
    q, k, v, do = _rand(n, d), _rand(n, d), _rand(n, d), _rand(n, d)
    rows = np.arange(n)
    S = orc.ordinary_logits(q, k, rows)
    P = np.exp(S - np.max(S, axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    o, _ = orc.head_forward(q, k, v, False)
    np.testing.assert_allclose(np.sum(P * (do @ v.T), axis=1), np.sum(do * o, axis=1),
                               rtol=1e-12, atol=1e-13)


def test_pattern_gradient_matches_central_finite_differences():
    """Gradients of the trainable-pattern variant: da and dr of sum(O * dO),
    summed over the batch, against central differences of the loss in a and r."""
    B, H, N, d = 2, 2, 7, 3
    Q, K, V, dO = (_rand(B, H, N, d) for _ in range(4))
    a, r = _rand(H, N), _rand(H, N)
    is_fixed = np.array([1, 0], dtype=np.uint8)
    da, dr = orc.layer_pattern_grad(V, dO, is_fixed, a, r, row_block=3)
    eps = 1e-6
    for X, G in ((a, da), (r, dr)):
        num = np.zeros_like(X)
        for idx in np.ndindex(X.shape):
            old = X[idx]
            X[idx] = old + eps
            fp = _loss(Q, K, V, dO, is_fixed, a, r)
            X[idx] = old - eps
            fm = _loss(Q, K, V, dO, is_fixed, a, r)
            X[idx] = old
            num[idx] = (fp - fm) / (2 * eps)
        err = np.linalg.norm(G - num) / np.linalg.norm(num)
        assert err < 1e-7, err
    assert not da[1].any() and not dr[1].any()          # ordinary head: no pattern
    # A row's logits all shift with a common constant: the gradients sum to 0.
    np.testing.assert_allclose(da.sum(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose(dr.sum(axis=1), 0.0, atol=1e-12)


def test_pattern_gradient_matches_autograd():
    """Autograd through a dense torch float64 build of Eq. compact-prior."""
    torch = pytest.importorskip("torch")
    n, d = 21, 4
    a0, r0 = _rand(n) * 2, _rand(n) * 2
    V, dO = _rand(n, d), _rand(n, d)
    a = torch.tensor(a0, requires_grad=True)
    r = torch.tensor(r0, requires_grad=True)
    i = torch.arange(n)
    off = i[:, None] - i[None, :]
    logits = a[None, :] + r[off.clamp(min=0)]
    logits = logits.masked_fill(off < 0, float("-inf"))
    P = torch.softmax(logits, dim=1)
    (P @ torch.tensor(V)).backward(torch.tensor(dO))
    da, dr = orc.fixed_pattern_grad(V, dO, a0, r0, row_block=5)
    np.testing.assert_allclose(da, a.grad.numpy(), rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(dr, r.grad.numpy(), rtol=1e-11, atol=1e-13)


def test_pattern_gradient_of_uniform_values_is_zero():
    """V with identical rows gives O independent of the pattern: no gradient."""
    n, d = 15, 3
    V = np.tile(_rand(1, d), (n, 1))
    da, dr = orc.fixed_pattern_grad(V, _rand(n, d), _rand(n), _rand(n))
    np.testing.assert_allclose(da, 0.0, atol=1e-13)
    np.testing.assert_allclose(dr, 0.0, atol=1e-13)


def test_gqa_forward_equals_expanded_heads():
    """Grouped-query forward = the multi-head forward with each key/value head
    repeated for its group; with one query head per group it is the layer
    forward itself (and d = 96 uses 1/sqrt(96))."""
    B, Hq, Hkv, N, d = 2, 6, 2, 11, 96
    Q = _rand(B, Hq, N, d)
    K, V = _rand(B, Hkv, N, d), _rand(B, Hkv, N, d)
    a, r = _rand(Hq, N), _rand(Hq, N)
    is_fixed = np.array([0, 1, 0, 0, 1, 1], dtype=np.uint8)
    O, LSE = orc.layer_forward_gqa(Q, K, V, is_fixed, a, r)
    Ke, Ve = np.repeat(K, Hq // Hkv, axis=1), np.repeat(V, Hq // Hkv, axis=1)
    O2, LSE2 = orc.layer_forward(Q, Ke, Ve, is_fixed, a, r)
    np.testing.assert_allclose(O, O2, rtol=0, atol=0)
    np.testing.assert_allclose(LSE, LSE2, rtol=0, atol=0)
    # An ordinary head against torch's scaled_dot_product_attention at d = 96.
    torch = pytest.importorskip("torch")
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(Q[:, 0:1]), torch.tensor(K[:, 0:1]), torch.tensor(V[:, 0:1]), is_causal=True)
    np.testing.assert_allclose(O[:, 0:1], ref.numpy(), rtol=1e-12, atol=1e-13)


def test_gqa_backward_matches_autograd_of_expanded_heads():
    """Grouped-query gradients against torch autograd (float64) through the
    forward with each key/value head repeated for its group: the repeat's
    backward sums the group, which is what dK and dV must hold.  Fixed heads
    read V only (pattern from Eq. compact-prior), so their Q rows get no
    gradient; with one query head per group the result is the layer
    backward."""
    torch = pytest.importorskip("torch")
    B, Hq, Hkv, N, d = 2, 6, 2, 9, 96
    Q, dO = _rand(B, Hq, N, d), _rand(B, Hq, N, d)
    K, V = _rand(B, Hkv, N, d), _rand(B, Hkv, N, d)
    a, r = _rand(Hq, N), _rand(Hq, N)
    is_fixed = np.array([1, 0, 0, 1, 1, 0], dtype=np.uint8)
    dQ, dK, dV = orc.layer_backward_gqa(Q, K, V, dO, is_fixed, a, r)
    tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (Q, K, V))
    ke = tk.repeat_interleave(Hq // Hkv, dim=1)
    ve = tv.repeat_interleave(Hq // Hkv, dim=1)
    i = torch.arange(N)
    off = i[:, None] - i[None, :]
    outs = []
    for h in range(Hq):
        if is_fixed[h]:
            L = (torch.tensor(a[h])[None, :] + torch.tensor(r[h])[off.clamp(min=0)]).masked_fill(off < 0, -np.inf)
            outs.append(torch.softmax(L, dim=-1) @ ve[:, h])
        else:
            S = (tq[:, h] @ ke[:, h].transpose(-1, -2)) / np.sqrt(d)
            outs.append(torch.softmax(S.masked_fill(off < 0, -np.inf), dim=-1) @ ve[:, h])
    (torch.stack(outs, dim=1) * torch.tensor(dO)).sum().backward()
    np.testing.assert_allclose(dQ, tq.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dK, tk.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dV, tv.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert not dQ[:, is_fixed.astype(bool)].any()
    # One query head per group: the layer backward.
    G1 = orc.layer_backward_gqa(Q[:, :2], K, V, dO[:, :2], is_fixed[:2], a[:2], r[:2])
    G2 = orc.layer_backward(Q[:, :2], K, V, dO[:, :2], is_fixed[:2], a[:2], r[:2])
    for x, y in zip(G1, G2):
        np.testing.assert_array_equal(x, y)


def test_fixed_heads_never_read_queries_or_keys():
    B, H, N, d = 2, 3, 16, 4
    Q, K, V, dO = (_rand(B, H, N, d) for _ in range(4))
    a, r = _rand(H, N), _rand(H, N)
    is_fixed = np.array([0, 1, 0], dtype=np.uint8)
    O0, L0 = orc.layer_forward(Q, K, V, is_fixed, a, r)
    G0 = orc.layer_backward(Q, K, V, dO, is_fixed, a, r)
    Qn, Kn = Q.copy(), K.copy()
    Qn[:, 1] = np.nan
    Kn[:, 1] = np.nan
    O1, L1 = orc.layer_forward(Qn, Kn, V, is_fixed, a, r)
    G1 = orc.layer_backward(Qn, Kn, V, dO, is_fixed, a, r)
    np.testing.assert_array_equal(O1, O0)
    np.testing.assert_array_equal(L1, L0)
    for g0, g1 in zip(G0, G1):
        np.testing.assert_array_equal(g1, g0)


def test_row_blocking_does_not_change_results():
    n, d = 41, 4
    q, k, v, do = _rand(n, d), _rand(n, d), _rand(n, d), _rand(n, d)
    a, r = _rand(n), _rand(n)
    for fixed in (False, True):
        o1, l1 = orc.head_forward(q, k, v, fixed, a, r, row_block=512)
        o2, l2 = orc.head_forward(q, k, v, fixed, a, r, row_block=5)
        np.testing.assert_allclose(o2, o1, rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(l2, l1, rtol=1e-14)
        for g1, g2 in zip(orc.head_backward(q, k, v, do, fixed, a, r, row_block=512),
                          orc.head_backward(q, k, v, do, fixed, a, r, row_block=5)):
            np.testing.assert_allclose(g2, g1, rtol=1e-12, atol=1e-13)


def test_sampled_rows_match_full_head():
    n, d = 70, 4
    q, k, v = _rand(n, d), _rand(n, d), _rand(n, d)
    a, r = _rand(n), _rand(n)
    rows = np.array([0, 5, 69, 33, 33])
    for fixed in (False, True):
        o, l = orc.head_forward(q, k, v, fixed, a, r)
        os_, ls = orc.head_forward(q, k, v, fixed, a, r, rows=rows, row_block=2)
        np.testing.assert_allclose(os_, o[rows], rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(ls, l[rows], rtol=1e-14)


def test_sampled_heads_match_full_layer():
    B, H, N, d = 2, 3, 12, 4
    Q, K, V, dO = (_rand(B, H, N, d) for _ in range(4))
    a, r = _rand(H, N), _rand(H, N)
    is_fixed = np.array([1, 0, 0], dtype=np.uint8)
    O, L = orc.layer_forward(Q, K, V, is_fixed, a, r)
    Os, Ls = orc.layer_forward(Q, K, V, is_fixed, a, r, heads=[(1, 0), (0, 2)])
    np.testing.assert_array_equal(Os[1, 0], O[1, 0])
    np.testing.assert_array_equal(Os[0, 2], O[0, 2])
    assert np.isnan(Os[0, 0]).all()


def test_parallel_driver_runs():
    B, H, N, d = 1, 2, 16, 4
    Q, K, V, dO = (_rand(B, H, N, d) for _ in range(4))
    a, r = _rand(H, N), _rand(H, N)
    used = orc.layer_forward_backward_parallel(Q, K, V, dO, np.array([0, 1]), a, r,
                                               heads=[(0, 0), (0, 1)], workers=2)
    assert used == 2


def _golden_compact_prior():
    """Parse tests/golden/compact_prior_n4.txt (hand-derived P and Z)."""
    import os
    from fractions import Fraction
    path = os.path.join(os.path.dirname(__file__), "golden", "compact_prior_n4.txt")
    a = r = z = None
    rows = {}
    for line in open(path):
        if not line.strip() or line.startswith("#"):
            continue
        parts = line.split()
        if parts[0] == "a_exp":
            a = np.log(np.array([float(x) for x in parts[1:]]))
        elif parts[0] == "r_exp":
            r = np.log(np.array([float(x) for x in parts[1:]]))
        elif parts[0] == "P":
            rows[int(parts[1])] = [float(Fraction(x)) for x in parts[2:]]
        elif parts[0] == "Z":
            z = np.array([float(x) for x in parts[1:]])
    n = len(a)
    P = np.zeros((n, n))
    for i, vals in rows.items():
        P[i, : len(vals)] = vals
    return a, r, P, np.log(z)


def test_golden_compact_prior_by_hand():
    """The oracle's fixed pattern and normaliser equal the hand-derived
    values of the golden fixture (Eq. compact-prior)."""
    a, r, P, lz = _golden_compact_prior()
    np.testing.assert_allclose(orc.fixed_pattern(a, r), P, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(orc.fixed_log_normaliser(a, r), lz, rtol=1e-14, atol=1e-15)
    # A fixed head with V = identity returns P itself.
    n = len(a)
    o, lse = orc.head_forward(None, None, np.eye(n), True, a, r)
    np.testing.assert_allclose(o, P, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lse, lz, rtol=1e-14, atol=1e-15)
