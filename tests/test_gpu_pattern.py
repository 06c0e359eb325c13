"""GPU parity of the trainable-pattern gradients (saf_hybrid_attn_bwd_pattern)
against the fp64 oracle (``oracle.saf_oracle.layer_pattern_grad``).

Both sides take V, dO, a, r from the seeded generator; the GPU side runs its
own forward for O and LSE, as a caller would.

Bars are per entry.  An entry of da (or dr) is a sum over batch elements and
query rows of ``dL(i, j) = P(i, j) (dP(i, j) - D_i)``; its error has two
sources, each bounded from oracle quantities of that same entry:
* float32 accumulation of the terms: at most a small multiple of the
  rounding unit times ``S(j) = sum |dL(i, j)|`` (the terms' absolute sum);
  the bar allows ``1e-4 S(j)``, far above the ~1e-6 seen;
* the kernel's D comes from the forward output as stored, rounded to the
  element type: ``|D_kernel - D| <= u sum_c |dO_ic O_ic|`` with ``u`` the
  unit roundoff (2^-9 for bf16, 2^-24 for float32), which moves the entry by
  at most ``u E(j)``, ``E(j) = sum P(i, j) sum_c |dO_ic O_ic|``; the bar
  allows ``2u E(j)``.
So ``|gpu - oracle| <= 1e-6 + 1e-4 S + 2u E`` element by element.  Both also
check that each head's da and dr sum to zero (a common shift of a row's
logits changes nothing).
"""

import numpy as np
import pytest

from gpu_helpers import announce, to_device, torch_cuda

pytestmark = pytest.mark.gpu


def _run(dtype, B, H, N, fixed, stream_id):
    torch = torch_cuda()
    from oracle import saf_oracle as orc
    from paper_2609_34650_amd import binding, inputs
    inp = inputs.make_inputs(B, H, N, 64, fixed, dtype, stream_id=stream_id)
    t = to_device(inp, dtype)
    O, LSE = binding.saf_hybrid_attn_fwd(t["Q"], t["K"], t["V"], t["is_fixed"], t["a"], t["r"])
    da, dr = binding.saf_hybrid_attn_bwd_pattern(t["V"], O, t["dO"], LSE, t["is_fixed"], t["a"], t["r"])
    torch.cuda.synchronize()
    g_da, g_dr = da.double().cpu().numpy(), dr.double().cpu().numpy()
    o_da, o_dr = orc.layer_pattern_grad(inp["V"], inp["dO"], inp["is_fixed"], inp["a"], inp["r"])
    return (g_da, g_dr), (o_da, o_dr), inp


def _diag_sums(m: np.ndarray) -> np.ndarray:
    """sum over i - j = delta of a lower-triangular [n, n] array, per delta."""
    n = m.shape[0]
    out = np.zeros(n)
    for i in range(n):
        out[: i + 1] += m[i, i::-1]
    return out


def _error_scales(inp):
    """Per fixed head and entry: S (absolute sum of the terms) and E (the
    D-rounding sensitivity) for da and dr, from the oracle's pattern."""
    from oracle import saf_oracle as orc
    V, dO = inp["V"].astype(np.float64), inp["dO"].astype(np.float64)
    B, H, N, _ = V.shape
    S = np.zeros((2, H, N))
    E = np.zeros((2, H, N))
    for h in np.flatnonzero(inp["is_fixed"]):
        P = orc.fixed_pattern(inp["a"][h], inp["r"][h], N)
        for b in range(B):
            v, do = V[b, h], dO[b, h]
            dp = do @ v.T
            D = np.sum(P * dp, axis=1)
            dl = np.abs(P * (dp - D[:, None]))
            w = P * np.sum(np.abs(do * (P @ v)), axis=1)[:, None]
            S[0, h] += dl.sum(axis=0)
            S[1, h] += _diag_sums(dl)
            E[0, h] += w.sum(axis=0)
            E[1, h] += _diag_sums(w)
    return S, E


def _check(dtype, g, o, inp):
    S, E = _error_scales(inp)
    u = 2.0 ** -9 if dtype == "bf16" else 2.0 ** -24
    is_fixed = inp["is_fixed"]
    for k, name in enumerate(("da", "dr")):
        gv, ov = g[k], o[k]
        bound = 1e-6 + 1e-4 * S[k] + 2.0 * u * E[k]
        err = np.abs(gv - ov)
        excess = err - bound
        i = np.unravel_index(int(np.argmax(excess)), excess.shape)
        assert excess[i] <= 0, (f"{name}[{i}]: |gpu - oracle| = {err[i]:.3e} > bar {bound[i]:.3e} "
                                f"(S {S[k][i]:.3e}, E {E[k][i]:.3e})")
        ordinary = np.asarray(is_fixed) == 0
        assert not gv[ordinary].any(), f"{name}: ordinary heads must get zeros"
        # Each head's entries sum to zero; the sum's error is bounded by the
        # sum of the entries' bars.
        np.testing.assert_allclose(gv.sum(axis=1), 0.0, atol=float(bound.sum(axis=1).max()) + 1e-9)


@pytest.mark.parametrize("dtype,B,H,N,fixed", [
    ("f32", 2, 3, 200, (0, 2)),       # ragged key block and query tile
    ("f32", 1, 2, 64, (1,)),          # one tile
    ("bf16", 2, 4, 300, (1, 2)),
    ("bf16", 1, 2, 129, (0,)),        # last key block holds one key
    ("bf16", 1, 1, 1, (0,)),          # a single position: no gradient
    ("bf16", 3, 2, 1000, (0, 1)),     # several key blocks, every head fixed
    ("f32", 1, 2, 2200, (1,)),        # key blocks cut into up to three chunks
])
def test_pattern_gradient_matches_oracle(dtype, B, H, N, fixed):
    announce(f"pattern grad {dtype} B={B} H={H} N={N} fixed={fixed}")
    g, o, inp = _run(dtype, B, H, N, list(fixed), stream_id=31)
    _check(dtype, g, o, inp)


@pytest.mark.slow
def test_pattern_gradient_124m_shape():
    """The 124M layer shape (12 heads, 3 fixed, N = 4096, bf16) on two batch
    elements (the oracle is dense float64)."""
    from paper_2609_34650_amd import inputs
    w = inputs.WORKLOADS["gpt124m_4k"]
    fixed = inputs.fixed_heads(w.H, w.n_fixed, stream_id=w.stream_id)
    announce(f"pattern grad 124m shape B=2 fixed={fixed}")
    g, o, inp = _run("bf16", 2, w.H, w.N, fixed, stream_id=32)
    _check("bf16", g, o, inp)


def test_pattern_gradient_is_deterministic():
    """The partial sums are added in a fixed order: two calls give the same
    bits, and ordinary heads' rows are zeros even over stale outputs."""
    torch = torch_cuda()
    from paper_2609_34650_amd import binding, inputs
    announce("pattern grad determinism")
    inp = inputs.make_inputs(3, 4, 700, 64, [0, 2], "bf16", stream_id=33)
    t = to_device(inp, "bf16")
    O, LSE = binding.saf_hybrid_attn_fwd(t["Q"], t["K"], t["V"], t["is_fixed"], t["a"], t["r"])
    da1, dr1 = binding.saf_hybrid_attn_bwd_pattern(t["V"], O, t["dO"], LSE, t["is_fixed"], t["a"], t["r"])
    da2 = torch.full_like(da1, 7.0)
    dr2 = torch.full_like(dr1, 7.0)
    binding.saf_hybrid_attn_bwd_pattern(t["V"], O, t["dO"], LSE, t["is_fixed"], t["a"], t["r"], da=da2, dr=dr2)
    torch.cuda.synchronize()
    assert torch.equal(da1, da2) and torch.equal(dr1, dr2)
    assert not da2[[1, 3]].any() and not dr2[[1, 3]].any()
