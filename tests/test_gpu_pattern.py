"""GPU parity of the trainable-pattern gradients (saf_hybrid_attn_bwd_pattern)
against the fp64 oracle (``oracle.saf_oracle.layer_pattern_grad``).

Both sides take V, dO, a, r from the seeded generator; the GPU side runs its
own forward for O and LSE, as a caller would.  da and dr are sums of up to
B*N terms of size ~|dP| / (i+1), so the bars scale with the largest entry
``m = max |oracle|``:
* float32: ``|gpu - oracle| <= 1e-4 * max(1, m)``;
* bf16:    ``|gpu - oracle| <= 1e-2 * max(1, m) + 2e-2 * |oracle|`` (the
  kernel's D comes from the bf16-rounded forward output, as in the layer's
  own backward, whose bf16 bar this is).
Both also check that each head's da and dr sum to zero (a common shift of a
row's logits changes nothing).
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
    return (g_da, g_dr), (o_da, o_dr), inp["is_fixed"]


def _check(dtype, g, o, is_fixed):
    for gv, ov, name in ((g[0], o[0], "da"), (g[1], o[1], "dr")):
        m = max(1.0, float(np.abs(ov).max()))
        err = np.abs(gv - ov)
        if dtype == "f32":
            bound = 1e-4 * m
        else:
            bound = 1e-2 * m + 2e-2 * np.abs(ov)
        worst = float(np.max(err - bound))
        assert worst <= 0, f"{name}: max excess {worst:.3e} (max err {err.max():.3e}, scale {m:.3e})"
        ordinary = np.asarray(is_fixed) == 0
        assert not gv[ordinary].any(), f"{name}: ordinary heads must get zeros"
        np.testing.assert_allclose(gv.sum(axis=1), 0.0, atol=(1e-4 if dtype == "f32" else 2e-2) * m * 10)


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
    g, o, is_fixed = _run(dtype, B, H, N, list(fixed), stream_id=31)
    _check(dtype, g, o, is_fixed)


@pytest.mark.slow
def test_pattern_gradient_124m_shape():
    """The 124M layer shape (12 heads, 3 fixed, N = 4096, bf16) on two batch
    elements (the oracle is dense float64)."""
    from paper_2609_34650_amd import inputs
    w = inputs.WORKLOADS["gpt124m_4k"]
    fixed = inputs.fixed_heads(w.H, w.n_fixed, stream_id=w.stream_id)
    announce(f"pattern grad 124m shape B=2 fixed={fixed}")
    g, o, is_fixed = _run("bf16", 2, w.H, w.N, fixed, stream_id=32)
    _check("bf16", g, o, is_fixed)


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
