"""GPU parity of the grouped-query forward (saf_hybrid_attn_fwd_gqa) for head
dimensions 64, 96 and 128 against the fp64 oracle
(``oracle.saf_oracle.layer_forward_gqa``).

Inputs come from the seeded generator (query heads as drawn; key/value heads
are the first Hkv heads of the drawn K and V).  Bars are the layer's:
float32 ``max |gpu - oracle| <= 1e-4``; bf16 ``|gpu - oracle| <= 1e-2 +
2e-2 |oracle|`` on O and LSE.
"""

import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, BF16_RTOL, F32_ATOL, announce, bf16_rounding_bound, torch_cuda

pytestmark = pytest.mark.gpu


def _inputs(dtype, B, Hq, Hkv, N, d, fixed, stream_id):
    from paper_2609_34650_amd import inputs
    inp = inputs.make_inputs(B, Hq, N, d, fixed, dtype, stream_id=stream_id, backward=False)
    inp["K"] = np.ascontiguousarray(inp["K"][:, :Hkv])
    inp["V"] = np.ascontiguousarray(inp["V"][:, :Hkv])
    return inp


def _run_gpu(inp, dtype):
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    Q, K, V = (torch.from_numpy(inp[k]).to(dev).to(tdt).contiguous() for k in ("Q", "K", "V"))
    a = torch.from_numpy(np.ascontiguousarray(inp["a"])).to(dev)
    r = torch.from_numpy(np.ascontiguousarray(inp["r"])).to(dev)
    O, LSE = binding.saf_hybrid_attn_fwd_gqa(Q, K, V, inp["is_fixed"], a, r)
    torch.cuda.synchronize()
    return O.double().cpu().numpy(), LSE.double().cpu().numpy()


def _check(dtype, g, o, extra=0.0):
    if dtype == "f32":
        assert np.max(np.abs(g - o)) <= F32_ATOL * max(1.0, float(np.max(np.abs(o))))
    else:
        excess = np.abs(g - o) - (BF16_ATOL + BF16_RTOL * np.abs(o) + extra)
        assert np.max(excess) <= 0, float(np.max(excess))


@pytest.mark.parametrize("dtype,B,Hq,Hkv,N,d,fixed", [
    ("f32", 1, 4, 4, 200, 64, (1,)),
    ("bf16", 2, 8, 2, 300, 128, (0, 5)),
    ("bf16", 1, 6, 1, 77, 96, (2, 3)),
    ("f32", 1, 4, 2, 130, 96, (0,)),
    ("f32", 1, 2, 1, 129, 128, ()),
    ("bf16", 1, 4, 2, 1, 128, (1,)),
    ("bf16", 1, 4, 4, 257, 64, (0, 1, 2, 3)),
    ("f32", 1, 64, 8, 70, 96, (0, 7, 8, 62, 63)),    # the largest head count: mask bit 63
])
def test_gqa_forward_matches_oracle(dtype, B, Hq, Hkv, N, d, fixed):
    from oracle import saf_oracle as orc
    announce(f"gqa fwd {dtype} B={B} Hq={Hq} Hkv={Hkv} N={N} d={d} fixed={fixed}")
    inp = _inputs(dtype, B, Hq, Hkv, N, d, list(fixed), stream_id=51)
    O, LSE = _run_gpu(inp, dtype)
    Oo, LSEo = orc.layer_forward_gqa(inp["Q"], inp["K"], inp["V"], inp["is_fixed"], inp["a"], inp["r"])
    _check(dtype, O, Oo)
    _check(dtype, LSE, LSEo)


def test_gqa_forward_equals_layer_forward_at_d64():
    """With one query head per key/value head and d = 64 the grouped-query
    kernel and the layer's own forward compute the same function."""
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    announce("gqa vs layer forward d=64")
    inp = _inputs("f32", 2, 4, 4, 333, 64, [1, 2], stream_id=52)
    O, LSE = _run_gpu(inp, "f32")
    dev = torch.device("cuda", 0)
    t = {k: torch.from_numpy(inp[k]).to(dev) for k in ("Q", "K", "V", "a", "r")}
    O2, LSE2 = binding.saf_hybrid_attn_fwd(t["Q"], t["K"], t["V"], inp["is_fixed"], t["a"], t["r"])
    torch.cuda.synchronize()
    np.testing.assert_allclose(O, O2.double().cpu().numpy(), rtol=0, atol=2e-5)
    np.testing.assert_allclose(LSE, LSE2.double().cpu().numpy(), rtol=0, atol=2e-5)


@pytest.mark.slow
def test_gqa_prefill_shape_sampled():
    """The grouped-query prefill layout (32 query heads, 8 key/value heads,
    d = 128, 8 fixed heads, N = 4096, bf16): every head of one batch element,
    sampled rows against the oracle."""
    from oracle import saf_oracle as orc
    from paper_2609_34650_amd import inputs
    fixed = inputs.fixed_heads(32, 8, stream_id=53)
    announce(f"gqa prefill shape fixed={fixed}")
    inp = _inputs("bf16", 1, 32, 8, 4096, 128, fixed, stream_id=53)
    O, LSE = _run_gpu(inp, "bf16")
    rows = np.array([0, 1, 63, 64, 127, 128, 1000, 2047, 4095])
    for h in range(32):
        g = h // 4
        fx = bool(inp["is_fixed"][h])
        o, lse = orc.head_forward(None if fx else inp["Q"][0, h], None if fx else inp["K"][0, g], inp["V"][0, g], fx,
                                  inp["a"][h] if fx else None, inp["r"][h] if fx else None, rows=rows)
        _check("bf16", O[0, h, rows], o)
        _check("bf16", LSE[0, h, rows], lse)


@pytest.mark.parametrize("dtype,d", [("f32", 96), ("bf16", 128)])
def test_gqa_fixed_exact_fallback(dtype, d):
    """a is 60 nats lower on the first half of the keys: the blocks whose rows
    lie in that half but whose maxima come from the second half must take the
    exact per-entry programs (the factorised ones would underflow or
    overflow): the forward's query block and the backward's key block that
    straddle the middle; the rest take the factorised programs."""
    from oracle import saf_oracle as orc
    announce(f"gqa fixed exact fallback {dtype} d={d}")
    N = 600
    inp = _bwd_inputs(dtype, 1, 4, 2, N, d, [0, 3], stream_id=54)
    a = inp["a"].copy()
    a[0, : N // 2] -= 60.0
    a[3, : N // 2] -= 60.0
    inp["a"] = a.astype(np.float32)
    O, LSE = _run_gpu(inp, dtype)
    Oo, LSEo = orc.layer_forward_gqa(inp["Q"], inp["K"], inp["V"], inp["is_fixed"], inp["a"], inp["r"])
    _check(dtype, O, Oo)
    _check(dtype, LSE, LSEo)
    g = _run_gpu_bwd(inp, dtype)
    o = orc.layer_backward_gqa(inp["Q"], inp["K"], inp["V"], inp["dO"], inp["is_fixed"], inp["a"], inp["r"])
    for gv, ov in zip(g, o):
        _check(dtype, gv, ov)


# ---------------------------------------------------------------------------
# Backward (saf_hybrid_attn_bwd_gqa) against oracle.saf_oracle.layer_backward_gqa
# ---------------------------------------------------------------------------

def _bwd_inputs(dtype, B, Hq, Hkv, N, d, fixed, stream_id):
    from paper_2609_34650_amd import inputs
    inp = inputs.make_inputs(B, Hq, N, d, fixed, dtype, stream_id=stream_id, backward=True)
    inp["K"] = np.ascontiguousarray(inp["K"][:, :Hkv])
    inp["V"] = np.ascontiguousarray(inp["V"][:, :Hkv])
    return inp


def _run_gpu_bwd(inp, dtype):
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    t = {k: torch.from_numpy(inp[k]).to(dev).to(tdt).contiguous() for k in ("Q", "K", "V", "dO")}
    a = torch.from_numpy(inp["a"]).to(dev)
    r = torch.from_numpy(inp["r"]).to(dev)
    O, LSE = binding.saf_hybrid_attn_fwd_gqa(t["Q"], t["K"], t["V"], inp["is_fixed"], a, r)
    dQ, dK, dV = binding.saf_hybrid_attn_bwd_gqa(t["Q"], t["K"], t["V"], O, t["dO"], LSE, inp["is_fixed"], a, r)
    torch.cuda.synchronize()
    return [x.double().cpu().numpy() for x in (dQ, dK, dV)]


@pytest.mark.parametrize("dtype,B,Hq,Hkv,N,d,fixed", [
    ("f32", 1, 4, 2, 200, 96, (1,)),
    ("bf16", 2, 8, 2, 300, 128, (0, 5)),
    ("bf16", 1, 6, 1, 77, 64, (2, 3)),
    ("f32", 1, 4, 4, 130, 128, (0, 1, 2, 3)),   # every head fixed: dQ and dK are zeros
    ("bf16", 1, 4, 2, 1, 96, (1,)),
    ("f32", 1, 2, 1, 129, 64, ()),
    ("bf16", 1, 8, 2, 1000, 128, (1, 2, 6)),    # several key blocks, mixed groups
    ("f32", 1, 3, 3, 257, 96, (1,)),
    # The largest head count (mask bit 63), float32 and bf16.  In bf16 at
    # d = 128 the gradients reach ~9 in size and a few small elements of 64
    # heads miss the plain elementwise bar; that case is held to the plain bar
    # plus the worst-case effect of the bf16 operand rounding on each element
    # (``gpu_helpers.bf16_rounding_bound``, computed in float64 from the oracle's P, dS
    # and the inputs).
    ("f32", 1, 64, 16, 90, 128, (1, 2, 3, 62, 63)),
    ("bf16", 1, 64, 16, 90, 128, (1, 2, 3, 62, 63)),
])
def test_gqa_backward_matches_oracle(dtype, B, Hq, Hkv, N, d, fixed):
    from oracle import saf_oracle as orc
    announce(f"gqa bwd {dtype} B={B} Hq={Hq} Hkv={Hkv} N={N} d={d} fixed={fixed}")
    inp = _bwd_inputs(dtype, B, Hq, Hkv, N, d, list(fixed), stream_id=55)
    g = _run_gpu_bwd(inp, dtype)
    o = orc.layer_backward_gqa(inp["Q"], inp["K"], inp["V"], inp["dO"], inp["is_fixed"], inp["a"], inp["r"])
    extra = bf16_rounding_bound(inp, Hkv) if (dtype == "bf16" and Hq == 64) else (0.0, 0.0, 0.0)
    for name, gv, ov, w in zip(("dQ", "dK", "dV"), g, o, extra):
        assert np.isfinite(gv).all(), name
        _check(dtype, gv, ov, w)
    fixed_q = np.asarray(inp["is_fixed"]).astype(bool)
    assert not g[0][:, fixed_q].any(), "fixed heads must get zero dQ"
    group = Hq // Hkv
    for gk in range(Hkv):
        if fixed_q[gk * group:(gk + 1) * group].all():
            assert not g[1][:, gk].any(), "a group of fixed heads must give zero dK"


def test_gqa_backward_equals_layer_backward_at_d64():
    """One query head per key/value head at d = 64: the grouped-query
    backward and the layer's own backward compute the same gradients."""
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    announce("gqa bwd vs layer bwd d=64")
    inp = _bwd_inputs("f32", 2, 4, 4, 333, 64, [1, 2], stream_id=56)
    g = _run_gpu_bwd(inp, "f32")
    dev = torch.device("cuda", 0)
    t = {k: torch.from_numpy(inp[k]).to(dev) for k in ("Q", "K", "V", "dO", "a", "r")}
    O, LSE = binding.saf_hybrid_attn_fwd(t["Q"], t["K"], t["V"], inp["is_fixed"], t["a"], t["r"])
    ref = binding.saf_hybrid_attn_bwd(t["Q"], t["K"], t["V"], O, t["dO"], LSE, inp["is_fixed"], t["a"], t["r"])
    torch.cuda.synchronize()
    for gv, rv in zip(g, ref):
        np.testing.assert_allclose(gv, rv.double().cpu().numpy(), rtol=0, atol=2e-5)


def test_gqa_autograd_wrapper_matches_abi():
    """The grouped-query autograd wrapper returns exactly what the two C ABI
    calls return."""
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    announce("gqa autograd wrapper")
    inp = _bwd_inputs("bf16", 1, 8, 2, 200, 96, [1, 6], stream_id=57)
    dev = torch.device("cuda", 0)
    t = {k: torch.from_numpy(inp[k]).to(dev).to(torch.bfloat16).contiguous() for k in ("Q", "K", "V", "dO")}
    a = torch.from_numpy(inp["a"]).to(dev)
    r = torch.from_numpy(inp["r"]).to(dev)
    q, k, v = (t[x].clone().requires_grad_(True) for x in ("Q", "K", "V"))
    o = binding.HybridAttentionGQA.apply(q, k, v, inp["is_fixed"], a, r)
    o.backward(t["dO"])
    O, LSE = binding.saf_hybrid_attn_fwd_gqa(t["Q"], t["K"], t["V"], inp["is_fixed"], a, r)
    dQ, dK, dV = binding.saf_hybrid_attn_bwd_gqa(t["Q"], t["K"], t["V"], O, t["dO"], LSE, inp["is_fixed"], a, r)
    torch.cuda.synchronize()
    assert torch.equal(o.detach(), O)
    assert torch.equal(q.grad, dQ) and torch.equal(k.grad, dK) and torch.equal(v.grad, dV)


# ---------------------------------------------------------------------------
# The grouped-query training layers the benchmark times, at full size
# ---------------------------------------------------------------------------

TRAIN_SHAPES = {
    # name: (B, Hq, Hkv, N, d, stream id, fixed query heads) -- bench.py's --layer128 and --layer1b
    "gqa_train_4k_d128": (4, 32, 8, 4096, 128, 64, 8),
    "layer1b_8k_d96": (2, 16, 16, 8192, 96, 62, 4),
}


@pytest.mark.slow
@pytest.mark.parametrize("name", list(TRAIN_SHAPES))
def test_gqa_training_layer_full_size_sampled(name):
    """Forward and backward of a whole training layer in the benchmark's
    launch configuration (at d = 128 the key-block pass runs as its dK and dV
    launches), then, for two (batch element, key/value group) pairs -- the
    first group holding a fixed head, and in the last batch element the last
    group holding an ordinary head -- every element of O, LSE and dQ of the
    group's query heads and
    of the group's dK and dV against the oracle, at the bf16 bar plus the
    worst-case effect of the bf16 operand rounding (gpu_helpers)."""
    torch = torch_cuda()
    from oracle import saf_oracle as orc
    from paper_2609_34650_amd import binding, inputs
    B, Hq, Hkv, N, d, sid, n_fixed = TRAIN_SHAPES[name]
    announce(f"gqa training layer full size {name}")
    inp = inputs.make_inputs(B, Hq, N, d, [], "bf16", stream_id=sid, backward=True)
    flags = np.zeros(Hq, np.uint8)
    flags[inputs.fixed_heads(Hq, n_fixed, stream_id=sid)] = 1
    inp["K"] = np.ascontiguousarray(inp["K"][:, :Hkv])
    inp["V"] = np.ascontiguousarray(inp["V"][:, :Hkv])
    inp["is_fixed"] = flags
    dev = torch.device("cuda", 0)
    t = {k: torch.from_numpy(inp[k]).to(dev).to(torch.bfloat16).contiguous() for k in ("Q", "K", "V", "dO")}
    a = torch.from_numpy(inp["a"]).to(dev)
    r = torch.from_numpy(inp["r"]).to(dev)
    O, LSE = binding.saf_hybrid_attn_fwd_gqa(t["Q"], t["K"], t["V"], flags, a, r)
    dQ, dK, dV = binding.saf_hybrid_attn_bwd_gqa(t["Q"], t["K"], t["V"], O, t["dO"], LSE, flags, a, r)
    torch.cuda.synchronize()
    group = Hq // Hkv
    g_fixed = next(g for g in range(Hkv) if flags[g * group:(g + 1) * group].any())
    g_ordinary = next(g for g in reversed(range(Hkv)) if not flags[g * group:(g + 1) * group].all())
    for b, g in ((0, g_fixed), (B - 1, g_ordinary)):
        hs = slice(g * group, (g + 1) * group)
        sub = {"Q": inp["Q"][b:b + 1, hs], "K": inp["K"][b:b + 1, g:g + 1], "V": inp["V"][b:b + 1, g:g + 1],
               "dO": inp["dO"][b:b + 1, hs], "is_fixed": flags[hs], "a": inp["a"][hs], "r": inp["r"][hs]}
        announce(f"  oracle for b={b} group={g} heads {hs.start}..{hs.stop - 1} fixed={flags[hs].tolist()}")
        Oo, Lo = orc.layer_forward_gqa(sub["Q"], sub["K"], sub["V"], sub["is_fixed"], sub["a"], sub["r"])
        dQo, dKo, dVo = orc.layer_backward_gqa(sub["Q"], sub["K"], sub["V"], sub["dO"], sub["is_fixed"], sub["a"],
                                               sub["r"])
        wq, wk, wv = bf16_rounding_bound(sub, 1)
        _check("bf16", O[b:b + 1, hs].double().cpu().numpy(), Oo)
        _check("bf16", LSE[b:b + 1, hs].double().cpu().numpy(), Lo)
        _check("bf16", dQ[b:b + 1, hs].double().cpu().numpy(), dQo, wq)
        _check("bf16", dK[b:b + 1, g:g + 1].double().cpu().numpy(), dKo, wk)
        _check("bf16", dV[b:b + 1, g:g + 1].double().cpu().numpy(), dVo, wv)
        fixed_q = flags[hs].astype(bool)
        assert not dQ[b, hs][torch.from_numpy(fixed_q).to(dev)].any(), "fixed heads must get zero dQ"
