"""The backward entry point that allocates nothing
(saf_hybrid_attn_bwd_noalloc, whose scratch is the library's per-GPU device
array) against the workspace entry point saf_hybrid_attn_bwd, through the C
ABI, on the same inputs: two calls in a row, the second with a smaller
problem, each compared element by element (the two run the same kernels on
the same D, so the gradients are bit-identical), plus the oracle on the
small call.  Also: the size limit is rejected before anything is launched.
"""

import numpy as np
import pytest

from gpu_helpers import announce, compare_layer, to_device, torch_cuda
from paper_2609_34650_amd import inputs as gen

pytestmark = pytest.mark.gpu


def _grads(binding, t, O, LSE, noalloc):
    torch = torch_cuda()
    outs = [torch.full_like(t["V"], float("nan")) for _ in range(3)]
    fn = binding.saf_hybrid_attn_bwd_noalloc if noalloc else binding.saf_hybrid_attn_bwd
    fn(t["Q"], t["K"], t["V"], O, t["dO"], LSE, t["is_fixed"], t["a"], t["r"], dQ=outs[0], dK=outs[1],
       dV=outs[2])
    return outs


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_backward_equals_workspace_backward(dtype):
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    # A large call first, then a smaller one: the second must not see the
    # first call's D (it writes every row it reads).
    cases = [(4, 12, 1000, [3, 7, 11]), (2, 5, 261, [1, 4])]
    for B, H, N, fixed in cases:
        announce(f"noalloc {dtype} B={B} H={H} N={N}")
        inp = gen.make_inputs(B, H, N, 64, fixed, dtype, seed=5, stream_id=900 + N)
        t = to_device(inp, dtype)
        O, LSE = binding.saf_hybrid_attn_fwd(t["Q"], t["K"], t["V"], t["is_fixed"], t["a"], t["r"])
        ref = _grads(binding, t, O, LSE, noalloc=False)
        got = _grads(binding, t, O, LSE, noalloc=True)
        torch.cuda.synchronize()
        for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
            assert torch.equal(g, r), f"{name} differs from saf_hybrid_attn_bwd at B={B} H={H} N={N}"
        if N < 500:
            res = {"O": O, "LSE": LSE, "dQ": got[0], "dK": got[1], "dV": got[2]}
            res = {k: v.float().cpu().numpy().astype(np.float64) for k, v in res.items()}
            compare_layer(res, inp, dtype)


def test_noalloc_rejects_problems_beyond_its_scratch():
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    lib = binding.load()
    # B * H * N = 2 * 1 * (2^21 + 1) rows > 2^22: rejected before launch, so
    # the (aligned, never dereferenced) stand-in pointers are never touched.
    fake = 1 << 20
    flags = np.zeros(1, np.uint8)
    N = (1 << 21) + 1
    code = lib.saf_hybrid_attn_bwd_noalloc(1, fake, fake, fake, fake, fake, fake, flags.ctypes.data, None, None,
                                           N, 2, 1, N, 64, fake, fake, fake, None)
    assert code == 2
    torch.cuda.synchronize()


def test_noalloc_at_its_largest_problem():
    """B * H * N = 2^22 rows exactly (B = 16, H = 64, the largest head mask,
    N = 4096, bf16, fixed heads on mask bits 0 and 63): the whole scratch
    array is used, and the result is bit-identical to the workspace entry
    point's.  Inputs are drawn on the device from a seeded generator."""
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    B, H, N, d = 16, 64, 4096, 64
    assert B * H * N == 1 << 22
    announce(f"noalloc at the limit B={B} H={H} N={N}")
    dev = torch.device("cuda", 0)
    gen_ = torch.Generator(device=dev).manual_seed(1337)
    t = {k: torch.randn((B, H, N, d), generator=gen_, device=dev).to(torch.bfloat16) for k in ("Q", "K", "V", "dO")}
    flags = np.zeros(H, np.uint8)
    flags[[0, 63]] = 1
    t["is_fixed"] = flags
    t["a"] = torch.randn((H, N), generator=gen_, device=dev)
    t["r"] = -torch.log1p(torch.arange(N, device=dev, dtype=torch.float32)).expand(H, N).contiguous()
    O, LSE = binding.saf_hybrid_attn_fwd(t["Q"], t["K"], t["V"], t["is_fixed"], t["a"], t["r"])
    ref = _grads(binding, t, O, LSE, noalloc=False)
    got = _grads(binding, t, O, LSE, noalloc=True)
    torch.cuda.synchronize()
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
        assert torch.isfinite(r).all(), name
        assert torch.equal(g, r), f"{name} differs from saf_hybrid_attn_bwd at the scratch limit"
