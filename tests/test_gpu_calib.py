"""GPU parity of the calibration statistics (include/saf_calib.h) against the
fp64 oracle (``oracle.calib_oracle``).

Both sides take Q and K from the seeded generator in
``paper_2609_34650_amd.inputs``.  The GPU side gets LSE from its own forward
(``saf_hybrid_attn_fwd`` with every head ordinary), as a caller would; the
oracle computes its own softmax.  Tolerances follow from float32 statistics
of weights computed from float32 scores: a weight carries a relative error of
a few 1e-6 (LSE rounding and exp2), so
* mean attention, marginals: ``|gpu - oracle| <= 1e-6 + 1e-4 |oracle|``;
* variance score: relative 1e-3 (Welford sums in float32);
* KL score: absolute 1e-4 (a difference of two float64 sums of float32 terms
  of size ~ln T).
"""

import functools
import os

import numpy as np
import pytest

from gpu_helpers import announce, torch_cuda

pytestmark = pytest.mark.gpu

A_ATOL, A_RTOL = 1e-6, 1e-4
SVAR_RTOL = 1e-3
SKL_ATOL = 1e-4


def _gpu_stats(Q, K, dtype, micro, state=None, reuse_garbage=False, keep_m2=False):
    """Run the forward for LSE and fold the inputs in micro-batches of the
    listed sizes.  Returns (numpy dict, state)."""
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    N, H, T, d = Q.shape
    if state is None:
        state = binding.CalibState(H, T, dev, keep_m2=keep_m2)
        if reuse_garbage:
            state.mean.fill_(float("nan"))
            if state.m2 is not None:
                state.m2.fill_(float("nan"))
            state.stats.fill_(float("nan"))
    start = 0
    for m in micro:
        q = torch.from_numpy(np.ascontiguousarray(Q[start:start + m])).to(dev).to(tdt).contiguous()
        k = torch.from_numpy(np.ascontiguousarray(K[start:start + m])).to(dev).to(tdt).contiguous()
        _, lse = binding.saf_hybrid_attn_fwd(q, k, q, np.zeros(H, np.uint8))
        binding.saf_calib_accumulate(q, k, lse, state)
        start += m
    assert start == N
    out = binding.saf_calib_finalize(state)
    torch.cuda.synchronize()
    res = {k: v.double().cpu().numpy() for k, v in out.items()}
    if state.m2 is not None:
        res["m2"] = state.m2.double().cpu().numpy()
    return res, state


def _inputs(N, H, T, dtype, stream_id):
    from paper_2609_34650_amd import inputs
    return inputs.calib_inputs(N, H, T, 64, dtype, stream_id=stream_id)


def _compare(g, o, T):
    np.testing.assert_allclose(g["A_mean"], o["A_mean"], rtol=A_RTOL, atol=A_ATOL)
    if "m2" in g:
        np.testing.assert_allclose(g["m2"], o["sq_dev"], rtol=SVAR_RTOL, atol=1e-9)
    assert np.all(np.triu(g["A_mean"], 1) == 0)
    np.testing.assert_allclose(g["eta_abs"], o["eta_abs"], rtol=A_RTOL, atol=A_ATOL * T)
    np.testing.assert_allclose(g["eta_rel"], o["eta_rel"], rtol=A_RTOL, atol=A_ATOL * T)
    np.testing.assert_allclose(g["s_var"], o["s_var"], rtol=SVAR_RTOL)
    np.testing.assert_allclose(g["s_kl"], o["s_kl"], rtol=0, atol=SKL_ATOL)


@pytest.mark.parametrize("dtype,N,H,T,micro,keep_m2", [
    ("f32", 5, 2, 200, (2, 3), True),          # two tiles, ragged tail
    ("f32", 3, 1, 130, (1, 2), False),
    ("bf16", 4, 3, 300, (1, 2, 1), True),      # three tiles, odd micro-batches
    ("bf16", 4, 2, 260, (3, 1), False),
    ("bf16", 3, 1, 128, (3,), False),          # exactly one tile
    ("bf16", 2, 2, 37, (2,), True),            # one partial tile
    # The accumulation path the benchmark times (no per-entry squared
    # deviations, micro-batches of two) over eight 128-query tiles.
    ("bf16", 8, 2, 1024, (2, 2, 2, 2), False),
    ("f32", 8, 1, 1024, (2, 2, 2, 2), False),
])
def test_calib_matches_oracle(dtype, N, H, T, micro, keep_m2):
    from oracle import calib_oracle as co
    announce(f"calib parity {dtype} N={N} H={H} T={T} micro={micro} keep_m2={keep_m2}")
    inp = _inputs(N, H, T, dtype, stream_id=21)
    g, _ = _gpu_stats(inp["Q"], inp["K"], dtype, micro, keep_m2=keep_m2)
    o = co.calibration_stats(inp["Q"], inp["K"])
    _compare(g, o, T)


def test_calib_split_equals_single_call_and_ignores_old_state():
    """Welford's recurrence runs in input order either way, so the mean after
    micro-batches (1, 2, 1) is bitwise the mean after one call of 4 (the
    squared deviations are added per call, so they agree to rounding); and
    n_seen = 0 ignores whatever the state buffers held."""
    announce("calib split vs single call")
    inp = _inputs(4, 2, 260, "bf16", stream_id=22)
    a, _ = _gpu_stats(inp["Q"], inp["K"], "bf16", (4,), reuse_garbage=True, keep_m2=True)
    b, _ = _gpu_stats(inp["Q"], inp["K"], "bf16", (1, 2, 1), keep_m2=True)
    c, _ = _gpu_stats(inp["Q"], inp["K"], "bf16", (2, 2), keep_m2=False)
    np.testing.assert_array_equal(a["A_mean"], b["A_mean"])
    np.testing.assert_array_equal(a["A_mean"], c["A_mean"])
    np.testing.assert_allclose(a["m2"], b["m2"], rtol=1e-5, atol=1e-12)
    np.testing.assert_allclose(a["s_var"], c["s_var"], rtol=1e-5)
    # The variance score's sum of squared deviations is the sum of the
    # per-entry ones.
    np.testing.assert_allclose(b["s_var"], b["m2"].sum(axis=(1, 2)) / (3 * 260 * 260), rtol=1e-5)
    # ent gathers float32 per-lane partials per call: equal to rounding only.
    np.testing.assert_allclose(a["s_kl"], b["s_kl"], rtol=0, atol=1e-6)
    assert np.all(np.isfinite(a["A_mean"]))


def test_calib_single_input_and_single_position():
    from oracle import calib_oracle as co
    announce("calib N=1 T=1 and N=1 T=70")
    inp = _inputs(1, 2, 1, "f32", stream_id=23)
    g, _ = _gpu_stats(inp["Q"], inp["K"], "f32", (1,))
    # exp(S - LSE) with LSE = S: one up to the rounding of both in float32.
    np.testing.assert_allclose(g["A_mean"], np.ones((2, 1, 1)), rtol=0, atol=1e-6)
    np.testing.assert_allclose(g["eta_abs"], np.ones((2, 1)), rtol=0, atol=1e-6)
    assert np.all(np.isnan(g["s_var"]))
    np.testing.assert_allclose(g["s_kl"], 0.0, atol=1e-6)
    inp = _inputs(1, 2, 70, "bf16", stream_id=24)
    g, _ = _gpu_stats(inp["Q"], inp["K"], "bf16", (1,))
    o = co.calibration_stats(inp["Q"], inp["K"])
    np.testing.assert_allclose(g["A_mean"], o["A_mean"], rtol=A_RTOL, atol=A_ATOL)
    assert np.all(np.isnan(g["s_var"]))
    np.testing.assert_allclose(g["s_kl"], 0.0, atol=SKL_ATOL)


@functools.lru_cache(maxsize=1)
def _full_inputs():
    from paper_2609_34650_amd import inputs
    w = inputs.CALIB_WORKLOADS["calib124m_4k"]
    return w, inputs.calib_inputs(w.n_cal, w.H, w.T, w.d, w.dtype, stream_id=w.stream_id)


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "calib124m_4k_head0.npz")


@pytest.mark.slow
def test_calib_full_size_no_m2():
    """The accumulation path the benchmark times (no per-entry squared
    deviations) on the 124M-style workload (32 inputs of T = 4096 in
    micro-batches of two, 12 heads, bf16): head 0 against the oracle's
    statistics over every row (tests/golden/calib124m_4k_head0.npz, written by
    make_calib124m_head0.py from the oracle alone) -- mean rows, both
    marginals elementwise, both scores -- and sampled mean rows of every head
    against the oracle computed here."""
    from oracle import calib_oracle as co
    w, inp = _full_inputs()
    announce(f"calib full size {w.name} without m2")
    g, _ = _gpu_stats(inp["Q"], inp["K"], w.dtype, (w.micro,) * (w.n_cal // w.micro), keep_m2=False)
    ref = np.load(GOLDEN)
    rows = ref["rows"]
    np.testing.assert_allclose(g["A_mean"][0, rows], ref["A_mean_rows"], rtol=A_RTOL, atol=A_ATOL)
    np.testing.assert_allclose(g["eta_abs"][0], ref["eta_abs"], rtol=A_RTOL, atol=A_ATOL * w.T)
    np.testing.assert_allclose(g["eta_rel"][0], ref["eta_rel"], rtol=A_RTOL, atol=A_ATOL * w.T)
    np.testing.assert_allclose(g["s_var"][0], float(ref["s_var"]), rtol=SVAR_RTOL)
    np.testing.assert_allclose(g["s_kl"][0], float(ref["s_kl"]), rtol=0, atol=SKL_ATOL)
    o = co.calibration_stats(inp["Q"], inp["K"], rows=rows)
    np.testing.assert_allclose(g["A_mean"][:, rows], o["A_mean"], rtol=A_RTOL, atol=A_ATOL)
    np.testing.assert_allclose(g["eta_abs"].sum(axis=1), w.T, rtol=1e-4)
    np.testing.assert_allclose(g["eta_rel"].sum(axis=1), w.T, rtol=1e-4)


@pytest.mark.slow
def test_calib_full_size_sampled_rows():
    """The same workload with the per-entry squared deviations kept: sampled
    rows of the mean attention and their share of the variance score against
    the oracle; the marginals and the scores against sums over the GPU's own
    state (float64), which hold at any size; the marginals sum to T."""
    from oracle import calib_oracle as co
    w, inp = _full_inputs()
    announce(f"calib full size {w.name} with m2")
    g, _ = _gpu_stats(inp["Q"], inp["K"], w.dtype, (w.micro,) * (w.n_cal // w.micro), keep_m2=True)
    rows = np.array([0, 1, 127, 128, 2049, 4000, w.T - 1])
    o = co.calibration_stats(inp["Q"], inp["K"], rows=rows)
    np.testing.assert_allclose(g["A_mean"][:, rows], o["A_mean"], rtol=A_RTOL, atol=A_ATOL)
    share = g["m2"][:, rows].sum(axis=(1, 2)) / ((w.n_cal - 1) * w.T * w.T)
    np.testing.assert_allclose(share, o["s_var"], rtol=SVAR_RTOL)
    A = g["A_mean"]
    np.testing.assert_allclose(g["eta_abs"], A.sum(axis=1), rtol=1e-4, atol=1e-3)
    rel = np.stack([[np.trace(A[h], offset=-dl) for dl in range(w.T)] for h in range(w.H)])
    np.testing.assert_allclose(g["eta_rel"], rel, rtol=1e-4, atol=1e-3)
    np.testing.assert_allclose(g["eta_abs"].sum(axis=1), w.T, rtol=1e-4)
    np.testing.assert_allclose(g["eta_rel"].sum(axis=1), w.T, rtol=1e-4)
    np.testing.assert_allclose(g["s_var"], g["m2"].sum(axis=(1, 2)) / ((w.n_cal - 1) * w.T * w.T), rtol=1e-4)
    ref = np.load(GOLDEN)
    np.testing.assert_allclose(g["s_var"][0], float(ref["s_var"]), rtol=SVAR_RTOL)
    np.testing.assert_allclose(g["s_kl"][0], float(ref["s_kl"]), rtol=0, atol=SKL_ATOL)
    assert np.all(g["s_kl"] > 0) and np.all(np.isfinite(g["s_kl"]))
