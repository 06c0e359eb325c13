"""Host-side checks of bench.py's accounting (no GPU): the counted FLOP of
each layer workload against the counting rule worked out by hand, and the
refusal of multi-GPU runs."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _by_hand(B, H, N, d, n_fixed, backward=True):
    # One causal N x N x d contraction: d multiply-adds for each of the
    # N(N+1)/2 visible (query, key) pairs.  Ordinary head: 2 forward + 5
    # backward; fixed head: 1 + 1.
    pairs = N * (N + 1) // 2
    c = 2 * d * pairs * B
    per_ord = 7 if backward else 2
    per_fix = 2 if backward else 1
    return c * (per_ord * (H - n_fixed) + per_fix * n_fixed)


@pytest.mark.parametrize("B,H,N,d,n_fixed,backward,expected", [
    (8, 12, 4096, 64, 3, True, 5.9285e11),     # the 124M layer, 3 of 12 heads fixed
    (8, 12, 4096, 64, 0, True, 7.2173e11),     # the same, every head ordinary
    (2, 32, 8192, 64, 8, True, 1.5807e12),     # the 1B-style 8K layer
    (1, 12, 32768, 64, 3, False, 1.4432e12),   # the 32K prefill, forward only
    (8, 12, 4096, 64, 12, True, 2.062e11),     # every head fixed
])
def test_layer_flop_matches_counting_rule(B, H, N, d, n_fixed, backward, expected):
    got = sum(bench.layer_flop(B, H, N, d, n_fixed, backward).values())
    assert got == pytest.approx(_by_hand(B, H, N, d, n_fixed, backward), rel=1e-12)
    assert got == pytest.approx(expected, rel=2e-4)


def test_layer_flop_stages():
    """Forward 2C per ordinary and 1C per fixed head; the query-block pass 1C
    per ordinary head; the key-block pass 4C per ordinary and 1C per fixed."""
    c = bench.contraction_flop(256, 64)
    f = bench.layer_flop(1, 4, 256, 64, 1)
    assert f == {"fwd": 7 * c, "bwd_dq": 3 * c, "bwd_dkdv": 13 * c}


def test_multi_gpu_request_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert out.returncode == 2
    msg = json.loads(out.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]
