"""Seeded synthetic inputs for the hybrid causal-attention layer.

This module only draws random numbers and rounds them to the storage type; it
holds none of the layer's arithmetic.  Both the GPU path's tests and the CPU
oracle take their inputs from here, so both see bit-identical values.

Value recipe (stand-ins for trained FineWeb-Edu weights and fitted
preference vectors, which are not available):

* ``Q, K, V, dO ~ N(0, 1)``, drawn in float32 and, for bf16 workloads,
  rounded once to bfloat16 (round to nearest even).
* ``a ~ N(0, 1)`` in float32 -- the structured-random control of the paper
  draws its absolute-position preferences this way.
* ``r[k] = -ln(1 + k) + N(0, 0.1^2)`` in float32: a recency decay over the
  key offset ``k = 0..N-1`` standing in for a fitted relative-distance
  preference.
* Fixed heads: the first ``n_fixed`` entries of a seeded permutation of the
  heads, so smaller fixed sets are nested inside larger ones.

Generator: ``numpy.random.Generator(PCG64(SeedSequence([seed, stream_id])))``
with one spawned child stream per tensor.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

SEED = 1337


@dataclass(frozen=True)
class Workload:
    """One layer shape.  ``fixed`` lists the fixed heads explicitly, or is
    ``None`` to draw ``n_fixed`` heads from the seeded permutation."""
    name: str
    B: int
    H: int
    N: int
    d: int
    dtype: str                 # "f32" or "bf16"
    backward: bool
    n_fixed: int = 0
    fixed: Optional[Sequence[int]] = None
    stream_id: int = 0


# The five layer shapes: a tiny fp32 correctness case, a 124M-style layer
# (12 heads, d_h 64, 4K), a 1B-style layer (32 heads, 8K), a long forward-only
# prefill (32K), and the 124M-shape replacement-rate sweep.
WORKLOADS: Dict[str, Workload] = {
    "tiny_f32": Workload("tiny_f32", 1, 4, 256, 64, "f32", True, 1, fixed=(3,), stream_id=1),
    "gpt124m_4k": Workload("gpt124m_4k", 8, 12, 4096, 64, "bf16", True, 3, stream_id=2),
    "gpt1b_8k": Workload("gpt1b_8k", 2, 32, 8192, 64, "bf16", True, 8, stream_id=3),
    "prefill_32k": Workload("prefill_32k", 1, 12, 32768, 64, "bf16", False, 3, stream_id=4),
}
for _nf in (0, 3, 6, 12):
    WORKLOADS[f"sweep124m_{_nf}"] = Workload(
        f"sweep124m_{_nf}", 8, 12, 4096, 64, "bf16", True, _nf, stream_id=5)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns
    float32 holding exactly representable bf16 values.  NaN stays NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    out = rounded.view(np.float32)
    nan = np.isnan(x)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The upper 16 bits of bf16-representable float32 values (uint16)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def _streams(seed: int, stream_id: int, count: int):
    ss = np.random.SeedSequence([seed, stream_id])
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(count)]


def fixed_heads(H: int, n_fixed: int, seed: int = SEED, stream_id: int = 0) -> List[int]:
    """The first ``n_fixed`` heads of a seeded permutation (nested in
    ``n_fixed``)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream_id, 7])))
    perm = g.permutation(H)
    return sorted(int(h) for h in perm[:n_fixed])


def make_inputs(B: int, H: int, N: int, d: int, fixed: Sequence[int], dtype: str,
                seed: int = SEED, stream_id: int = 0, backward: bool = True,
                prior_len: Optional[int] = None) -> dict:
    """Draw one layer's inputs.  Returns float32 arrays ``Q, K, V`` (and
    ``dO`` if ``backward``) of shape ``[B, H, N, d]``, ``a`` and ``r`` of shape
    ``[H, prior_len]`` (default ``N``) and the ``uint8`` head flags
    ``is_fixed`` ``[H]``.  For ``dtype == "bf16"`` the activations hold
    bf16-representable values; ``a`` and ``r`` always stay float32."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(dtype)
    L = N if prior_len is None else prior_len
    gq, gk, gv, gdo, ga, gr = _streams(seed, stream_id, 6)
    shape = (B, H, N, d)

    def act(g):
        x = g.standard_normal(shape, dtype=np.float32)
        return round_to_bf16(x) if dtype == "bf16" else x

    out = {"Q": act(gq), "K": act(gk), "V": act(gv)}
    if backward:
        out["dO"] = act(gdo)
    a = ga.standard_normal((H, L), dtype=np.float32)
    k = np.arange(L, dtype=np.float64)
    r = (-np.log1p(k)[None, :] + 0.1 * gr.standard_normal((H, L))).astype(np.float32)
    is_fixed = np.zeros(H, dtype=np.uint8)
    for h in fixed:
        is_fixed[int(h)] = 1
    out.update(a=a, r=r, is_fixed=is_fixed)
    return out


def workload_inputs(w: Workload, seed: int = SEED) -> dict:
    fixed = list(w.fixed) if w.fixed is not None else fixed_heads(w.H, w.n_fixed, seed, w.stream_id)
    return make_inputs(w.B, w.H, w.N, w.d, fixed, w.dtype, seed, w.stream_id, w.backward)


# ---------------------------------------------------------------------------
# Calibration inputs (the statistics pass that precedes head replacement)
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class CalibWorkload:
    """Queries and keys of one layer on ``n_cal`` calibration inputs of length
    ``T``, folded in micro-batches of ``micro`` inputs."""
    name: str
    n_cal: int
    micro: int
    H: int
    T: int
    d: int
    dtype: str
    stream_id: int = 0


# The 124M-style layer at 4K: 32 calibration sequences in micro-batches of two.
CALIB_WORKLOADS: Dict[str, CalibWorkload] = {
    "calib124m_4k": CalibWorkload("calib124m_4k", 32, 2, 12, 4096, 64, "bf16", stream_id=11),
}

# Calibration queries and keys share a per-head component across inputs, so
# the attention patterns have an input-independent part and an input-dependent
# part: X_n = SHARED * X_common + NOISE * eps_n with SHARED^2 + NOISE^2 = 1.
CALIB_SHARED = 0.8
CALIB_NOISE = 0.6


def calib_inputs(n_cal: int, H: int, T: int, d: int, dtype: str, seed: int = SEED, stream_id: int = 0,
                 first: int = 0, count: Optional[int] = None) -> dict:
    """Draw ``Q, K`` ``[count, H, T, d]`` float32 (bf16-representable for
    ``dtype == "bf16"``) for calibration inputs ``first .. first+count-1`` of
    ``n_cal``.  Input n always gets the same values, whichever slice asks."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(dtype)
    count = n_cal - first if count is None else count
    if first < 0 or count < 0 or first + count > n_cal:
        raise ValueError("input range outside the calibration set")
    gq, gk = _streams(seed, stream_id, 2)
    common_q = gq.standard_normal((H, T, d), dtype=np.float32)
    common_k = gk.standard_normal((H, T, d), dtype=np.float32)
    out = {}
    for name, common, sid in (("Q", common_q, 0), ("K", common_k, 1)):
        x = np.empty((count, H, T, d), dtype=np.float32)
        for i in range(count):
            g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream_id, 100 + sid, first + i])))
            x[i] = CALIB_SHARED * common + CALIB_NOISE * g.standard_normal((H, T, d), dtype=np.float32)
        out[name] = round_to_bf16(x) if dtype == "bf16" else x
    return out


# ---------------------------------------------------------------------------
# Target patterns for the compact fit (stand-ins for calibration means)
# ---------------------------------------------------------------------------

def fit_target_means(H: int, T: int, seed: int = SEED, stream_id: int = 0) -> np.ndarray:
    """Draw ``[H, T, T]`` float32 causal row-stochastic patterns shaped like
    mean attention: per head a sink weight on key 0, a recency decay and
    Gaussian noise, ``s(i, j) = sink [j == 0] - decay ln(1 + i - j) + noise``,
    then a softmax over ``j <= i`` in float64, rounded to float32 (zeros
    above the diagonal)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream_id, 13])))
    out = np.zeros((H, T, T), dtype=np.float32)
    i = np.arange(T)
    off = i[:, None] - i[None, :]
    causal = off >= 0
    for h in range(H):
        sink, decay, noise = g.uniform(0.0, 4.0), g.uniform(0.2, 1.5), g.uniform(0.2, 1.5)
        s = -decay * np.log1p(np.clip(off, 0, None)) + noise * g.standard_normal((T, T))
        s[:, 0] += sink
        s = np.where(causal, s, -np.inf)
        s -= s.max(axis=1, keepdims=True)
        e = np.exp(s)
        out[h] = (e / e.sum(axis=1, keepdims=True)).astype(np.float32)
    return out
