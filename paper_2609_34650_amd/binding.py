"""Thin ctypes binding to libsaf.so (C ABI in ``include/saf.h``,
``include/saf_calib.h`` and ``include/saf_fit.h``).

Only argument marshalling happens here: tensor checks, pointers, the head
flags and the caller's current HIP stream.  Every step of the layer runs in
the library's kernels; there is no fallback.  If ``libsaf.so`` is missing or
fails to load, every call raises.

Function names match the C entry points.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsaf.so")

SAF_DTYPE_F32 = 0
SAF_DTYPE_BF16 = 1
SAF_BWD_PREPROCESS = 0
SAF_BWD_DKDV = 1
SAF_BWD_DQ = 2
SAF_BWD_DQ_WITH_D = 3

STATUS = {
    0: "SAF_OK",
    1: "SAF_ERR_NULL",
    2: "SAF_ERR_SHAPE",
    3: "SAF_ERR_UNSUPPORTED",
    4: "SAF_ERR_MISSING_PRIOR",
    5: "SAF_ERR_LAUNCH",
    6: "SAF_ERR_ALIGNMENT",
    7: "SAF_ERR_FLAG",
}

EXPORTS = (
    "saf_hybrid_attn_fwd",
    "saf_hybrid_attn_fwd_gqa",
    "saf_hybrid_attn_bwd_gqa_workspace_bytes",
    "saf_hybrid_attn_bwd_gqa",
    "saf_hybrid_attn_bwd_workspace_bytes",
    "saf_hybrid_attn_bwd",
    "saf_hybrid_attn_bwd_stage",
    "saf_hybrid_attn_bwd_pattern_workspace_bytes",
    "saf_hybrid_attn_bwd_pattern",
    "saf_status_str",
    "saf_calib_accumulate",
    "saf_calib_stats_bytes",
    "saf_calib_finalize_workspace_bytes",
    "saf_calib_finalize",
    "saf_fit_workspace_bytes",
    "saf_fit_targets",
    "saf_compact_fit",
    "saf_hybrid_attn_bwd_noalloc",
    "saf_clock_probe",
    "saf_lds_read_probe",
    "saf_lds_pattern_probe",
    "saf_mfma_rate_probe",
)


class SafError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {STATUS.get(code, code)} ({status_str(code)})")


_lib = None


def lib_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load libsaf.so once; raise if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"{_LIB_PATH} is not built; run `python -m paper_2609_34650_amd.build` "
            "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i, f32p, u8p = ctypes.c_void_p, ctypes.c_int, ctypes.POINTER(ctypes.c_float), ctypes.c_void_p
    lib.saf_hybrid_attn_fwd.restype = ctypes.c_int
    lib.saf_hybrid_attn_fwd.argtypes = [i, vp, vp, vp, u8p, vp, vp, i, i, i, i, i, vp, vp, vp]
    lib.saf_hybrid_attn_fwd_gqa.restype = ctypes.c_int
    lib.saf_hybrid_attn_fwd_gqa.argtypes = [i, vp, vp, vp, u8p, vp, vp, i, i, i, i, i, i, vp, vp, vp]
    lib.saf_hybrid_attn_bwd_gqa_workspace_bytes.restype = ctypes.c_size_t
    lib.saf_hybrid_attn_bwd_gqa_workspace_bytes.argtypes = [i, i, i, i, i, i]
    lib.saf_hybrid_attn_bwd_gqa.restype = ctypes.c_int
    lib.saf_hybrid_attn_bwd_gqa.argtypes = [i, vp, vp, vp, vp, vp, vp, u8p, vp, vp, i, i, i, i, i, i, vp, vp, vp,
                                            vp, ctypes.c_size_t, vp]
    lib.saf_hybrid_attn_bwd_workspace_bytes.restype = ctypes.c_size_t
    lib.saf_hybrid_attn_bwd_workspace_bytes.argtypes = [i, i, i, i, i]
    bwd_args = [i, vp, vp, vp, vp, vp, vp, u8p, vp, vp, i, i, i, i, i, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.saf_hybrid_attn_bwd.restype = ctypes.c_int
    lib.saf_hybrid_attn_bwd.argtypes = bwd_args
    lib.saf_hybrid_attn_bwd_noalloc.restype = ctypes.c_int
    lib.saf_hybrid_attn_bwd_noalloc.argtypes = bwd_args[:18] + [vp]
    lib.saf_hybrid_attn_bwd_stage.restype = ctypes.c_int
    lib.saf_hybrid_attn_bwd_stage.argtypes = [i] + bwd_args
    lib.saf_hybrid_attn_bwd_pattern_workspace_bytes.restype = ctypes.c_size_t
    lib.saf_hybrid_attn_bwd_pattern_workspace_bytes.argtypes = [i, i, i, i, i]
    lib.saf_hybrid_attn_bwd_pattern.restype = ctypes.c_int
    lib.saf_hybrid_attn_bwd_pattern.argtypes = [i, vp, vp, vp, vp, u8p, vp, vp, i, i, i, i, i, vp, vp, vp,
                                                ctypes.c_size_t, vp]
    lib.saf_calib_accumulate.restype = ctypes.c_int
    lib.saf_calib_accumulate.argtypes = [i, vp, vp, vp, i, i, i, i, i, vp, vp, vp, vp]
    lib.saf_calib_stats_bytes.restype = ctypes.c_size_t
    lib.saf_calib_stats_bytes.argtypes = [i, i]
    lib.saf_calib_finalize_workspace_bytes.restype = ctypes.c_size_t
    lib.saf_calib_finalize_workspace_bytes.argtypes = [i, i]
    lib.saf_calib_finalize.restype = ctypes.c_int
    lib.saf_calib_finalize.argtypes = [i, i, i, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.saf_fit_workspace_bytes.restype = ctypes.c_size_t
    lib.saf_fit_workspace_bytes.argtypes = [i, i]
    lib.saf_fit_targets.restype = ctypes.c_int
    lib.saf_fit_targets.argtypes = [i, i, vp, ctypes.c_float, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.saf_compact_fit.restype = ctypes.c_int
    lib.saf_compact_fit.argtypes = [i, i, vp, vp, vp, i, ctypes.c_float, ctypes.c_float, vp, vp, vp, vp, vp,
                                    ctypes.c_size_t, vp]
    lib.saf_clock_probe.restype = ctypes.c_int
    lib.saf_clock_probe.argtypes = [vp, i, vp]
    lib.saf_lds_read_probe.restype = ctypes.c_int
    lib.saf_lds_read_probe.argtypes = [vp, ctypes.c_size_t, vp, vp]
    lib.saf_lds_pattern_probe.restype = ctypes.c_int
    lib.saf_lds_pattern_probe.argtypes = [i, i, vp, vp]
    lib.saf_mfma_rate_probe.restype = ctypes.c_int
    lib.saf_mfma_rate_probe.argtypes = [i, i, i, vp, vp, vp]
    lib.saf_status_str.restype = ctypes.c_char_p
    lib.saf_status_str.argtypes = [i]
    del f32p
    _lib = lib
    return lib


def status_str(code: int) -> str:
    return load().saf_status_str(int(code)).decode()


# ---------------------------------------------------------------------------
# Marshalling helpers
# ---------------------------------------------------------------------------

def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SAF_DTYPE_BF16
    if t.dtype == torch.float32:
        return SAF_DTYPE_F32
    raise TypeError(f"activations must be bfloat16 or float32, got {t.dtype}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _check_act(name: str, t: Optional[torch.Tensor], shape, dtype, device, allow_none=False):
    if t is None:
        if allow_none:
            return
        raise ValueError(f"{name} is required")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous [B, H, N, d]")


def _flags(head_is_fixed, H: int) -> np.ndarray:
    if isinstance(head_is_fixed, torch.Tensor):
        head_is_fixed = head_is_fixed.detach().cpu().numpy()
    flags = np.ascontiguousarray(np.asarray(head_is_fixed, dtype=np.uint8).reshape(-1))
    if flags.shape[0] != H:
        raise ValueError(f"head_is_fixed has {flags.shape[0]} entries for {H} heads")
    return flags


def _prior(name: str, t: Optional[torch.Tensor], H: int, N: int, device) -> Tuple[Optional[int], int]:
    if t is None:
        return None, N
    if t.dim() != 2 or t.shape[0] != H or t.shape[1] < N:
        raise ValueError(f"{name} must be [H, >=N] float32, got {tuple(t.shape)}")
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32")
    if t.device != device or t.stride(1) != 1 or t.stride(0) < N:
        raise ValueError(f"{name} must be on {device} with unit stride along positions")
    return t.data_ptr(), t.stride(0)


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _raise(code: int, what: str):
    if code != 0:
        raise SafError(code, what)


# ---------------------------------------------------------------------------
# Entry points
# ---------------------------------------------------------------------------

def saf_hybrid_attn_fwd(Q: Optional[torch.Tensor], K: Optional[torch.Tensor], V: torch.Tensor,
                        head_is_fixed: Sequence[int], a: Optional[torch.Tensor] = None,
                        r: Optional[torch.Tensor] = None, O: Optional[torch.Tensor] = None,
                        LSE: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Forward of the hybrid layer on the current stream.  Returns ``(O, LSE)``.
    ``Q`` and ``K`` may be ``None`` when every head is fixed."""
    lib = load()
    B, H, N, d = V.shape
    dev = V.device
    _check_act("V", V, V.shape, V.dtype, dev)
    _check_act("Q", Q, V.shape, V.dtype, dev, allow_none=True)
    _check_act("K", K, V.shape, V.dtype, dev, allow_none=True)
    if O is None:
        O = torch.empty_like(V)
    if LSE is None:
        LSE = torch.empty((B, H, N), dtype=torch.float32, device=dev)
    _check_act("O", O, V.shape, V.dtype, dev)
    _check_act("LSE", LSE, (B, H, N), torch.float32, dev)
    flags = _flags(head_is_fixed, H)
    pa, lda = _prior("a", a, H, N, dev)
    pr, ldr = _prior("r", r, H, N, dev)
    if pa is not None and pr is not None and lda != ldr:
        raise ValueError("a and r must share one row stride")
    code = lib.saf_hybrid_attn_fwd(
        _dtype_code(V), _ptr(Q), _ptr(K), _ptr(V), flags.ctypes.data, pa, pr, lda,
        B, H, N, d, _ptr(O), _ptr(LSE), _stream(dev))
    _raise(code, "saf_hybrid_attn_fwd")
    return O, LSE


def saf_hybrid_attn_fwd_gqa(Q: Optional[torch.Tensor], K: Optional[torch.Tensor], V: torch.Tensor,
                            head_is_fixed: Sequence[int], a: Optional[torch.Tensor] = None,
                            r: Optional[torch.Tensor] = None, O: Optional[torch.Tensor] = None,
                            LSE: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Grouped-query forward: ``Q`` ``[B, Hq, N, d]``, ``K``, ``V``
    ``[B, Hkv, N, d]`` (d in 64, 96, 128).  Returns ``(O, LSE)``."""
    lib = load()
    B, Hkv, N, d = V.shape
    dev = V.device
    _check_act("V", V, V.shape, V.dtype, dev)
    _check_act("K", K, V.shape, V.dtype, dev, allow_none=True)
    flags = np.ascontiguousarray(np.asarray(
        head_is_fixed.detach().cpu().numpy() if isinstance(head_is_fixed, torch.Tensor) else head_is_fixed,
        dtype=np.uint8).reshape(-1))
    Hq = flags.shape[0]
    _check_act("Q", Q, (B, Hq, N, d), V.dtype, dev, allow_none=True)
    if O is None:
        O = torch.empty((B, Hq, N, d), dtype=V.dtype, device=dev)
    if LSE is None:
        LSE = torch.empty((B, Hq, N), dtype=torch.float32, device=dev)
    _check_act("O", O, (B, Hq, N, d), V.dtype, dev)
    _check_act("LSE", LSE, (B, Hq, N), torch.float32, dev)
    pa, lda = _prior("a", a, Hq, N, dev)
    pr, ldr = _prior("r", r, Hq, N, dev)
    if pa is not None and pr is not None and lda != ldr:
        raise ValueError("a and r must share one row stride")
    code = lib.saf_hybrid_attn_fwd_gqa(_dtype_code(V), _ptr(Q), _ptr(K), _ptr(V), flags.ctypes.data, pa, pr, lda,
                                       B, Hq, Hkv, N, d, _ptr(O), _ptr(LSE), _stream(dev))
    _raise(code, "saf_hybrid_attn_fwd_gqa")
    return O, LSE


def saf_hybrid_attn_bwd_gqa(Q, K, V, O, dO, LSE, head_is_fixed, a=None, r=None, dQ=None, dK=None, dV=None,
                            workspace: Optional[torch.Tensor] = None):
    """Grouped-query backward for ``sum(O * dO)``: ``Q``, ``O``, ``dO``
    ``[B, Hq, N, d]``, ``K``, ``V`` ``[B, Hkv, N, d]``.  Returns ``(dQ, dK,
    dV)`` with dK and dV summed over each group."""
    lib = load()
    B, Hkv, N, d = V.shape
    dev = V.device
    if isinstance(head_is_fixed, torch.Tensor):
        head_is_fixed = head_is_fixed.detach().cpu().numpy()
    flags = np.ascontiguousarray(np.asarray(head_is_fixed, dtype=np.uint8).reshape(-1))
    Hq = flags.shape[0]
    qshape = (B, Hq, N, d)
    _check_act("V", V, V.shape, V.dtype, dev)
    _check_act("K", K, V.shape, V.dtype, dev, allow_none=True)
    _check_act("Q", Q, qshape, V.dtype, dev, allow_none=True)
    for name, t in (("O", O), ("dO", dO)):
        _check_act(name, t, qshape, V.dtype, dev)
    _check_act("LSE", LSE, (B, Hq, N), torch.float32, dev)
    dQ = torch.empty(qshape, dtype=V.dtype, device=dev) if dQ is None else dQ
    dK = torch.empty_like(V) if dK is None else dK
    dV = torch.empty_like(V) if dV is None else dV
    _check_act("dQ", dQ, qshape, V.dtype, dev)
    _check_act("dK", dK, V.shape, V.dtype, dev)
    _check_act("dV", dV, V.shape, V.dtype, dev)
    code = SAF_DTYPE_BF16 if V.dtype == torch.bfloat16 else SAF_DTYPE_F32
    nbytes = int(lib.saf_hybrid_attn_bwd_gqa_workspace_bytes(code, B, Hq, Hkv, N, d))
    if workspace is None:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    pa, lda = _prior("a", a, Hq, N, dev)
    pr, ldr = _prior("r", r, Hq, N, dev)
    if pa is not None and pr is not None and lda != ldr:
        raise ValueError("a and r must share one row stride")
    _raise(lib.saf_hybrid_attn_bwd_gqa(_dtype_code(V), _ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(dO), _ptr(LSE),
                                       flags.ctypes.data, pa, pr, lda, B, Hq, Hkv, N, d, _ptr(dQ), _ptr(dK),
                                       _ptr(dV), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                       _stream(dev)), "saf_hybrid_attn_bwd_gqa")
    return dQ, dK, dV


def saf_hybrid_attn_bwd_workspace_bytes(dtype: torch.dtype, B: int, H: int, N: int, d: int) -> int:
    code = SAF_DTYPE_BF16 if dtype == torch.bfloat16 else SAF_DTYPE_F32
    return int(load().saf_hybrid_attn_bwd_workspace_bytes(code, B, H, N, d))


def _bwd_common(Q, K, V, O, dO, LSE, head_is_fixed, a, r, dQ, dK, dV, workspace):
    B, H, N, d = V.shape
    dev = V.device
    for name, t in (("V", V), ("O", O), ("dO", dO)):
        _check_act(name, t, V.shape, V.dtype, dev)
    _check_act("Q", Q, V.shape, V.dtype, dev, allow_none=True)
    _check_act("K", K, V.shape, V.dtype, dev, allow_none=True)
    _check_act("LSE", LSE, (B, H, N), torch.float32, dev)
    dQ = torch.empty_like(V) if dQ is None else dQ
    dK = torch.empty_like(V) if dK is None else dK
    dV = torch.empty_like(V) if dV is None else dV
    for name, t in (("dQ", dQ), ("dK", dK), ("dV", dV)):
        _check_act(name, t, V.shape, V.dtype, dev)
    nbytes = saf_hybrid_attn_bwd_workspace_bytes(V.dtype, B, H, N, d)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    flags = _flags(head_is_fixed, H)
    pa, lda = _prior("a", a, H, N, dev)
    pr, ldr = _prior("r", r, H, N, dev)
    if pa is not None and pr is not None and lda != ldr:
        raise ValueError("a and r must share one row stride")
    args = [_dtype_code(V), _ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(dO), _ptr(LSE), flags.ctypes.data,
            pa, pr, lda, B, H, N, d, _ptr(dQ), _ptr(dK), _ptr(dV), workspace.data_ptr(),
            workspace.numel() * workspace.element_size(), _stream(dev)]
    return args, (dQ, dK, dV), flags, workspace


def saf_hybrid_attn_bwd(Q, K, V, O, dO, LSE, head_is_fixed, a=None, r=None, dQ=None, dK=None, dV=None,
                        workspace: Optional[torch.Tensor] = None):
    """Backward of the hybrid layer for ``sum(O * dO)`` on the current
    stream.  Returns ``(dQ, dK, dV)``; fixed heads get zeros in dQ and dK."""
    lib = load()
    args, outs, _flags_keep, _ws_keep = _bwd_common(Q, K, V, O, dO, LSE, head_is_fixed, a, r, dQ, dK, dV,
                                                    workspace)
    _raise(lib.saf_hybrid_attn_bwd(*args), "saf_hybrid_attn_bwd")
    return outs


def saf_hybrid_attn_bwd_noalloc(Q, K, V, O, dO, LSE, head_is_fixed, a=None, r=None, dQ=None, dK=None,
                                dV=None):
    """Backward through ``saf_hybrid_attn_bwd_noalloc``: no workspace (the
    library's per-GPU scratch array holds D).  Returns ``(dQ, dK, dV)``, the
    outputs as passed (or allocated here when None)."""
    lib = load()
    args, outs, _flags_keep, _ws_keep = _bwd_common(Q, K, V, O, dO, LSE, head_is_fixed, a, r, dQ, dK, dV,
                                                    torch.empty(0, dtype=torch.uint8, device=V.device))
    _raise(lib.saf_hybrid_attn_bwd_noalloc(*(args[:18] + [args[-1]])), "saf_hybrid_attn_bwd_noalloc")
    return outs


def saf_hybrid_attn_bwd_stage(stage: int, Q, K, V, O, dO, LSE, head_is_fixed, a=None, r=None, dQ=None,
                              dK=None, dV=None, workspace: Optional[torch.Tensor] = None):
    """One launch of the backward (``SAF_BWD_PREPROCESS``, ``SAF_BWD_DKDV``,
    ``SAF_BWD_DQ``, ``SAF_BWD_DQ_WITH_D``); returns ``(dQ, dK, dV)`` as passed
    or allocated.  Pass the same ``workspace`` to every stage:
    ``SAF_BWD_DQ_WITH_D`` then ``SAF_BWD_DKDV`` are the launches of
    ``saf_hybrid_attn_bwd``."""
    lib = load()
    args, outs, _flags_keep, _ws_keep = _bwd_common(Q, K, V, O, dO, LSE, head_is_fixed, a, r, dQ, dK, dV,
                                                    workspace)
    _raise(lib.saf_hybrid_attn_bwd_stage(int(stage), *args), "saf_hybrid_attn_bwd_stage")
    return outs


def saf_hybrid_attn_bwd_pattern(V, O, dO, LSE, head_is_fixed, a, r, da=None, dr=None,
                                workspace: Optional[torch.Tensor] = None):
    """Gradients ``(da, dr)`` ``[H, N]`` float32 of ``sum(O * dO)`` with
    respect to the fixed heads' ``a`` and ``r`` (summed over the batch); rows
    of ordinary heads are zero."""
    lib = load()
    B, H, N, d = V.shape
    dev = V.device
    for name, t in (("V", V), ("O", O), ("dO", dO)):
        _check_act(name, t, V.shape, V.dtype, dev)
    _check_act("LSE", LSE, (B, H, N), torch.float32, dev)
    da = torch.empty((H, N), dtype=torch.float32, device=dev) if da is None else da
    dr = torch.empty((H, N), dtype=torch.float32, device=dev) if dr is None else dr
    _check_act("da", da, (H, N), torch.float32, dev)
    _check_act("dr", dr, (H, N), torch.float32, dev)
    code = SAF_DTYPE_BF16 if V.dtype == torch.bfloat16 else SAF_DTYPE_F32
    nbytes = int(lib.saf_hybrid_attn_bwd_pattern_workspace_bytes(code, B, H, N, d))
    if workspace is None:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    flags = _flags(head_is_fixed, H)
    pa, lda = _prior("a", a, H, N, dev)
    pr, ldr = _prior("r", r, H, N, dev)
    if pa is not None and pr is not None and lda != ldr:
        raise ValueError("a and r must share one row stride")
    code = lib.saf_hybrid_attn_bwd_pattern(
        _dtype_code(V), _ptr(V), _ptr(O), _ptr(dO), _ptr(LSE), flags.ctypes.data, pa, pr, lda, B, H, N, d,
        _ptr(da), _ptr(dr), workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(dev))
    _raise(code, "saf_hybrid_attn_bwd_pattern")
    return da, dr


class HybridAttention(torch.autograd.Function):
    """Autograd wrapper over the forward/backward pair.  Fixed heads return
    zero gradients for Q and K.  ``a`` and ``r`` take a gradient only when
    they require one (trainable fixed patterns): then the backward also runs
    ``saf_hybrid_attn_bwd_pattern``; its ``[H, N]`` result goes into the
    first N columns of a gradient shaped like ``a`` (later columns and
    ordinary heads' rows are zero)."""

    @staticmethod
    def forward(ctx, Q, K, V, head_is_fixed, a, r):
        O, LSE = saf_hybrid_attn_fwd(Q, K, V, head_is_fixed, a, r)
        ctx.save_for_backward(Q, K, V, O, LSE, a, r)
        ctx.flags = _flags(head_is_fixed, V.shape[1])
        return O

    @staticmethod
    def backward(ctx, dO):
        Q, K, V, O, LSE, a, r = ctx.saved_tensors
        dO = dO.contiguous()
        dQ, dK, dV = saf_hybrid_attn_bwd(Q, K, V, O, dO, LSE, ctx.flags, a, r)
        ga = gr = None
        if ctx.needs_input_grad[4] or ctx.needs_input_grad[5]:
            N = V.shape[2]
            da, dr = saf_hybrid_attn_bwd_pattern(V, O, dO, LSE, ctx.flags, a.detach(), r.detach())
            if ctx.needs_input_grad[4]:
                ga = torch.zeros_like(a)
                ga[:, :N] = da
            if ctx.needs_input_grad[5]:
                gr = torch.zeros_like(r)
                gr[:, :N] = dr
        return dQ, dK, dV, None, ga, gr


class HybridAttentionGQA(torch.autograd.Function):
    """Autograd wrapper over the grouped-query pair (Q ``[B, Hq, N, d]``, K
    and V ``[B, Hkv, N, d]``, d in {64, 96, 128}).  Patterns are frozen:
    ``a`` and ``r`` take no gradient; fixed query heads get zero dQ and add
    only to their group's dV."""

    @staticmethod
    def forward(ctx, Q, K, V, head_is_fixed, a, r):
        O, LSE = saf_hybrid_attn_fwd_gqa(Q, K, V, head_is_fixed, a, r)
        ctx.save_for_backward(Q, K, V, O, LSE, a, r)
        ctx.flags = _flags(head_is_fixed, Q.shape[1])
        return O

    @staticmethod
    def backward(ctx, dO):
        Q, K, V, O, LSE, a, r = ctx.saved_tensors
        dQ, dK, dV = saf_hybrid_attn_bwd_gqa(Q, K, V, O, dO.contiguous(), LSE, ctx.flags, a, r)
        return dQ, dK, dV, None, None, None


# ---------------------------------------------------------------------------
# Calibration statistics
# ---------------------------------------------------------------------------

class CalibState:
    """Running calibration statistics of one layer on one device: ``mean``
    ``[H, T, T]`` float32, optionally ``m2`` ``[H, T, T]`` float32 (per-entry
    squared deviations), the library's float64 partial sums ``stats``, and the
    number of inputs folded in so far."""

    def __init__(self, H: int, T: int, device, keep_m2: bool = False):
        self.mean = torch.empty((H, T, T), dtype=torch.float32, device=device)
        self.m2 = torch.empty((H, T, T), dtype=torch.float32, device=device) if keep_m2 else None
        nbytes = int(load().saf_calib_stats_bytes(H, T))
        if nbytes == 0:
            raise ValueError(f"unsupported calibration shape H={H} T={T}")
        self.stats = torch.empty((nbytes // 8,), dtype=torch.float64, device=device)
        self.n_seen = 0


def saf_calib_accumulate(Q: torch.Tensor, K: torch.Tensor, LSE: torch.Tensor, state: CalibState) -> CalibState:
    """Fold one micro-batch (``Q, K`` ``[B, H, T, d]``, ``LSE`` ``[B, H, T]``
    from the all-ordinary forward) into ``state`` on the current stream."""
    lib = load()
    B, H, T, d = Q.shape
    dev = Q.device
    _check_act("Q", Q, Q.shape, Q.dtype, dev)
    _check_act("K", K, Q.shape, Q.dtype, dev)
    _check_act("LSE", LSE, (B, H, T), torch.float32, dev)
    _check_act("mean", state.mean, (H, T, T), torch.float32, dev)
    _check_act("m2", state.m2, (H, T, T), torch.float32, dev, allow_none=True)
    _check_act("stats", state.stats, (int(lib.saf_calib_stats_bytes(H, T)) // 8,), torch.float64, dev)
    code = lib.saf_calib_accumulate(_dtype_code(Q), _ptr(Q), _ptr(K), _ptr(LSE), B, H, T, d, state.n_seen,
                                    _ptr(state.mean), _ptr(state.m2), _ptr(state.stats), _stream(dev))
    _raise(code, "saf_calib_accumulate")
    state.n_seen += B
    return state


def saf_calib_finalize_workspace_bytes(H: int, T: int) -> int:
    return int(load().saf_calib_finalize_workspace_bytes(H, T))


def saf_calib_finalize(state: CalibState, workspace: Optional[torch.Tensor] = None):
    """Scores and marginals of ``state`` on the current stream.  Returns a dict
    with ``A_mean`` (the state's ``mean``), ``eta_abs``, ``eta_rel`` ``[H, T]``
    and ``s_var``, ``s_kl`` ``[H]`` (float32)."""
    lib = load()
    H, T, _ = state.mean.shape
    dev = state.mean.device
    out = {name: torch.empty(shape, dtype=torch.float32, device=dev)
           for name, shape in (("eta_abs", (H, T)), ("eta_rel", (H, T)), ("s_var", (H,)), ("s_kl", (H,)))}
    nbytes = saf_calib_finalize_workspace_bytes(H, T)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    code = lib.saf_calib_finalize(H, T, state.n_seen, _ptr(state.mean), _ptr(state.stats),
                                  _ptr(out["eta_abs"]), _ptr(out["eta_rel"]), _ptr(out["s_var"]),
                                  _ptr(out["s_kl"]), workspace.data_ptr(),
                                  workspace.numel() * workspace.element_size(), _stream(dev))
    _raise(code, "saf_calib_finalize")
    out["A_mean"] = state.mean
    return out


# ---------------------------------------------------------------------------
# Compact fit
# ---------------------------------------------------------------------------

FIT_FLOOR = 1e-9
FIT_STEPS = 400
FIT_LR = 0.05
FIT_ACCEPT_KL = 0.2


def _fit_workspace(H: int, T: int, dev, workspace):
    nbytes = int(load().saf_fit_workspace_bytes(H, T))
    if nbytes == 0:
        raise ValueError(f"unsupported fit shape H={H} T={T}")
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    return workspace


def saf_fit_targets(mean: torch.Tensor, floor_value: float = FIT_FLOOR, workspace: Optional[torch.Tensor] = None):
    """Target marginals of the compact fit from the calibration mean
    ``[H, T, T]``: returns ``(eta_abs, eta_rel, neg_entropy)``."""
    lib = load()
    H, T, _ = mean.shape
    dev = mean.device
    _check_act("mean", mean, (H, T, T), torch.float32, dev)
    eta_abs = torch.empty((H, T), dtype=torch.float32, device=dev)
    eta_rel = torch.empty_like(eta_abs)
    neg_entropy = torch.empty((H,), dtype=torch.float64, device=dev)
    workspace = _fit_workspace(H, T, dev, workspace)
    code = lib.saf_fit_targets(H, T, _ptr(mean), float(floor_value), _ptr(eta_abs), _ptr(eta_rel), _ptr(neg_entropy),
                               workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(dev))
    _raise(code, "saf_fit_targets")
    return eta_abs, eta_rel, neg_entropy


def saf_compact_fit(eta_abs: torch.Tensor, eta_rel: torch.Tensor, neg_entropy: torch.Tensor,
                    steps: int = FIT_STEPS, lr: float = FIT_LR, floor_value: float = FIT_FLOOR,
                    workspace: Optional[torch.Tensor] = None):
    """Fit every head: returns ``(a, r, log_z, kl)`` (``[H, T]``, ``[H, T]``,
    ``[H, T]``, ``[H]`` float32); a head passes when ``kl <= 0.2``."""
    lib = load()
    H, T = eta_abs.shape
    dev = eta_abs.device
    _check_act("eta_abs", eta_abs, (H, T), torch.float32, dev)
    _check_act("eta_rel", eta_rel, (H, T), torch.float32, dev)
    _check_act("neg_entropy", neg_entropy, (H,), torch.float64, dev)
    a = torch.empty((H, T), dtype=torch.float32, device=dev)
    r = torch.empty_like(a)
    log_z = torch.empty_like(a)
    kl = torch.empty((H,), dtype=torch.float32, device=dev)
    workspace = _fit_workspace(H, T, dev, workspace)
    code = lib.saf_compact_fit(H, T, _ptr(eta_abs), _ptr(eta_rel), _ptr(neg_entropy), int(steps), float(lr),
                               float(floor_value), _ptr(a), _ptr(r), _ptr(log_z), _ptr(kl), workspace.data_ptr(),
                               workspace.numel() * workspace.element_size(), _stream(dev))
    _raise(code, "saf_compact_fit")
    return a, r, log_z, kl


# ---------------------------------------------------------------------------
# Measurement aids (include/saf_measure.h)
# ---------------------------------------------------------------------------

def saf_clock_probe(out: torch.Tensor, duration_us: int, stream: Optional["torch.cuda.Stream"] = None):
    """Enqueue the shader-clock probe on `stream` (default: the current
    stream).  `out` is a device int64 tensor of 2 elements; after the stream
    completes, out[0] / out[1] * 100 is the mean shader clock in MHz."""
    if out.dtype != torch.int64 or out.numel() < 2 or not out.is_cuda:
        raise ValueError("out must be a device int64 tensor with 2 elements")
    st = (stream or torch.cuda.current_stream(out.device)).cuda_stream
    _raise(load().saf_clock_probe(out.data_ptr(), int(duration_us), st), "saf_clock_probe")


def saf_lds_read_probe(src: torch.Tensor, sink: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Read every byte of the contiguous device tensor `src` once through
    buffer loads straight to LDS (a known-size reference for HBM byte
    counters); returns the per-workgroup sink."""
    nbytes = src.numel() * src.element_size()
    if not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous device tensor")
    n_wg = (nbytes + (1 << 20) - 1) >> 20
    if sink is None:
        sink = torch.empty(n_wg, dtype=torch.float32, device=src.device)
    _raise(load().saf_lds_read_probe(src.data_ptr(), nbytes, sink.data_ptr(), _stream(src.device)),
           "saf_lds_read_probe")
    return sink


LDS_PATTERNS = ("row operand 32x32", "transposed 32x32 (accumulator order)", "row operand 16x16",
                "transposed 16x16", "row floats 32x32 order", "row floats 16x16 order",
                "transposed 32x32 (natural order)")


def saf_lds_pattern_probe(pattern: int, iters: int, sink: torch.Tensor):
    """Enqueue one LDS read pattern of the layer kernels (LDS_PATTERNS) on the
    current stream; `sink` is a device int32 tensor of at least 65536
    elements (written only under a condition no pattern meets)."""
    if sink.dtype != torch.int32 or sink.numel() < 65536 or not sink.is_cuda:
        raise ValueError("sink must be a device int32 tensor with at least 65536 elements")
    _raise(load().saf_lds_pattern_probe(int(pattern), int(iters), sink.data_ptr(), _stream(sink.device)),
           "saf_lds_pattern_probe")


def saf_mfma_rate_probe(shape: int, waves_per_simd: int, iters: int, clk: torch.Tensor, sink: torch.Tensor):
    """Enqueue the MFMA rate probe (shape 0: 32x32x16 bf16, 1: 16x16x32 bf16)
    on the current stream.  `clk`: device int64 tensor of 2 (shader cycles and
    100 MHz ticks of workgroup 0); `sink`: device float32 tensor of at least
    16384 elements.  FLOP per launch: 2 * 131072 * iters * 1024 *
    waves_per_simd."""
    if clk.dtype != torch.int64 or clk.numel() < 2 or not clk.is_cuda:
        raise ValueError("clk must be a device int64 tensor with 2 elements")
    if sink.dtype != torch.float32 or sink.numel() < 16384 or not sink.is_cuda:
        raise ValueError("sink must be a device float32 tensor with at least 16384 elements")
    _raise(load().saf_mfma_rate_probe(int(shape), int(waves_per_simd), int(iters), clk.data_ptr(), sink.data_ptr(),
                                      _stream(clk.device)), "saf_mfma_rate_probe")
