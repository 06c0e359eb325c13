"""C ABI checks that need no GPU: libsaf.so loads, exports exactly the entry
points include/*.h declare, and rejects bad arguments with the documented
status before anything is launched.  Device pointers here are fake (aligned
integers that are never dereferenced: every call below fails validation)."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
                 if f.endswith(".h"))


@pytest.fixture(scope="module")
def lib():
    from paper_2609_34650_amd import binding
    return binding.load()


def _declared():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(saf_\w+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    from paper_2609_34650_amd import binding
    assert _declared() == sorted(binding.EXPORTS)


def test_library_exports_every_declared_symbol_and_nothing_else(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", lib._name], capture_output=True, text=True, check=True)
    exported = sorted(ln.split()[-1] for ln in out.stdout.splitlines() if ln.split()[-1].startswith("saf_"))
    assert exported == _declared()
    for name in _declared():
        assert getattr(lib, name) is not None


FAKE = 1 << 20  # aligned, never dereferenced


def _fwd(lib, dt=1, Q=FAKE, K=FAKE, V=FAKE, flags=(0, 1), a=FAKE, r=FAKE, ld=None, B=1, N=8, d=64,
         O=FAKE, LSE=FAKE):
    f = np.asarray(flags, dtype=np.uint8)
    H = f.shape[0]
    ld = N if ld is None else ld
    return lib.saf_hybrid_attn_fwd(dt, Q, K, V, f.ctypes.data if H else None, a, r, ld, B, H, N, d, O, LSE,
                                   None)


def _bwd(lib, stage=None, dt=1, Q=FAKE, K=FAKE, V=FAKE, O=FAKE, dO=FAKE, LSE=FAKE, flags=(0, 1), a=FAKE,
         r=FAKE, ld=None, B=1, N=8, d=64, dQ=FAKE, dK=FAKE, dV=FAKE, ws=FAKE, ws_bytes=None):
    f = np.asarray(flags, dtype=np.uint8)
    H = f.shape[0]
    ld = N if ld is None else ld
    if ws_bytes is None:
        ws_bytes = lib.saf_hybrid_attn_bwd_workspace_bytes(dt, B, H, N, d)
    args = [dt, Q, K, V, O, dO, LSE, f.ctypes.data, a, r, ld, B, H, N, d, dQ, dK, dV, ws, ws_bytes, None]
    if stage is None:
        return lib.saf_hybrid_attn_bwd(*args)
    return lib.saf_hybrid_attn_bwd_stage(stage, *args)


def test_forward_argument_errors(lib):
    assert _fwd(lib, dt=7) == 3                       # unknown dtype
    assert _fwd(lib, d=32) == 3                       # only d = 64
    assert _fwd(lib, d=128) == 3
    assert _fwd(lib, flags=[0] * 65) == 3             # H > 64
    assert _fwd(lib, N=-1) == 2
    assert _fwd(lib, B=-2) == 2
    assert _fwd(lib, N=(1 << 24) + 1) == 2
    assert _fwd(lib, dt=0, N=(1 << 23) + 1) == 2      # float32 slice would pass 2^31 bytes
    assert _fwd(lib, B=1 << 12, flags=[0] * 64, N=1 << 20) == 2   # grid above 2^31 - 1 workgroups
    assert _fwd(lib, a=None) == 4                     # a fixed head needs a and r
    assert _fwd(lib, r=None) == 4
    assert _fwd(lib, ld=7) == 2                       # prior shorter than N
    assert _fwd(lib, V=None) == 1
    assert _fwd(lib, O=None) == 1
    assert _fwd(lib, LSE=None) == 1
    assert _fwd(lib, Q=None) == 1                     # an ordinary head needs Q and K
    assert _fwd(lib, K=None) == 1
    assert _fwd(lib, V=FAKE + 8) == 6                 # 16-byte alignment
    assert _fwd(lib, LSE=FAKE + 4) == 6
    assert _fwd(lib, flags=(0, 2)) == 7               # flags are 0 or 1
    assert lib.saf_hybrid_attn_fwd(1, FAKE, FAKE, FAKE, None, FAKE, FAKE, 8, 1, 2, 8, 64, FAKE, FAKE, None) == 1


def test_empty_problems_are_no_ops(lib):
    assert _fwd(lib, B=0) == 0
    assert _fwd(lib, N=0, V=None, O=None) == 0
    assert lib.saf_hybrid_attn_fwd(1, None, None, None, None, None, None, 0, 4, 0, 16, 64, None, None, None) == 0


def test_backward_argument_errors(lib):
    for stage in (None, 0, 1, 2, 3):
        assert _bwd(lib, stage, dt=9) == 3
        assert _bwd(lib, stage, d=96) == 3
        assert _bwd(lib, stage, a=None) == 4
        assert _bwd(lib, stage, dO=None) == 1
        assert _bwd(lib, stage, ws=None) == 1
        assert _bwd(lib, stage, ws=FAKE + 16) == 6    # workspace is 256-byte aligned
        assert _bwd(lib, stage, ws_bytes=0) == 2       # workspace too small
        assert _bwd(lib, stage, dK=FAKE + 2) == 6
        assert _bwd(lib, stage, flags=(3, 0)) == 7
        assert _bwd(lib, stage, B=0) == 0
    assert _bwd(lib, 4) == 3                           # unknown stage
    assert _bwd(lib, -1) == 3


def test_workspace_size(lib):
    assert lib.saf_hybrid_attn_bwd_workspace_bytes(1, 8, 12, 4096, 64) == 8 * 12 * 4096 * 4
    assert lib.saf_hybrid_attn_bwd_workspace_bytes(0, 1, 1, 3, 64) == 256
    assert lib.saf_hybrid_attn_bwd_workspace_bytes(1, 1, 1, 1, 32) == 0
    assert lib.saf_hybrid_attn_bwd_workspace_bytes(1, 0, 1, 1, 64) == 0
    assert lib.saf_hybrid_attn_bwd_workspace_bytes(4, 1, 1, 1, 64) == 0


def test_status_strings(lib):
    from paper_2609_34650_amd import binding
    for code in range(8):
        assert binding.status_str(code) and binding.status_str(code) != "unknown status"
    assert binding.status_str(99) == "unknown status"


# ---------------------------------------------------------------------------
# Calibration statistics (include/saf_calib.h)
# ---------------------------------------------------------------------------

def _acc(lib, dt=1, Q=FAKE, K=FAKE, LSE=FAKE, B=2, H=3, T=16, d=64, n_seen=0, mean=FAKE, m2=FAKE, stats=FAKE):
    return lib.saf_calib_accumulate(dt, Q, K, LSE, B, H, T, d, n_seen, mean, m2, stats, None)


def _fin(lib, H=3, T=16, n=4, mean=FAKE, stats=FAKE, ea=FAKE, er=FAKE, sv=FAKE, sk=FAKE, ws=FAKE, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.saf_calib_finalize_workspace_bytes(max(H, 1), max(T, 1))
    return lib.saf_calib_finalize(H, T, n, mean, stats, ea, er, sv, sk, ws, ws_bytes, None)


def test_calib_accumulate_rejects_bad_arguments(lib):
    assert _acc(lib, dt=7) == 3
    assert _acc(lib, d=128) == 3
    assert _acc(lib, H=65) == 3
    assert _acc(lib, B=-1) == 2
    assert _acc(lib, n_seen=-1) == 2
    assert _acc(lib, T=(1 << 16) + 1) == 2
    assert _acc(lib, n_seen=(1 << 24) - 1, B=2) == 2
    assert _acc(lib, Q=None) == 1
    assert _acc(lib, LSE=None) == 1
    assert _acc(lib, stats=None) == 1
    assert _acc(lib, mean=None) == 1
    assert _acc(lib, mean=FAKE + 4) == 6
    assert _acc(lib, m2=FAKE + 4) == 6
    assert _acc(lib, stats=FAKE + 4) == 6
    # Empty problems launch nothing.
    assert _acc(lib, B=0, Q=None, K=None, LSE=None, mean=None, m2=None, stats=None) == 0
    assert _acc(lib, T=0, Q=None, K=None, LSE=None, mean=None, m2=None, stats=None) == 0


def test_calib_finalize_rejects_bad_arguments(lib):
    assert lib.saf_calib_finalize_workspace_bytes(3, 16) % 256 == 0
    assert lib.saf_calib_finalize_workspace_bytes(3, 16) >= 3 * 8
    assert lib.saf_calib_finalize_workspace_bytes(2, 1000) >= 2 * 4 * 4 * 8
    assert lib.saf_calib_stats_bytes(3, 16) >= 3 * 2 * 8
    assert lib.saf_calib_stats_bytes(2, 300) >= 2 * 3 * 3 * 2 * 8
    assert lib.saf_calib_stats_bytes(2, 300) % 256 == 0
    assert lib.saf_calib_stats_bytes(0, 16) == 0
    assert lib.saf_calib_stats_bytes(2, (1 << 16) + 1) == 0
    assert lib.saf_calib_finalize_workspace_bytes(0, 16) == 0
    assert lib.saf_calib_finalize_workspace_bytes(65, 16) == 0
    assert _fin(lib, n=0) == 2
    assert _fin(lib, H=65) == 3
    assert _fin(lib, T=-1) == 2
    assert _fin(lib, mean=None) == 1
    assert _fin(lib, sk=None) == 1
    assert _fin(lib, ws=FAKE + 16) == 6
    assert _fin(lib, ws_bytes=8) == 2
    assert _fin(lib, H=0, mean=None) == 0


# ---------------------------------------------------------------------------
# Trainable-pattern gradients (saf_hybrid_attn_bwd_pattern)
# ---------------------------------------------------------------------------

def _pat(lib, dt=1, V=FAKE, O=FAKE, dO=FAKE, LSE=FAKE, flags=(0, 1), a=FAKE, r=FAKE, ld=None, B=1, N=8, d=64,
         da=FAKE, dr=FAKE, ws=FAKE, ws_bytes=None):
    f = np.asarray(flags, dtype=np.uint8)
    H = f.shape[0]
    ld = N if ld is None else ld
    if ws_bytes is None:
        ws_bytes = lib.saf_hybrid_attn_bwd_pattern_workspace_bytes(dt, max(B, 1), max(H, 1), max(N, 1), 64)
    return lib.saf_hybrid_attn_bwd_pattern(dt, V, O, dO, LSE, f.ctypes.data if H else None, a, r, ld, B, H, N, d,
                                           da, dr, ws, ws_bytes, None)


def test_pattern_gradient_rejects_bad_arguments(lib):
    assert _pat(lib, dt=5) == 3
    assert _pat(lib, d=32) == 3
    assert _pat(lib, flags=(0, 2)) == 7
    assert _pat(lib, a=None) == 4
    assert _pat(lib, ld=4) == 2
    assert _pat(lib, V=None) == 1
    assert _pat(lib, da=None) == 1
    assert _pat(lib, dr=None) == 1
    assert _pat(lib, ws=None) == 1
    assert _pat(lib, O=FAKE + 8) == 6
    assert _pat(lib, ws=FAKE + 64) == 6
    assert _pat(lib, ws_bytes=16) == 2
    # D, da partials, and per key block and chunk of query tiles a row of the
    # offsets it touches (16 tiles of 64 queries + 127).
    need = lib.saf_hybrid_attn_bwd_pattern_workspace_bytes(1, 2, 3, 300, 64)
    assert need >= 2 * 3 * 300 * 4 * 2 + 2 * 3 * 3 * (16 * 64 + 127) * 4 and need % 256 == 0
    assert _pat(lib, ws_bytes=lib.saf_hybrid_attn_bwd_pattern_workspace_bytes(1, 1, 2, 8, 64) - 1) == 2
    assert _pat(lib, B=0, V=None, O=None, dO=None, LSE=None, da=None, dr=None, ws=None) == 0


# ---------------------------------------------------------------------------
# Compact fit (include/saf_fit.h)
# ---------------------------------------------------------------------------

def test_fit_entry_points_reject_bad_arguments(lib):
    import ctypes
    ws_bytes = lib.saf_fit_workspace_bytes(3, 100)
    assert ws_bytes % 256 == 0 and ws_bytes >= 3 * 100 * 4 * 8  # rowsum, moments (4), marginals (2), log Z
    assert lib.saf_fit_workspace_bytes(0, 100) == 0 and lib.saf_fit_workspace_bytes(65, 100) == 0
    assert lib.saf_fit_workspace_bytes(3, (1 << 16) + 1) == 0
    f = ctypes.c_float
    tg = lambda H=3, T=100, mean=FAKE, fl=1e-9, ea=FAKE, er=FAKE, ne=FAKE, ws=FAKE, wb=ws_bytes: \
        lib.saf_fit_targets(H, T, mean, f(fl), ea, er, ne, ws, wb, None)
    assert tg(H=65) == 3
    assert tg(T=-1) == 2
    assert tg(fl=0.0) == 2 and tg(fl=1.5) == 2
    assert tg(mean=None) == 1 and tg(ne=None) == 1
    assert tg(mean=FAKE + 4) == 6 and tg(ne=FAKE + 4) == 6 and tg(ws=FAKE + 64) == 6
    assert tg(wb=ws_bytes - 1) == 2
    assert tg(H=0, mean=None) == 0
    cf = lambda H=3, T=100, ea=FAKE, er=FAKE, ne=FAKE, steps=400, lr=0.05, fl=1e-9, a=FAKE, r=FAKE, lz=None, \
        kl=FAKE, ws=FAKE, wb=ws_bytes: lib.saf_compact_fit(H, T, ea, er, ne, steps, f(lr), f(fl), a, r, lz, kl, ws, wb,
                                                           None)
    assert cf(steps=-1) == 2 and cf(lr=-1.0) == 2 and cf(fl=0.0) == 2
    assert cf(ea=None) == 1 and cf(a=None) == 1 and cf(kl=None) == 1
    assert cf(ne=FAKE + 4) == 6 and cf(ws=FAKE + 8) == 6
    assert cf(wb=16) == 2
    assert cf(T=0, ea=None) == 0


# ---------------------------------------------------------------------------
# Grouped-query forward (saf_hybrid_attn_fwd_gqa)
# ---------------------------------------------------------------------------

def _gqa(lib, dt=1, Q=FAKE, K=FAKE, V=FAKE, flags=(0, 1, 0, 0), a=FAKE, r=FAKE, ld=None, B=1, Hkv=2, N=8, d=128,
         O=FAKE, LSE=FAKE):
    f = np.asarray(flags, dtype=np.uint8)
    Hq = f.shape[0]
    ld = N if ld is None else ld
    return lib.saf_hybrid_attn_fwd_gqa(dt, Q, K, V, f.ctypes.data if Hq else None, a, r, ld, B, Hq, Hkv, N, d, O,
                                       LSE, None)


def test_gqa_forward_rejects_bad_arguments(lib):
    assert _gqa(lib, d=80) == 3
    assert _gqa(lib, dt=9) == 3
    assert _gqa(lib, Hkv=3) == 2          # 4 query heads are not a multiple of 3
    assert _gqa(lib, Hkv=0) == 2
    assert _gqa(lib, flags=(0, 2, 0, 0)) == 7
    assert _gqa(lib, a=None) == 4
    assert _gqa(lib, ld=4) == 2
    assert _gqa(lib, V=None) == 1
    assert _gqa(lib, Q=None) == 1         # an ordinary head needs Q and K
    assert _gqa(lib, Q=None, K=None, flags=(1, 1, 1, 1)) != 1
    assert _gqa(lib, O=FAKE + 2) == 6
    assert _gqa(lib, N=(1 << 23), d=128) == 2   # 2^23 rows x 256 B reaches 2^31
    assert _gqa(lib, flags=[0] * 65, Hkv=5) == 3
    assert _gqa(lib, N=0, Q=None, K=None, V=None, O=None, LSE=None) == 0


# ---------------------------------------------------------------------------
# Grouped-query backward (saf_hybrid_attn_bwd_gqa)
# ---------------------------------------------------------------------------

def test_gqa_backward_workspace_and_rejects(lib):
    wsb = lib.saf_hybrid_attn_bwd_gqa_workspace_bytes
    assert wsb(1, 2, 8, 2, 100, 128) == 6400          # B * Hq * N floats, rounded up to 256 bytes
    assert wsb(0, 1, 4, 4, 33, 96) == 768
    assert wsb(1, 2, 8, 2, 100, 80) == 0 and wsb(1, 2, 8, 3, 100, 64) == 0 and wsb(1, 0, 8, 2, 100, 64) == 0

    def bwd(dt=1, Q=FAKE, K=FAKE, V=FAKE, O=FAKE, dO=FAKE, LSE=FAKE, flags=(0, 1, 0, 0), a=FAKE, r=FAKE, ld=8,
            B=1, Hkv=2, N=8, d=96, dQ=FAKE, dK=FAKE, dV=FAKE, ws=FAKE, wsn=256):
        f = np.asarray(flags, dtype=np.uint8)
        return lib.saf_hybrid_attn_bwd_gqa(dt, Q, K, V, O, dO, LSE, f.ctypes.data, a, r, ld, B, f.shape[0], Hkv, N,
                                           d, dQ, dK, dV, ws, wsn, None)
    assert bwd(d=80) == 3 and bwd(dt=7) == 3
    assert bwd(Hkv=3) == 2 and bwd(ld=4) == 2
    assert bwd(flags=(0, 3, 0, 0)) == 7 and bwd(r=None) == 4
    assert bwd(dQ=None) == 1 and bwd(ws=None) == 1 and bwd(K=None) == 1
    assert bwd(wsn=64) == 2                           # 4 heads x 8 rows x 4 bytes rounds to 256
    assert bwd(ws=FAKE + 16) == 6 and bwd(dV=FAKE + 4) == 6
    assert bwd(N=0, Q=None, K=None, V=None, O=None, dO=None, LSE=None, dQ=None, dK=None, dV=None, ws=None) == 0


def test_measurement_probe_argument_errors(lib):
    # shader-clock probe
    assert lib.saf_clock_probe(None, 100, None) == 1
    assert lib.saf_clock_probe(FAKE, 0, None) == 2
    assert lib.saf_clock_probe(FAKE, 1000001, None) == 2
    assert lib.saf_clock_probe(FAKE + 4, 100, None) == 6
    # known-size read
    assert lib.saf_lds_read_probe(None, 4096, FAKE, None) == 1
    assert lib.saf_lds_read_probe(FAKE, 4096, None, None) == 1
    assert lib.saf_lds_read_probe(FAKE, 0, FAKE, None) == 2
    assert lib.saf_lds_read_probe(FAKE, 4095, FAKE, None) == 2
    assert lib.saf_lds_read_probe(FAKE, 6000, FAKE, None) == 2
    assert lib.saf_lds_read_probe(FAKE, (1 << 40) + 4096, FAKE, None) == 2
    assert lib.saf_lds_read_probe(FAKE + 8, 4096, FAKE, None) == 6
    assert lib.saf_lds_read_probe(FAKE, 4096, FAKE + 2, None) == 6
    # LDS read patterns
    assert lib.saf_lds_pattern_probe(0, 10, None, None) == 1
    assert lib.saf_lds_pattern_probe(-1, 10, FAKE, None) == 2
    assert lib.saf_lds_pattern_probe(7, 10, FAKE, None) == 2
    assert lib.saf_lds_pattern_probe(0, 0, FAKE, None) == 2
    assert lib.saf_lds_pattern_probe(0, (1 << 20) + 1, FAKE, None) == 2
    assert lib.saf_lds_pattern_probe(0, 10, FAKE + 2, None) == 6
    # MFMA rate
    assert lib.saf_mfma_rate_probe(0, 1, 10, None, FAKE, None) == 1
    assert lib.saf_mfma_rate_probe(0, 1, 10, FAKE, None, None) == 1
    assert lib.saf_mfma_rate_probe(2, 1, 10, FAKE, FAKE, None) == 2
    assert lib.saf_mfma_rate_probe(0, 3, 10, FAKE, FAKE, None) == 2
    assert lib.saf_mfma_rate_probe(0, 0, 10, FAKE, FAKE, None) == 2
    assert lib.saf_mfma_rate_probe(1, 2, 0, FAKE, FAKE, None) == 2
    assert lib.saf_mfma_rate_probe(0, 1, 10, FAKE + 4, FAKE, None) == 6
    assert lib.saf_mfma_rate_probe(0, 1, 10, FAKE, FAKE + 2, None) == 6
