"""The C-ABI library: it loads without a GPU, exports every entry point
include/ozaki2.h declares, and rejects invalid arguments before touching the
device (no compute calls here)."""
import os
import re

import pytest

import paper_2606_06510_amd as oz
from paper_2606_06510_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header):
    src = open(os.path.join(ROOT, "include", header)).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ozaki2_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = oz.load()
    names = _declared("ozaki2.h")
    assert len(names) == 19
    for n in names:
        assert hasattr(L, n), n
    assert sorted(_lib.EXPORTS) == names
    probes = _declared("ozaki2_probes.h")
    assert len(probes) == 8
    for n in probes:
        assert hasattr(L, n), n
    assert sorted(_lib.PROBE_EXPORTS) == probes
    headers = sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))
    assert headers == ["ozaki2.h", "ozaki2_probes.h"]


def test_probe_argument_checks():
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_e4m3(0, 0, -1, 0)
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_accum(0, 0, 1, 0, 0)          # null pointers
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_copy(16, 32, 15, 0)           # size not a multiple of 16
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_mfma_peak(0)
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_mfma_digits(3)                # odd iteration count
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_copy_peak(1 << 20, 1)         # below 16 MiB
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_crt(12, FAKE, FAKE, -1, FAKE, FAKE, 0)     # n < 0
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_crt(7, FAKE, FAKE, 4, FAKE, FAKE, 0)       # r outside [8, 16]
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_probe_crt(12, FAKE, None, 4, FAKE, FAKE, 0)      # null pointer
    for bad in [dict(m=65), dict(k=0), dict(lda=3), dict(batch=-1), dict(r=17), dict(W=None)]:
        a = dict(m=4, n=4, k=4, lda=4, ldb=4, batch=2, r=12, W=FAKE)
        a.update(bad)
        with pytest.raises(oz.Ozaki2Error):
            oz.ozaki2_probe_batched_integers(a["m"], a["n"], a["k"], FAKE, a["lda"], 16, FAKE,
                                             a["ldb"], 16, a["batch"], a["r"], a["W"], 0)


def test_status_strings():
    assert oz.ozaki2_status_string(0) == "ok"
    assert "workspace" in oz.ozaki2_status_string(-5)


def test_moduli_table():
    assert oz.ozaki2_moduli(12) == [487, 491, 499, 503, 509, 511, 529, 625, 841, 961, 1024, 1089]
    assert oz.ozaki2_moduli(16)[:4] == [463, 467, 479, 481]
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_moduli(7)
    with pytest.raises(oz.Ozaki2Error):
        oz.ozaki2_moduli(17)


def test_workspace_bytes():
    # planes 30 B per padded element of A and B, residues 12 bits per padded
    # output and modulus (18 B at r = 12)
    b = oz.ozaki2_workspace_bytes(4096, 4096, 4096, 12)
    assert b >= 30 * 2 * 4096 * 4096 + 18 * 4096 * 4096
    assert b < 1.05 * (31 * 2 * 4096 * 4096 + 18 * 4096 * 4096) + (1 << 20)
    # the fused route keeps no residues (nor a fallback panel: compared
    # without one): 1.5 r B per padded output less
    mp = np_ = 512
    nf = oz.OZ2_NO_FALLBACK
    assert oz.ozaki2_workspace_bytes(300, 400, 500, 12, nf) - \
        oz.ozaki2_workspace_bytes(300, 400, 500, 12, nf | oz.OZ2_FUSED) in \
        range(18 * mp * np_, 18 * mp * np_ + 256 * 4)
    # the native fallback's panel of gathered rows: min(mp, 1024) x k doubles,
    # absent with OZ2_NO_FALLBACK
    for m, k in [(4096, 4096), (300, 200), (32768, 256)]:
        mp = (m + 255) // 256 * 256
        diff = oz.ozaki2_workspace_bytes(m, 512, k, 12) - \
            oz.ozaki2_workspace_bytes(m, 512, k, 12, oz.OZ2_NO_FALLBACK)
        panel = min(mp, 1024) * k * 8
        assert panel <= diff < panel + 256, (m, k, diff, panel)
    assert oz.ozaki2_workspace_bytes(10, 10, 10, 7) == 0
    assert oz.ozaki2_workspace_bytes(10, 10, 10, 12, 1 << 10) == 0
    assert oz.ozaki2_workspace_bytes(-1, 10, 10, 12) == 0


FAKE = 1 << 40      # never dereferenced: validation rejects before any launch


@pytest.mark.parametrize("args", [
    dict(m=-1), dict(n=-1), dict(k=-1), dict(lda=3), dict(ldb=4), dict(ldc=3), dict(r=7),
    dict(r=17), dict(A=0), dict(B=0), dict(C=0), dict(flags=1 << 8),
])
def test_invalid_arguments_rejected(args):
    p = dict(m=4, n=5, k=6, A=FAKE, lda=4, B=FAKE + (1 << 20), ldb=6, C=FAKE + (2 << 20), ldc=4,
             r=12, flags=0)
    p.update(args)
    L = oz.load()
    st = L.ozaki2_dgemm_ex(p["m"], p["n"], p["k"], p["A"] or None, p["lda"], p["B"] or None,
                           p["ldb"], p["C"] or None, p["ldc"], p["r"], p["flags"], FAKE + (3 << 20),
                           1 << 30, None)
    assert st == _lib.OZ2_E_INVALID


def test_overlapping_output_rejected():
    L = oz.load()
    st = L.ozaki2_dgemm_ex(4, 5, 6, FAKE, 4, FAKE + (1 << 20), 6, FAKE + 8, 4, 12, 0,
                           FAKE + (3 << 20), 1 << 30, None)
    assert st == _lib.OZ2_E_INVALID


def test_zero_sized_output_is_a_noop():
    L = oz.load()
    assert L.ozaki2_dgemm_ex(0, 5, 6, None, 1, None, 6, None, 1, 12, 0, None, 0, None) == 0
    assert L.ozaki2_dgemm(4, 0, 6, None, 4, None, 6, None, 4, 12, None) == 0


def test_skinny_route_workspace_serves_both_routes():
    """With OZ2_SCALE_FIXED and n <= 16 ozaki2_dgemm_ex takes the fused GEMV;
    the workspace size covers that route and a plan of the same shape."""
    f = oz.OZ2_SCALE_FIXED
    for m, n, k in [(300, 8, 500), (5000, 16, 20000), (64, 1, 1)]:
        both = oz.ozaki2_workspace_bytes(m, n, k, 12, f)
        assert both == max(oz.ozaki2_gemv_workspace_bytes(m, k, n, 12),
                           oz.ozaki2_workspace_bytes(m, n, k, 12, f | oz.OZ2_KEEP_RESIDUES))
    # n = 17, or accumulation: the staged path alone
    assert oz.ozaki2_workspace_bytes(300, 17, 500, 12, f) == \
        oz.ozaki2_workspace_bytes(300, 17, 500, 12, f | oz.OZ2_KEEP_RESIDUES)
    assert oz.ozaki2_workspace_bytes(300, 8, 500, 12, f | oz.OZ2_ACCUMULATE) == \
        oz.ozaki2_workspace_bytes(300, 8, 500, 12, f | oz.OZ2_KEEP_RESIDUES)


def test_stage_timing_flag_is_for_plans_only():
    L = oz.load()
    st = L.ozaki2_dgemm_ex(4, 5, 6, FAKE, 4, FAKE + (1 << 20), 6, FAKE + (2 << 20), 4, 12,
                           oz.OZ2_TIME_STAGES, FAKE + (3 << 20), 1 << 30, None)
    assert st == _lib.OZ2_E_INVALID
    # a known flag (KEEP_RESIDUES) leaves the workspace size as it is: the
    # staged route always materialises the residues
    assert oz.ozaki2_workspace_bytes(300, 200, 100, 12, oz.OZ2_KEEP_RESIDUES) == \
        oz.ozaki2_workspace_bytes(300, 200, 100, 12)


def test_plan_create_validation():
    L = oz.load()
    import ctypes
    h = ctypes.c_void_p()
    need = oz.ozaki2_workspace_bytes(8, 8, 8, 12)
    assert L.ozaki2_plan_create(ctypes.byref(h), 8, 8, 8, 12, 0, None, need) == _lib.OZ2_E_WORKSPACE
    assert L.ozaki2_plan_create(ctypes.byref(h), 8, 8, 8, 12, 0, FAKE, need - 1) == _lib.OZ2_E_WORKSPACE
    assert L.ozaki2_plan_create(ctypes.byref(h), 8, 8, 8, 12, 0, FAKE + 8, need) == _lib.OZ2_E_WORKSPACE
    assert L.ozaki2_plan_create(ctypes.byref(h), 8, 8, 8, 5, 0, FAKE, need) == _lib.OZ2_E_INVALID
    assert L.ozaki2_residue_gemm(None, None) == _lib.OZ2_E_INVALID
    assert L.ozaki2_reconstruct(None, FAKE, 8, None) == _lib.OZ2_E_INVALID


def test_static_entry_point_validation():
    """ozaki2_dgemm_static checks its arguments, and refuses a product whose
    workspace exceeds its static array, before touching the device."""
    L = oz.load()
    assert L.ozaki2_dgemm_static(4, 5, 6, FAKE, 3, FAKE + (1 << 20), 6, FAKE + (2 << 20), 4, 12,
                                 None) == _lib.OZ2_E_INVALID
    assert L.ozaki2_dgemm_static(4, 5, 6, FAKE, 4, FAKE + (1 << 20), 6, FAKE + (2 << 20), 4, 7,
                                 None) == _lib.OZ2_E_INVALID
    n = 1024
    assert oz.ozaki2_workspace_bytes(n, n, n, 12) > oz.OZ2_STATIC_SCRATCH_BYTES
    assert L.ozaki2_dgemm_static(n, n, n, FAKE, n, FAKE + (1 << 30), n, FAKE + (2 << 30), n, 12,
                                 None) == _lib.OZ2_E_WORKSPACE
    assert L.ozaki2_dgemm_static(0, 5, 6, None, 1, None, 6, None, 1, 12, None) == 0


@pytest.mark.parametrize("args", [
    dict(m=-1), dict(k=-1), dict(nrhs=17), dict(nrhs=-1), dict(lda=3), dict(ldx=5), dict(ldy=3),
    dict(r=7), dict(r=17), dict(A=0), dict(X=0), dict(Y=0), dict(flags=oz.OZ2_ACCUMULATE),
    dict(flags=oz.OZ2_SCALE_FIXED), dict(flags=1 << 9),
])
def test_gemv_invalid_arguments_rejected(args):
    p = dict(m=4, k=6, nrhs=3, A=FAKE, lda=4, X=FAKE + (1 << 20), ldx=6, Y=FAKE + (2 << 20), ldy=4,
             r=12, flags=0)
    p.update(args)
    L = oz.load()
    st = L.ozaki2_gemv_batched(p["m"], p["k"], p["nrhs"], p["A"] or None, p["lda"],
                               p["X"] or None, p["ldx"], p["Y"] or None, p["ldy"], p["r"],
                               p["flags"], FAKE + (3 << 20), 1 << 30, None)
    assert st == _lib.OZ2_E_INVALID


def test_gemv_workspace_bytes():
    # X's operand fragments (P planes x 2 KiB per 128 k) and the partial
    # residues (splits x r x rows padded to 64 x 16 x 2 bytes) dominate
    for m, k, nrhs, r in [(16384, 16384, 8, 13), (100, 70000, 3, 12), (1, 1, 1, 8)]:
        b = oz.ozaki2_gemv_workspace_bytes(m, k, nrhs, r)
        P = sum(2 if int(round(x ** 0.5)) ** 2 == x else 3 for x in oz.ozaki2_moduli(r))
        chunks = (k + 127) // 128
        assert b >= chunks * P * 2048 + r * ((m + 63) // 64 * 64) * 32, (m, k, b)
    assert oz.ozaki2_gemv_workspace_bytes(10, 10, 17, 12) == 0
    assert oz.ozaki2_gemv_workspace_bytes(10, 10, 4, 7) == 0
    L = oz.load()
    assert L.ozaki2_gemv_batched(0, 5, 3, None, 1, None, 5, None, 1, 12, 0, None, 0, None) == 0
    assert L.ozaki2_gemv_batched(4, 5, 3, FAKE, 4, FAKE + (1 << 20), 5, FAKE + (2 << 20), 4, 12, 0,
                                 None, 0, None) == _lib.OZ2_E_WORKSPACE
