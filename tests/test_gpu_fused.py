"""The fused residue-GEMM + reconstruction kernel (OZ2_FUSED: every output's
residues stay on chip, packed in registers and LDS, and the CRT runs in the
kernel's epilogue) against the oracle, through the C ABI: emulated entries
bit for bit, flagged entries within the FP64 dot-product bound.  Covers
ragged 128 x 128 tiles, k from 1 to one full slab, r = 8..12, accumulation,
the fallback flags, results in the subnormal and overflow ranges, and the
fused route of ozaki2_dgemm_ex in its smaller workspace."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import bits, compare_C, device

pytestmark = pytest.mark.gpu


def _fused_plan(A, B, r, flags=0, C_in=None):
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    m, k = A.shape
    n = B.shape[1]
    Ad, Bd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(B, dev)
    Cd = oz.to_device_colmajor(C_in if C_in is not None else np.full((m, n), np.nan), dev)
    plan = oz.Plan(m, n, k, r, flags | oz.OZ2_FUSED, device=dev)
    plan.deconstruct(Ad, Bd)
    plan.residue_gemm()
    plan.reconstruct(Cd)
    torch.cuda.synchronize()
    plan._keep = (Ad, Bd, Cd)
    return plan, oz.from_device_colmajor(Cd)


@pytest.mark.parametrize("m,n,k,r", [(1, 1, 1, 12), (128, 128, 64, 12), (300, 520, 256, 12),
                                     (129, 255, 100, 11), (513, 129, 1000, 10), (700, 300, 1024, 9),
                                     (256, 384, 2048, 12), (64, 700, 5, 8), (200, 136, 300, 12)])
def test_fused_matches_oracle(m, n, k, r):
    A, B = synth.lognormal(m, n, k, seed=m + 2 * n + k)
    res = oracle.dgemm(A, B, r)
    plan, C = _fused_plan(A, B, r)
    compare_C(C, A, B, res)
    import paper_2606_06510_amd as oz
    with pytest.raises(oz.Ozaki2Error):          # never materialised
        plan.query(oz.OZ2_Q_RESIDUES)


def test_fused_full_slab():
    """k = 32768, the longest exact FP32 slab the fused kernel takes."""
    A, B = synth.uniform(96, 80, 32768, seed=13)
    res = oracle.dgemm(A, B, 12)
    plan, C = _fused_plan(A, B, 12)
    compare_C(C, A, B, res)


def test_fused_accumulate_and_fallback():
    A, B, Cin = synth.rankk(300, 260, 256, seed=44)
    A, B = A.copy(), B.copy()
    A[3, 7] = np.nan
    A[50, ::2] *= 1e200
    B[::3, 20] *= 1e-250
    res = oracle.dgemm(A, B, 12, C_in=Cin)
    assert set(res.fallback_rows) == {3, 50} and set(res.fallback_cols) == {20}
    plan, C = _fused_plan(A, B, 12, flags=1, C_in=Cin)
    compare_C(C, A, B, res, C_in=Cin)


@pytest.mark.parametrize("flags,fb,force", [(8, False, False), (16, True, True)])
def test_fused_fallback_flags(flags, fb, force):
    A, B = synth.uniform(150, 140, 120, seed=5)
    A = A.copy()
    A[2, ::2] *= 1e200
    res = oracle.dgemm(A, B, 12, fallback=fb, force_fallback=force)
    plan, C = _fused_plan(A, B, 12, flags=flags)
    if fb:
        compare_C(C, A, B, res)
    else:
        assert np.array_equal(bits(C), bits(res.C))


def test_fused_subnormal_and_overflowing_results():
    m, n, k = 96, 80, 200
    A, B = synth.lognormal(m, n, k, seed=321)
    A, B = A.copy(), B.copy()
    A[:32] *= 2.0 ** -560
    A[64:] *= 2.0 ** 520
    B[:, :24] *= 2.0 ** -500
    B[:, 56:] *= 2.0 ** 520
    res = oracle.dgemm(A, B, 12)
    assert ((res.C != 0) & (np.abs(res.C) < 2.0 ** -1022)).sum() == 32 * 24
    plan, C = _fused_plan(A, B, 12)
    assert np.array_equal(bits(C), bits(res.C))


def test_fused_workspace_and_keep_residues():
    """ozaki2_dgemm_ex with OZ2_FUSED runs in the smaller workspace that holds
    no residues; the staged route (the default, or OZ2_KEEP_RESIDUES) needs
    them; both bit-exact, and OZ2_FUSED with OZ2_KEEP_RESIDUES is refused."""
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    A, B = synth.lognormal(260, 300, 500, seed=71)
    res = oracle.dgemm(A, B, 12)
    Ad, Bd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(B, dev)
    small = oz.ozaki2_workspace_bytes(260, 300, 500, 12, oz.OZ2_FUSED)
    assert small < oz.ozaki2_workspace_bytes(260, 300, 500, 12)
    ws = torch.empty(small, dtype=torch.uint8, device=dev)
    C1 = oz.matmul(Ad, Bd, 12, flags=oz.OZ2_FUSED, workspace=ws)
    C2 = oz.matmul(Ad, Bd, 12, flags=oz.OZ2_KEEP_RESIDUES)
    torch.cuda.synchronize()
    assert np.array_equal(bits(oz.from_device_colmajor(C1)), bits(res.C))
    assert np.array_equal(bits(oz.from_device_colmajor(C2)), bits(res.C))
    with pytest.raises(oz.Ozaki2Error):             # the staged route needs the residues
        oz.matmul(Ad, Bd, 12, workspace=ws)
    with pytest.raises(oz.Ozaki2Error):
        oz.matmul(Ad, Bd, 12, flags=oz.OZ2_FUSED | oz.OZ2_KEEP_RESIDUES)


def test_fused_refused_beyond_its_range():
    import paper_2606_06510_amd as oz
    dev = device()
    with pytest.raises(oz.Ozaki2Error):             # r = 13: five words of residues
        oz.Plan(100, 100, 100, 13, oz.OZ2_FUSED, device=dev)
    with pytest.raises(oz.Ozaki2Error):             # k beyond one exact slab
        oz.Plan(64, 64, 40000, 12, oz.OZ2_FUSED, device=dev)
