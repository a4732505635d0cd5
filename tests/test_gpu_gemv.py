"""Batched GEMV (the fused kernel of Alg. 2) against the oracle, through the
C ABI: Y = A X is the oracle's emulated product under the fixed scaling
(Alg. 1's mu = k max|A~| max|X~|), bit for bit on every entry whose row of A
and column of X are not flagged; flagged entries lie within the FP64
dot-product bound.  Shapes cover ragged row blocks (m not a multiple of 64),
ragged k chunks (k not a multiple of 128), 1..16 right-hand sides, k above
32768 (several exact k-splits) and the moduli range."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import bits, compare_C, device, fallback_ok

pytestmark = pytest.mark.gpu


def _gemv(A, X, r, flags=0):
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    m, k = A.shape
    nrhs = X.shape[1]
    Ad, Xd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(X, dev)
    Yd = oz.to_device_colmajor(np.full((m, nrhs), np.nan), dev)
    oz.gemv(Ad, Xd, num_moduli=r, flags=flags, Y=Yd)
    torch.cuda.synchronize()
    return oz.from_device_colmajor(Yd)


@pytest.mark.parametrize("m,k,nrhs,r", [(1, 1, 1, 12), (64, 128, 8, 12), (200, 300, 5, 13),
                                        (777, 4096, 8, 13), (130, 1000, 16, 16), (96, 250, 4, 8),
                                        (333, 70000, 3, 12), (1500, 129, 7, 15), (70, 5, 2, 11)])
def test_gemv_matches_oracle(m, k, nrhs, r):
    A, X = synth.lognormal(m, nrhs, k, seed=m + k + nrhs)
    Y = _gemv(A, X, r)
    res = oracle.dgemm(A, X, r, mode="fixed")
    assert len(res.fallback_rows) == 0 and len(res.fallback_cols) == 0
    assert np.array_equal(bits(Y), bits(res.C))


def test_gemv_fallback_rows_and_columns():
    A, X = synth.uniform(300, 6, 500, seed=9)
    A, X = A.copy(), X.copy()
    A[3, 7] = np.nan                      # T1 row
    A[100, 5] = np.inf
    A[50, ::2] *= 1e200                   # T2 row (intra-row span ~2^664)
    X[11, 4] = -np.inf                    # T1 column
    X[::3, 2] *= 1e-250                   # T2 column
    A[7] = 0.0                            # zero row: exact +0.0
    res = oracle.dgemm(A, X, 12, mode="fixed")
    assert set(res.fallback_rows) == {3, 50, 100} and set(res.fallback_cols) == {2, 4}
    Y = _gemv(A, X, 12)
    compare_C(Y, A, X, res)
    ok = [j for j in range(6) if j not in (2, 4)]   # columns 2, 4 are native (0 * -inf = NaN)
    assert not np.any(np.signbit(Y[7, ok])) and np.all(Y[7, ok] == 0)


@pytest.mark.parametrize("flags,quant,fb,force", [(4, "tz", True, False), (8, "rn", False, False),
                                                   (16, "rn", True, True)])
def test_gemv_flags(flags, quant, fb, force):
    A, X = synth.lognormal(150, 5, 400, seed=17)
    A = A.copy()
    A[9, ::2] *= 1e200
    res = oracle.dgemm(A, X, 12, mode="fixed", quant=quant, fallback=fb, force_fallback=force)
    Y = _gemv(A, X, 12, flags=flags)
    if fb:
        compare_C(Y, A, X, res)
    else:
        assert np.array_equal(bits(Y), bits(res.C))


def test_gemv_k0_and_empty():
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    Ad = oz.colmajor_empty(5, 0, device=dev)
    Xd = oz.colmajor_empty(0, 3, device=dev)
    Yd = oz.to_device_colmajor(np.full((5, 3), 7.0), dev)
    oz.ozaki2_gemv_batched(5, 0, 3, Ad, 5, Xd, 1, Yd, 5, 12, 0, None, 0)
    torch.cuda.synchronize()
    assert np.all(oz.from_device_colmajor(Yd) == 0.0)


def test_gemv_full_size_sampled():
    """The bench workload (16384 x 16384 times 8 columns, lognormal entries,
    r = 13): sampled rows bit-exact, componentwise error within 1e-15."""
    from oracle import refgemm
    import paper_2606_06510_amd as oz
    import torch
    A, X = synth.lognormal(16384, 8, 16384, seed=6)
    dev = device()
    Ad, Xd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(X, dev)
    Yd = oz.gemv(Ad, Xd, num_moduli=13)
    torch.cuda.synchronize()
    rng = np.random.default_rng(6)
    rows = np.sort(np.concatenate([rng.choice(16384, 60, replace=False), [0, 16383]]))
    Y = Yd.index_select(0, torch.as_tensor(rows, device=dev)).cpu().numpy()
    res = oracle.dgemm(A, X, 13, rows=rows, mode="fixed")
    assert np.array_equal(bits(Y), bits(res.C))
    rr, cc = np.meshgrid(rows, np.arange(8), indexing="ij")
    assert refgemm.componentwise_ratio(Y.ravel(), A, X, rr.ravel(), cc.ravel()) <= 1e-15
    del Ad, Xd, Yd
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("m,n,k,r", [(300, 8, 500, 12), (1000, 16, 3000, 13), (129, 1, 70, 8),
                                     (257, 17, 300, 12)])
@pytest.mark.parametrize("fallback", [False, True])
def test_fixed_scale_skinny_route_matches_staged(m, n, k, r, fallback):
    """ozaki2_dgemm_ex with OZ2_SCALE_FIXED and n <= 16 runs the fused GEMV
    kernel; its C equals the staged fixed-scale plan's bit for bit (and the
    oracle's on unflagged entries).  n = 17 takes the staged path itself."""
    import paper_2606_06510_amd as oz
    import torch
    from tests.gpu_util import run_staged
    A, B = synth.lognormal(m, n, k, seed=m + 3 * n + k)
    if fallback:
        A[min(5, m - 1), k // 2] = np.nan           # a T1 row of A
        B[k // 3, n - 1] *= 1e300                    # a huge entry: T2 in its column's span
    dev = device()
    Ad, Bd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(B, dev)
    Cd = oz.to_device_colmajor(np.full((m, n), np.nan), dev)
    oz.matmul(Ad, Bd, r, flags=oz.OZ2_SCALE_FIXED, C=Cd)
    torch.cuda.synchronize()
    got = oz.from_device_colmajor(Cd)
    _, staged = run_staged(A, B, r, oz.OZ2_SCALE_FIXED)
    assert np.array_equal(bits(got), bits(staged))
    res = oracle.dgemm(A, B, r, mode="fixed")
    emu = ~np.isin(np.arange(m), res.fallback_rows)[:, None] & \
        ~np.isin(np.arange(n), res.fallback_cols)[None, :]
    assert np.array_equal(bits(got[emu]), bits(res.C[emu]))
    assert fallback == (not emu.all())


@pytest.mark.parametrize("m,k,n1,n2,r", [(300, 500, 8, 3, 12), (1000, 40000, 16, 16, 13)])
def test_reuse_a_scales_matches_full_call(m, k, n1, n2, r):
    """OZ2_REUSE_A_SCALES: a second call on the same A (a T1 row and a T2
    row in it) with a new X skips A's scan and gives exactly the full call's
    Y, flagged rows included."""
    import paper_2606_06510_amd as oz
    import torch
    A, X1 = synth.lognormal(m, n1, k, seed=m + k)
    A[3, k // 2] = np.inf                                # T1 row
    A[7, 1] *= 1e280                                     # T2 row (the rest quantises to 0)
    X2 = synth.lognormal(m, n2, k, seed=m + k + 1)[1]
    dev = device()
    Ad = oz.to_device_colmajor(A, dev)
    ws = torch.empty(oz.ozaki2_gemv_workspace_bytes(m, k, 16, r), dtype=torch.uint8, device=dev)
    Y1 = oz.gemv(Ad, oz.to_device_colmajor(X1, dev), num_moduli=r, workspace=ws)
    X2d = oz.to_device_colmajor(X2, dev)
    Y2 = oz.gemv(Ad, X2d, num_moduli=r, flags=oz.OZ2_REUSE_A_SCALES, workspace=ws)
    Y2ref = oz.gemv(Ad, X2d, num_moduli=r)                # fresh workspace, full call
    torch.cuda.synchronize()
    y2, y2ref = oz.from_device_colmajor(Y2), oz.from_device_colmajor(Y2ref)
    assert np.array_equal(bits(y2), bits(y2ref))
    res = oracle.dgemm(A, X2, r, mode="fixed")
    assert {3, 7} <= set(res.fallback_rows.tolist())
    emu = ~np.isin(np.arange(m), res.fallback_rows)
    assert np.array_equal(bits(y2[emu]), bits(res.C[emu]))
    del Y1
