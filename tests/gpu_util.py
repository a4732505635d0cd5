"""Helpers shared by the GPU tests: device transfer, running the staged API,
and the comparisons against the oracle."""
import numpy as np

import oracle
from oracle import e4m3, ozaki2 as oz2o


def device():
    import torch
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    return torch.device("cuda:0")


def run_staged(A, B, r=12, flags=0, C_in=None):
    """Run the three stages through the C ABI; returns (plan, C numpy)."""
    import paper_2606_06510_amd as oz
    dev = device()
    m, k = A.shape
    n = B.shape[1]
    Ad = oz.to_device_colmajor(A, dev)
    Bd = oz.to_device_colmajor(B, dev)
    Cd = oz.to_device_colmajor(C_in if C_in is not None else np.full((m, n), np.nan), dev)
    plan = oz.Plan(m, n, k, r, flags, device=dev)
    plan.deconstruct(Ad, Bd)
    plan.residue_gemm()
    plan.reconstruct(Cd)
    import torch
    torch.cuda.synchronize()
    plan._keep = (Ad, Bd, Cd)
    return plan, oz.from_device_colmajor(Cd)


def bits(x):
    return np.ascontiguousarray(x, dtype=np.float64).view(np.uint64)


def expected_bytes(vals):
    enc = np.vectorize(e4m3.encode_int, otypes=[np.uint8])
    return enc(np.asarray(vals, dtype=np.int64))


def fallback_ok(C, A, B, i, j, C_in=None):
    """A fallback entry: native FP64 within the dot-product error bound, or the
    same IEEE class (NaN / signed Inf) as the oracle's reference.  With C_in
    (C += A B) the entry is fl(C_in + native dot): one more rounding."""
    ref = oz2o.native_dot(A[i], B[:, j])
    got = C[i, j]
    cin = 0.0 if C_in is None else float(C_in[i, j])
    if np.isnan(ref):
        return np.isnan(got)
    if np.isinf(ref):
        return got == ref
    k = A.shape[1]
    den = float(np.abs(A[i]) @ np.abs(B[:, j]))
    return abs(got - (cin + ref)) <= (1.01 * (k + 1) * 2.0 ** -53 * den + k * 2.0 ** -1074
                                      + 2.0 ** -53 * abs(got))


def compare_all(plan, C, A, B, r, res, check_integers=True):
    """Stage-by-stage parity of a full (small) run against oracle Result res."""
    import paper_2606_06510_amd as oz
    m, k = A.shape
    n = B.shape[1]
    EA, EB = plan.query(oz.OZ2_Q_EXPONENTS)
    assert np.array_equal(EA, res.EA) and np.array_equal(EB, res.EB)
    fA, fB = plan.query(oz.OZ2_Q_FLAGS)
    assert np.array_equal((fA & 1) != 0, res.t1A) and np.array_equal((fB & 1) != 0, res.t1B)
    assert np.array_equal((fA & 2) != 0, res.t2A) and np.array_equal((fB & 2) != 0, res.t2B)
    if not (plan.flags & oz.OZ2_SCALE_FIXED):
        R, K = plan.query(oz.OZ2_Q_MAXIMA)
        okA, okB = ~res.t1A, ~res.t1B
        assert np.array_equal(R[okA], res.R[okA]) and np.array_equal(K[okB], res.K[okB])
        cA, cB = plan.query(oz.OZ2_Q_CODES)
        assert np.array_equal(cA, expected_bytes(oz2o.magnitude_codes(A, res.EA, res.t1A)))
        assert np.array_equal(cB, expected_bytes(oz2o.magnitude_codes(B.T, res.EB, res.t1B)))
    sA, tB = plan.query(oz.OZ2_Q_SCALES)
    assert np.array_equal(sA, res.sA) and np.array_equal(tB, res.tB)
    PA, PB = plan.query(oz.OZ2_Q_PLANES)
    Aq, Bq = res.extras["Aq"], res.extras["Bq"]
    pi = 0
    for mi in res.ms:
        pa = oz2o.planes_of(Aq, mi)
        pb = oz2o.planes_of(Bq.T, mi)
        for t in range(len(pa)):
            assert np.array_equal(PA[pi + t], expected_bytes(pa[t])), (mi, t, "A")
            assert np.array_equal(PB[pi + t], expected_bytes(pb[t])), (mi, t, "B")
        pi += len(pa)
    # the residue GEMMs leave a representative of each residue (not unique):
    # congruent to the oracle's centred residue, of magnitude <= m/2 + 32
    Rg = plan.query(oz.OZ2_Q_RESIDUES).astype(np.int64)
    for t, mi in enumerate(res.ms):
        assert np.all((Rg[t] - res.residues[t]) % mi == 0), ("residue", mi)
        assert np.all(np.abs(Rg[t]) <= mi // 2 + 32), ("representative range", mi)
    if check_integers:
        # the integers formed by the reconstruction's own routine (unique)
        X = plan.query(oz.OZ2_Q_INTEGERS)
        assert all(int(a) == int(b) for a, b in zip(X.ravel(), res.X.ravel()))
    compare_C(C, A, B, res)


def compare_C(C, A, B, res, C_in=None):
    fr = np.isin(res.rows, res.fallback_rows)
    fc = np.isin(res.cols, res.fallback_cols)
    emu = ~fr[:, None] & ~fc[None, :]
    assert np.array_equal(bits(C)[emu], bits(res.C)[emu]), "emulated entries differ"
    for ii, jj in zip(*np.nonzero(~emu)):
        assert fallback_ok(C, A, B, res.rows[ii], res.cols[jj], C_in), (ii, jj)
