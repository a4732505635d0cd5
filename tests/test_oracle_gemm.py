"""End-to-end pins of the oracle GEMM: brute-force integer products, the
plane route, the closed-form quantisation bound, textbook special cases and
the accuracy target against independent references."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from oracle import moduli, ozaki2, planes, refgemm


def _rand_tiny(rng, m, n, k, kind):
    if kind == "uniform":
        return rng.uniform(-1, 1, (m, k)), rng.uniform(-1, 1, (k, n))
    if kind == "wide":
        A = (rng.random((m, k)) - 0.5) * np.exp(4.0 * rng.standard_normal((m, k)))
        B = (rng.random((k, n)) - 0.5) * np.exp(4.0 * rng.standard_normal((k, n)))
        return A, B
    if kind == "adversarial":       # row/column maxima with all-equal codes
        A = np.where(rng.random((m, k)) < 0.5, 1.0, -1.0) * (1 - 2.0 ** -53)
        B = np.where(rng.random((k, n)) < 0.5, 1.0, -1.0) * (1 - 2.0 ** -53)
        return A, B
    if kind == "sparse":
        A = rng.uniform(-1, 1, (m, k)) * (rng.random((m, k)) < 0.3)
        B = rng.uniform(-1, 1, (k, n)) * (rng.random((k, n)) < 0.3)
        return A, B
    raise KeyError(kind)


@pytest.mark.parametrize("r", [8, 12, 16])
@pytest.mark.parametrize("kind", ["uniform", "wide", "adversarial", "sparse"])
@pytest.mark.parametrize("mode", ["bound", "fixed"])
def test_integer_core_brute_force(r, kind, mode):
    """The CRT integer equals the Python-int product A~ B~ exactly."""
    rng = np.random.default_rng(hash((r, kind, mode)) % 2 ** 32)
    for (m, n, k) in [(1, 1, 1), (3, 5, 7), (8, 8, 8), (2, 7, 1)]:
        A, B = _rand_tiny(rng, m, n, k, kind)
        res = oracle.dgemm(A, B, r, mode=mode)
        Aq, Bq = res.extras["Aq"], res.extras["Bq"]
        for i in range(m):
            for j in range(n):
                exact = sum(int(Aq[i, l]) * int(Bq[l, j]) for l in range(k))
                assert int(res.X[i, j]) == exact
                ms = res.ms
                for t, mt in enumerate(ms):
                    v = exact % mt
                    v = v - mt if v >= (mt + 1) // 2 else v
                    assert res.residues[t, i, j] == v


@pytest.mark.parametrize("r", [8, 12, 15])
def test_plane_route_matches_direct_route(r):
    """Residues via FP8 planes (three products per modulus, exact integer
    accumulation, epilogue coefficients, final reduction) equal the direct
    modular GEMM."""
    rng = np.random.default_rng(r)
    A, B = _rand_tiny(rng, 9, 6, 40, "wide")
    res = oracle.dgemm(A, B, r)
    Aq, Bq = res.extras["Aq"], res.extras["Bq"]
    for t, m in enumerate(res.ms):
        pa = ozaki2.planes_of(Aq, m)
        pb = ozaki2.planes_of(Bq.T, m)
        accs = [x @ y.T for x, y in _pairs(pa, pb, m)]
        v = planes.combine(accs, m)
        assert np.array_equal(ozaki2.centred_residue(v, m), res.residues[t])


def _pairs(pa, pb, m):
    if moduli.square_root(m):
        # acc0 = d0 e0 ; acc1 = d1 e0 + d0 e1, as one product over [d1|d0] x [e0|e1]
        return [(pa[0], pb[0]),
                (np.concatenate([pa[1], pa[0]], axis=1), np.concatenate([pb[0], pb[1]], axis=1))]
    return [(pa[2], pb[2]), (pa[0], pb[0]), (pa[1], pb[1])]


def test_scaling_bound_adversarial_long_k():
    """Eq. (M-bound) must hold with every code at its maximum and long k (the
    oracle asserts sum |A~||B~| < M/2 internally)."""
    for r in (8, 12):
        for k in (1, 1000, 20000):
            A = np.full((2, k), 1 - 2.0 ** -53)
            B = np.full((k, 2), -(1 - 2.0 ** -53))
            res = oracle.dgemm(A, B, r)
            assert np.all(res.C < 0)


@pytest.mark.parametrize("quant", ["rn", "tz"])
def test_closed_form_quantisation_bound(quant):
    """Derived from Eq. (scale): A~ = D A + dA with |dA| <= 1/2 (RN) or < 1
    (TZ), so |C - AB|_ij <= q 2^-s_i sum_l |B_lj| + q 2^-t_j sum_l |A_il| +
    q^2 k 2^-(s_i+t_j) + u |C_ij|, checked in exact rational arithmetic."""
    rng = np.random.default_rng(7)
    A, B = _rand_tiny(rng, 5, 4, 12, "wide")
    res = oracle.dgemm(A, B, 8, quant=quant)
    q = Fraction(1, 2) if quant == "rn" else Fraction(1)
    u = Fraction(1, 2 ** 53)
    k = A.shape[1]
    for i in range(5):
        for j in range(4):
            exact = refgemm.exact_dot_fraction(A[i], B[:, j])
            si, tj = int(res.sA[i]), int(res.tB[j])
            bound = (q * Fraction(2) ** -si * sum(Fraction(abs(float(b))) for b in B[:, j])
                     + q * Fraction(2) ** -tj * sum(Fraction(abs(float(a))) for a in A[i])
                     + q * q * k * Fraction(2) ** -(si + tj)
                     + u * abs(Fraction(float(res.C[i, j]))))
            assert abs(Fraction(float(res.C[i, j])) - exact) <= bound


def test_identity_times_binade_matrix_is_exact():
    rng = np.random.default_rng(3)
    n = 16
    B = rng.uniform(1, 2, (n, n)) * np.where(rng.random((n, n)) < 0.5, -1, 1)
    C = oracle.dgemm(np.eye(n), B, 12).C
    assert np.array_equal(C, B)


def test_small_integer_product_is_exact():
    rng = np.random.default_rng(4)
    A = rng.integers(-1000, 1001, (12, 30)).astype(np.float64)
    B = rng.integers(-1000, 1001, (30, 10)).astype(np.float64)
    assert np.array_equal(oracle.dgemm(A, B, 12).C, A @ B)


def test_powers_of_two_and_zeros():
    A = np.array([[2.0 ** 300, 0.0, -2.0 ** 299], [0.0, 0.0, 0.0]])
    B = np.array([[2.0 ** -700, 0.0], [5.0, 0.0], [2.0 ** -700, 0.0]])
    C = oracle.dgemm(A, B, 12).C
    assert C[0, 0] == 2.0 ** -400 - 2.0 ** -401
    assert np.all(C[1] == 0) and np.all(C[:, 1] == 0)
    assert not np.any(np.signbit(C[1])) and not np.any(np.signbit(C[:, 1]))


def test_bound_mode_widths_at_least_fixed():
    A, B = synth.lognormal(32, 32, 64, seed=11)
    rb = oracle.dgemm(A, B, 12, mode="bound")
    rf = oracle.dgemm(A, B, 12, mode="fixed")
    assert np.all(rb.extras["sigma"] >= rf.extras["sigma"])
    assert np.all(rb.extras["tau"] >= rf.extras["tau"])


def test_dd_gemm_and_exact_error_against_fractions():
    rng = np.random.default_rng(5)
    A, B = _rand_tiny(rng, 4, 3, 9, "wide")
    hi, lo = refgemm.dd_gemm(A, B)
    C = A @ B
    for i in range(4):
        for j in range(3):
            ex = refgemm.exact_dot_fraction(A[i], B[:, j])
            assert abs(Fraction(float(hi[i, j])) + Fraction(float(lo[i, j])) - ex) <= abs(ex) * Fraction(1, 2 ** 100)
            err = refgemm.exact_error(np.array([C[i, j]]), A, B, [i], [j])[0]
            assert err == float(Fraction(float(C[i, j])) - ex)


@pytest.mark.parametrize("name,r,size", [
    ("gemm256_uniform", 12, None),
    ("gemm4096_lognormal", 12, 192),
    ("gemm16384_wide", 15, 160),
])
def test_accuracy_target(name, r, size):
    """max |C - AB| / (|A||B|) <= 1e-15 at the FP64-grade moduli count, against
    the double-double reference (same distribution, reduced size)."""
    if size is None:
        A, B = synth.make(name)
    else:
        A, B, *_ = synth.make(name, m=size, n=size, k=size)
    res = oracle.dgemm(A, B, r)
    hi, lo = refgemm.dd_gemm(A, B)
    err = np.abs((res.C - hi) - lo)
    den = np.abs(A) @ np.abs(B)
    ok = np.ones(res.C.shape, bool)
    ok[np.isin(res.rows, res.fallback_rows), :] = False
    ok[:, np.isin(res.cols, res.fallback_cols)] = False
    assert np.max(err[ok] / den[ok]) <= 1e-15


def test_fallback_triggers_and_values():
    rng = np.random.default_rng(9)
    A, B = _rand_tiny(rng, 6, 5, 16, "uniform")
    A[1, 3] = np.nan
    B[2, 4] = np.inf
    A[3, ::2] *= 1e200            # intra-row span ~2^664: T2
    res = oracle.dgemm(A, B, 12)
    assert list(res.fallback_rows) == [1, 3]
    assert list(res.fallback_cols) == [4]
    assert np.all(np.isnan(res.C[1]))
    for i in (0, 2, 4, 5):
        expect = np.inf if np.any(A[i] * B[:, 4] == np.inf) else -np.inf
        if np.any(np.isnan(A[i] * B[:, 4])):
            expect = np.nan
        assert (np.isnan(res.C[i, 4]) and np.isnan(expect)) or res.C[i, 4] == expect
    for j in range(4):
        ex = refgemm.exact_dot_fraction(A[3], B[:, j])
        assert res.C[3, j] == float(ex)
    # whole-row 1e200 scaling is absorbed by per-row scaling: no fallback
    A2, B2 = _rand_tiny(rng, 6, 5, 16, "uniform")
    A2[2] *= 1e200
    r2 = oracle.dgemm(A2, B2, 12)
    assert len(r2.fallback_rows) == 0 and len(r2.fallback_cols) == 0
    hi, lo = refgemm.dd_gemm(A2, B2)
    assert np.max(np.abs((r2.C - hi) - lo) / (np.abs(A2) @ np.abs(B2))) <= 1e-15


def test_accumulate_mode():
    A, B = synth.lognormal(16, 12, 20, seed=1)
    C_in = np.random.default_rng(2).standard_normal((16, 12))
    r0 = oracle.dgemm(A, B, 12)
    r1 = oracle.dgemm(A, B, 12, C_in=C_in)
    assert np.array_equal(r1.C, C_in + r0.C)


def test_row_col_sampling_matches_full():
    A, B = synth.lognormal(40, 30, 50, seed=3)
    full = oracle.dgemm(A, B, 12)
    rows, cols = np.array([3, 17, 39]), np.array([0, 29])
    part = oracle.dgemm(A, B, 12, rows=rows, cols=cols)
    assert np.array_equal(part.C, full.C[np.ix_(rows, cols)])
    assert np.array_equal(part.residues, full.residues[:, rows][:, :, cols])


def _slab_bound_case(r):
    """1 x 196608 times 196608 x 1, every entry 1 - 2^-53: three full 65536-wide
    code slabs, every code 16 (the largest), so each slab's code product is
    256 * 65536 = 2^24.  Returns the oracle result, the exact
    sum_l |A~_l| |B~_l| (Python ints) and M."""
    k = 3 * ozaki2.CODE_SLAB
    x = 1.0 - 2.0 ** -53
    A = np.full((1, k), x)
    B = np.full((k, 1), x)
    res = oracle.dgemm(A, B, r)
    Aq, Bq = res.extras["Aq"], res.extras["Bq"]
    assert np.all(Aq == Aq[0, 0]) and np.all(Bq == Bq[0, 0])
    total = k * abs(int(Aq[0, 0])) * abs(int(Bq[0, 0]))
    return res, total, res.extras["M"], A, B


@pytest.mark.parametrize("r", [8, 9, 12, 15])
def test_code_slab_bound_beyond_65536(r):
    """k above one code slab: R_i and K_j are the sums of the three slab maxima
    (3 * 2^24), Eq. (M-bound) holds exactly (Python ints), and C is the
    correctly rounded value of the exact product A~ B~ 2^-(s+t), within the
    closed-form quantisation bound of the exact A B."""
    res, total, M, A, B = _slab_bound_case(r)
    assert int(res.R[0]) == 3 * 2 ** 24 and int(res.K[0]) == 3 * 2 ** 24
    assert 2 * total < M
    assert int(res.X[0, 0]) == total            # all terms positive and equal
    e = int(res.sA[0] + res.tB[0])
    want = Fraction(total, 2 ** e) if e >= 0 else Fraction(total * 2 ** -e)
    assert res.C[0, 0] == float(want)
    exact = Fraction(A.shape[1]) * Fraction(A[0, 0]) * Fraction(B[0, 0])
    k = A.shape[1]
    bound = (Fraction(1, 2) * Fraction(2) ** -int(res.sA[0]) * k * Fraction(B[0, 0])
             + Fraction(1, 2) * Fraction(2) ** -int(res.tB[0]) * k * Fraction(A[0, 0])
             + Fraction(k, 4) * Fraction(2) ** -e + Fraction(2) ** -53 * abs(exact))
    assert abs(Fraction(res.C[0, 0]) - exact) <= bound


@pytest.mark.parametrize("r", [8, 9, 15])
def test_code_slab_bound_catches_a_max_over_slabs_slip(r, monkeypatch):
    """The pin above is not vacuous: with the slip of taking the maximum over
    slabs instead of the sum (planted in the oracle here, on the CPU) the
    scales grow by one binary order on each side and the range condition
    Eq. (M-bound) fails for this input at r = 8, 9 and 15 (at r = 12 the
    factor-4 growth happens to stay below M/2)."""
    monkeypatch.setattr(ozaki2, "combine_slabs", np.maximum)
    try:
        res, total, M, A, B = _slab_bound_case(r)
        assert int(res.R[0]) == 2 ** 24             # the slip is in effect
        violated = 2 * total >= M
    except AssertionError as e:                     # the oracle's own range check
        violated = "range condition" in str(e)
    assert violated
