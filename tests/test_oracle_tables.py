"""Pins of the oracle's tables against values the paper prints and against
the definitions (number theory, the E4M3 format)."""
import math

import numpy as np
import pytest

from oracle import e4m3, moduli, planes


def test_set_S_matches_paper(golden):
    assert sorted(moduli.SET_S, reverse=True) == golden["set_S"]["value"]
    assert moduli.moduli(12) == sorted(golden["set_S"]["value"])


@pytest.mark.parametrize("r", range(8, 17))
def test_moduli_pairwise_coprime_ascending(r):
    ms = moduli.moduli(r)
    assert ms == sorted(ms) and len(set(ms)) == r
    for i in range(r):
        for j in range(i + 1, r):
            assert math.gcd(ms[i], ms[j]) == 1


def test_log2M_and_plane_counts(golden):
    ms = moduli.moduli(12)
    M = moduli.modulus_product(ms)
    assert abs(math.log2(M) - golden["log2_M_S"]["value"]) < golden["log2_M_S"]["tol"]
    assert moduli.p_store(ms) == golden["p_store_S"]["value"]
    assert moduli.p_mma(ms) == golden["p_mma_S"]["value"]
    assert moduli.alpha(ms) == golden["alpha_r12"]["value"]


def test_e4m3_format(golden):
    vals = [e4m3.decode(b) for b in range(256)]
    finite = [v for v in vals if v == v]
    assert max(finite) == golden["e4m3_max"]["value"]
    assert sum(1 for v in vals if v != v) == 2          # S.1111.111 only
    assert e4m3.decode(0x38) == 1.0 and e4m3.decode(0x00) == 0.0
    assert e4m3.decode(0x01) == 2.0 ** -9                # smallest subnormal
    E = set(e4m3.exact_integers())
    lim = golden["e4m3_consecutive_limit"]["value"]
    assert all(x in E for x in range(-lim, lim + 1)) and (lim + 1) not in E
    for x in golden["e4m3_exact_examples"]["value"]:
        assert x in E and -x in E
    for x in golden["e4m3_inexact_examples"]["value"]:
        assert x not in E
    # the paper's characterisation: M * 2^e with |M| <= 15, magnitude <= 448
    char = {s * M * 2 ** e for M in range(0, 16) for e in range(0, 9) for s in (1, -1)
            if M * 2 ** e <= 448}
    assert E == char


def test_e4m3_encoder_roundtrip():
    for x in e4m3.exact_integers():
        assert e4m3.decode(e4m3.encode_int(x)) == x
    assert e4m3.encode_int(0) == 0


# ------------------------------------------------------------ plane algebra

def _all_pairs(m):
    d = planes.centred_range(m)
    D, E = np.meshgrid(d, d, indexing="ij")
    return D.ravel(), E.ravel()


@pytest.mark.parametrize("m", moduli.POOL)
def test_plane_identity_exhaustive(m):
    """Every ordered centred pair (d, e): the three plane products, combined
    with the epilogue coefficients, reproduce d*e mod m (square: Eq.
    (sq-shortcut)) or d*e exactly (nonsquare: Eq. (kar))."""
    d, e = _all_pairs(m)
    pa = planes.split(d, m)
    pb = planes.split(e, m)
    for p in pa:
        assert np.all(planes.in_E(p))
    v = planes.combine(planes.products(pa, pb, m), m)
    if moduli.square_root(m):
        assert np.all(np.mod(v - d * e, m) == 0)
    else:
        assert np.all(v == d * e)


@pytest.mark.parametrize("m", moduli.POOL)
def test_plane_split_reassembles(m):
    d = planes.centred_range(m)
    pl = planes.split(d, m)
    s = moduli.square_root(m)
    base = s if s else planes.NONSQUARE_BASE
    assert np.all(pl[0] + base * pl[1] == d)
    if not s:
        assert np.all(pl[2] == pl[0] + pl[1])


def test_tail_bounds_and_corrected_fraction(golden):
    gb = golden["tail_digit_bounds"]
    fr = golden["tail_corrected_fraction"]
    for m in moduli.SET_S:
        if moduli.square_root(m):
            d = planes.centred_range(m)
            d0, d1 = planes.split(d, m)
            assert np.max(np.abs(d0)) <= 16 and np.max(np.abs(d1)) <= 16
            continue
        d = planes.centred_range(m)
        d0, d1, ds = planes.split(d, m)
        assert np.max(np.abs(d0)) == gb["d0"]
        assert np.max(np.abs(d1)) == gb["d1"]
        assert np.max(np.abs(ds)) == gb["sum"]
        canon0 = np.mod(d + 8, 16) - 8
        frac = np.mean(canon0 != d0)
        assert abs(frac - fr["value"]) <= fr["tol"], (m, frac)


def test_max_terms_and_slab(golden):
    sq = [planes.max_term(m) for m in moduli.SET_S if moduli.square_root(m)]
    ns = [planes.max_term(m) for m in moduli.SET_S if not moduli.square_root(m)]
    assert max(t[0] for t in sq) == golden["max_term_square_d0e0"]["value"]
    assert max(t[1] for t in sq) == golden["max_term_square_cross"]["value"]
    assert max(t[0] for t in ns) == golden["max_term_tail_sum"]["value"]
    worst = max(max(t) for t in sq + ns)
    # Eq. (accum-exact) with the slab length used by the GPU path
    kslab = 32768
    assert kslab * worst <= 2 ** golden["fp32_exact_integer_limit_log2"]["value"]


def _canonical_ok(m, B, redundant):
    d = planes.centred_range(m)
    d0 = np.mod(d + B // 2, B) - B // 2
    d1 = (d - d0) // B
    if redundant:
        bad = ~planes.in_E(d0 + d1)
        sg = np.sign(d0)
        d0 = np.where(bad, d0 - B * sg, d0)
        d1 = np.where(bad, d1 + sg, d1)
    return bool(np.all(planes.in_E(d0)) and np.all(planes.in_E(d1)) and np.all(planes.in_E(d0 + d1)))


def _envelope(B, redundant):
    m = 2
    while _canonical_ok(m + 1, B, redundant):
        m += 1
    return m


def test_layout_envelope(golden):
    """Eq. (envelope), found by exhaustive base search (the centred ranges are
    nested in m, so the envelope is the last m before the first failure)."""
    env = {B: _envelope(B, False) for B in range(4, 41)}
    best = max(env.values())
    assert best == golden["envelope_canonical_max"]["value"]
    assert env[golden["envelope_canonical_max"]["base"]] == best
    assert env[16] == golden["envelope_canonical_base16"]["value"]
    assert _envelope(16, True) == golden["envelope_redundant_base16"]["value"]
    assert _envelope(golden["envelope_redundant_max"]["base"], True) == golden["envelope_redundant_max"]["value"]
    # squares: balanced base-s digits of every centred residue stay exact up to s = 33
    smax = golden["envelope_square_max_s"]["value"]
    for s in range(2, smax + 1):
        d = planes.centred_range(s * s)
        d0 = np.mod(d + s // 2, s) - s // 2
        d1 = (d - d0) // s
        assert np.all(planes.in_E(d0)) and np.all(planes.in_E(d1))
    s = smax + 1            # tight: the next square fails
    d = planes.centred_range(s * s)
    d0 = np.mod(d + s // 2, s) - s // 2
    assert not np.all(planes.in_E((d - d0) // s))
