"""Pins of Garner / CRT and of the single final rounding."""
import math
import random

import numpy as np
import pytest

from oracle import garner, moduli


def _closed_form_r3(C, m1, m2, m3):
    """App. A: v1 = C1, v2 = (C2 - v1) m1^-1 mod m2,
    v3 = ((C3 - v1) m1^-1 - v2) m2^-1 mod m3."""
    c1, c2, c3 = C % m1, C % m2, C % m3
    v1 = c1
    v2 = ((c2 - v1) * pow(m1, -1, m2)) % m2
    v3 = (((c3 - v1) * pow(m1, -1, m3) - v2) * pow(m2, -1, m3)) % m3
    return v1, v2, v3


@pytest.mark.parametrize("ms", [(3, 5, 7), (29, 31, 32)])
def test_garner_r3_closed_form_exhaustive(ms):
    m1, m2, m3 = ms
    Ms = m1 * m2 * m3
    Cs = np.arange(Ms, dtype=np.int64)
    x = np.stack([Cs % m for m in ms])
    v = garner.garner_digits(x, list(ms))
    for C in range(Ms):
        cf = _closed_form_r3(C, m1, m2, m3)
        assert tuple(int(t) for t in v[:, C]) == cf
        assert cf[0] + cf[1] * m1 + cf[2] * m1 * m2 == C      # Eq. (mixedradix)


def _centred(X, m):
    v = X % m
    return v - m if v >= (m + 1) // 2 else v


@pytest.mark.parametrize("r", range(8, 17))
def test_crt_identity(r):
    ms = moduli.moduli(r)
    M = moduli.modulus_product(ms)
    rnd = random.Random(r)
    Xs = [0, 1, -1, -(M // 2), (M + 1) // 2 - 1, M // 2 - 1, -(M // 2) + 1]
    Xs += [rnd.randrange(-(M // 2), (M + 1) // 2) for _ in range(300)]
    # residues in the centred representatives, as the GPU produces them
    x = np.array([[_centred(X, m) for X in Xs] for m in ms], dtype=np.int64)
    got = garner.crt(x, ms)
    assert [int(g) for g in got] == Xs


def test_crt_brute_force_small():
    # all integers of a tiny symmetric range round-trip (the range is defined
    # by M alone; Garner must not depend on the set being the paper's)
    ms = [7, 9, 11, 13]
    M = 7 * 9 * 11 * 13
    Xs = list(range(-(M // 2), (M + 1) // 2))
    x = np.array([[X % m for X in Xs] for m in ms], dtype=np.int64)
    got = garner.crt(x, ms)
    assert [int(g) for g in got] == Xs


def _bits(f):
    return np.float64(f).view(np.uint64)


@pytest.mark.parametrize("X,e,want", [
    (1, 1074, 2.0 ** -1074),                  # smallest subnormal
    (1, 1075, 0.0),                           # exact half of it: tie to even -> 0
    (3, 1075, 2.0 ** -1073),                  # 1.5 ulp: tie to even -> 2 ulp
    (5, 1076, 2.0 ** -1074),                  # 1.25 ulp -> 1 ulp
    (2 ** 53 + 1, 0, 2.0 ** 53),              # tie to even (down)
    (2 ** 53 + 3, 0, 2.0 ** 53 + 4),          # tie to even (up)
    (2 ** 53 + 1, 1, 2.0 ** 52 + 0.5),        # exact
    ((2 ** 53 - 1), -971, 1.7976931348623157e308),   # DBL_MAX
    ((2 ** 54 - 1), -970, math.inf),          # rounds up past DBL_MAX
    (2 ** 1024, 0, math.inf),
    (-(2 ** 1024), 0, -math.inf),
    (-1, 1075, -0.0),                         # negative underflow keeps its sign
    (0, 5, 0.0),
    (0, -5, 0.0),
    (12345, 0, 12345.0),
    (-(2 ** 60 + 2 ** 7 + 1), 60, -(1.0 + 2.0 ** -52)),   # above half ulp -> up
])
def test_round_scaled_ieee(X, e, want):
    got = garner.round_scaled(X, e)
    assert _bits(got) == _bits(want), (got, want)
