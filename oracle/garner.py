"""CRT reconstruction and the single rounding back to FP64 (oracle).

* Garner's algorithm, Eq. (garner): with non-negative residues x_k of the
  integer C modulo m_k,
      v_1 = x_1,
      v_k = (x_k - sum_{j<k} v_j * P_{j-1}) * P_{k-1}^{-1}  (mod m_k),
  where P_j = m_1 ... m_j and the inverses are precomputed once; then
  C = v_1 + v_2 P_1 + v_3 P_2 + ... (mixed radix, Eq. (mixedradix), App. A).
* The symmetric range of Eq. (M-bound): the entry lies in [-M/2, M/2), so a
  reconstruction X in [0, M) with 2X >= M stands for X - M.
* Rescale, Alg. 1 last step: C = D^{-1} C~ E^{-1} with power-of-two D, E.
  The paper asks for one rounded conversion of the exact multi-limb integer
  (App. B, "one rounded cvt to fp64").  READING: that rounding is IEEE
  round-to-nearest-even of the exact rational X * 2^-(s_i + t_j), with
  gradual underflow and overflow to infinity, and an exact zero is +0.0.
"""
from __future__ import annotations

import numpy as np

from .moduli import garner_inverses, modulus_product, prefix_products


def garner_digits(x, ms):
    """Mixed-radix digits of Eq. (garner).

    x: int array of shape (r, ...) of residues (any representatives).
    Returns int64 array v of the same shape with 0 <= v_k < m_k.
    All intermediate values are below 2^40, so int64 is exact.
    """
    x = np.asarray(x, dtype=np.int64)
    r = len(ms)
    inv = garner_inverses(ms)
    P = prefix_products(ms)
    v = np.zeros_like(x)
    v[0] = np.mod(x[0], ms[0])
    for k in range(1, r):
        mk = ms[k]
        acc = np.zeros_like(x[0])
        for j in range(k):
            acc = acc + v[j] * (P[j] % mk)      # v_j * P_{j-1}, P indexed from P_0 = 1
        v[k] = np.mod(np.mod(x[k] - acc, mk) * inv[k], mk)
    return v


def mixed_radix_value(v, ms):
    """X = sum_k v_k P_{k-1} as Python ints (object array), X in [0, M)."""
    P = prefix_products(ms)
    v = np.asarray(v, dtype=np.int64)
    X = np.zeros(v.shape[1:], dtype=object)
    X[...] = 0
    for k in range(len(ms)):
        X = X + v[k].astype(object) * P[k]
    return X


def centre(X, ms):
    """Map X in [0, M) to the symmetric range [-M/2, M/2)."""
    M = modulus_product(ms)
    Xo = np.asarray(X, dtype=object)
    f = np.frompyfunc(lambda a: a - M if 2 * a >= M else a, 1, 1)
    return f(Xo)


def crt(x, ms):
    """Residues (r, ...) -> the unique integer in [-M/2, M/2)."""
    return centre(mixed_radix_value(garner_digits(x, ms), ms), ms)


def round_scaled(X: int, e: int) -> float:
    """Correctly rounded binary64 value of the exact rational X * 2^-e.

    Python's int/int true division and int->float conversion are correctly
    rounded (ties to even, gradual underflow); overflow raises, which maps to
    a signed infinity here.  An exact zero returns +0.0.
    """
    X = int(X)
    e = int(e)
    if X == 0:
        return 0.0
    try:
        if e <= 0:
            return float(X << (-e))
        return X / (1 << e)
    except OverflowError:
        return float("inf") if X > 0 else float("-inf")


def round_scaled_array(X, e):
    f = np.frompyfunc(round_scaled, 2, 1)
    return f(np.asarray(X, dtype=object), np.asarray(e, dtype=object)).astype(np.float64)
