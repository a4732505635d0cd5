"""Reference products for the accuracy metric (oracle; test infrastructure).

The target metric is the componentwise ratio
    max_ij |C_ij - (AB)_ij| / (|A||B|)_ij,
for which the exact product is needed to well below 1e-15 relative.

* ``dd_gemm``: a double-double GEMM (Ogita-Rump-Oishi Dot2: error-free
  TwoProduct and TwoSum, with the errors summed in a second word), accurate as
  if computed in twice the working precision.  Vectorised over outputs, with a
  Python loop over k: for small and medium sizes.
* ``exact_error``: for sampled entries, the error C_ij - (AB)_ij rounded
  once, via math.fsum (exactly rounded summation) of the error-free
  products and -C_ij.  Exact barring underflow in the products.
* ``exact_dot_fraction``: exact rational dot product (fractions.Fraction),
  for tiny brute-force pins.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np


def _two_sum(a, b):
    s = a + b
    bb = s - a
    e = (a - (s - bb)) + (b - bb)
    return s, e


def _split(a):
    t = 134217729.0 * a
    hi = t - (t - a)
    return hi, a - hi


def _two_product(a, b):
    p = a * b
    ah, al = _split(a)
    bh, bl = _split(b)
    e = ((ah * bh - p) + ah * bl + al * bh) + al * bl
    return p, e


def dd_gemm(A, B):
    """(hi, lo) with hi + lo ~= AB to about 2^-104 relative per term sum."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    n = B.shape[1]
    s = np.zeros((m, n))
    c = np.zeros((m, n))
    for l in range(k):
        p, e = _two_product(A[:, l:l + 1], B[l:l + 1, :])
        s, q = _two_sum(s, p)
        c = c + (q + e)
    hi, lo = _two_sum(s, c)
    return hi, lo


def exact_error(C, A, B, rows, cols):
    """err_t = RN((C - AB)_{rows[t], cols[t]}) for each sampled pair t."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    out = np.empty(len(rows))
    for t, (i, j) in enumerate(zip(rows, cols)):
        p, e = _two_product(A[i, :], B[:, j])
        terms = np.concatenate([-p, -e, [C[t] if np.ndim(C) == 1 else C[i, j]]])
        out[t] = math.fsum(terms.tolist())
    return out


def abs_product(A, B, rows, cols):
    """(|A||B|)_ij for the sampled pairs (fp64; only a denominator)."""
    A = np.abs(np.asarray(A, dtype=np.float64))
    B = np.abs(np.asarray(B, dtype=np.float64))
    return np.array([A[i, :] @ B[:, j] for i, j in zip(rows, cols)])


def componentwise_ratio(C, A, B, rows, cols):
    """max over sampled pairs of |C - AB| / (|A||B|) (0/0 counts as 0)."""
    err = np.abs(exact_error(C, A, B, rows, cols))
    den = abs_product(A, B, rows, cols)
    with np.errstate(invalid="ignore", divide="ignore"):
        q = np.where(den > 0, err / np.where(den > 0, den, 1.0), np.where(err > 0, np.inf, 0.0))
    return float(np.max(q)) if len(q) else 0.0


def exact_dot_fraction(a, b):
    return sum((Fraction(float(x)) * Fraction(float(y)) for x, y in zip(a, b)), Fraction(0))
