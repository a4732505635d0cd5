"""Moduli sets and CRT constants (oracle; test infrastructure only).

Paper sources:
* The published r = 12 set S: six squares 1089, 1024, 961, 841, 625, 529
  (33^2, 32^2, 31^2, 29^2, 25^2, 23^2) and the nonsquare tail
  511, 509, 503, 499, 491, 487 -- section "The frozen plane kernel",
  paragraph "Three distinct counts".
* Moduli are pairwise coprime and taken in ascending order m_1 < ... < m_r,
  Eq. (M-bound) and Alg. 1.
* Plane counts p_store = 6*2 + 6*3 = 30 and p_mma = 3r = 36, alpha = 3r+1
  ("Three distinct counts"; "Moduli count and the (3r+1) FP8 cost structure").

READING (r != 12): the paper names other sets but does not print them.  For
r != 12 we take the r largest of S plus the nonsquare extension
{481, 479, 467, 463}; the extension is pairwise coprime with S, and every
extra modulus is nonsquare and <= 513, where the carry-corrected base-16 split
applies.  This covers r = 8..16.
"""
from __future__ import annotations

import math
from functools import reduce

SET_S = (1089, 1024, 961, 841, 625, 529, 511, 509, 503, 499, 491, 487)
EXTENSION = (481, 479, 467, 463)
POOL = tuple(sorted(SET_S + EXTENSION, reverse=True))
R_MIN, R_MAX = 8, 16


def moduli(r: int) -> list[int]:
    """The r moduli in ascending (Garner) order."""
    if not (R_MIN <= r <= R_MAX):
        raise ValueError(f"num_moduli must be in [{R_MIN}, {R_MAX}], got {r}")
    return sorted(POOL[:r])


def modulus_product(ms) -> int:
    return reduce(lambda a, b: a * b, ms, 1)


def square_root(m: int) -> int | None:
    """s if m = s^2 (square modulus), else None."""
    s = math.isqrt(m)
    return s if s * s == m else None


def plane_count(m: int) -> int:
    """Stored E4M3 planes per scalar for modulus m: 2 (square), 3 (nonsquare)."""
    return 2 if square_root(m) else 3


def p_store(ms) -> int:
    return sum(plane_count(m) for m in ms)


def p_mma(ms) -> int:
    return 3 * len(ms)


def alpha(ms) -> int:
    """FP8 MMAs per emulated FMA: 3 per modulus plus the max-magnitude pass."""
    return 3 * len(ms) + 1


def width_budget(ms) -> tuple[int, int, int]:
    """(c, c_A, c_B) of the scaling rule: c = floor(log2 M) + 6, split
    c_A = floor(c/2), c_B = c - c_A.

    READING: the paper fixes only the condition M > 2 mu (Eq. (M-bound)) and
    that any valid bound mu serves (Alg. 1).  The widths below are chosen so
    that the code-product bound of the max-magnitude pass certifies
    sum_l |A~_il||B~_lj| < M/2 (see ``ozaki2.scaling``).
    """
    M = modulus_product(ms)
    c = (M.bit_length() - 1) + 6
    ca = c // 2
    return c, ca, c - ca


def garner_inverses(ms) -> list[int]:
    """inv[k] = (m_1 ... m_{k-1})^{-1} mod m_k (inv[0] unused = 0), the
    precomputed constants of Eq. (garner)."""
    out = [0]
    P = 1
    for k in range(1, len(ms)):
        P *= ms[k - 1]
        out.append(pow(P, -1, ms[k]))
    return out


def prefix_products(ms) -> list[int]:
    """P[j] = m_1 ... m_j with P[0] = 1."""
    P = [1]
    for m in ms:
        P.append(P[-1] * m)
    return P
