"""FP8 digit planes of a centred residue (oracle; test infrastructure only).

Section "The frozen plane kernel" of the paper:

* Square modulus m = s^2, Eq. (sq-shortcut): write the centred residue in
  balanced base s, d = d1*s + d0.  Then
  d*e = d0e0 + s*(d1e0 + d0e1) + s^2*d1e1 == d0e0 + s*(d1e0 + d0e1) (mod s^2):
  two stored planes, three products, and the two cross terms share one
  accumulator (coefficient s).
* Nonsquare modulus, Eq. (kar) with b = 4: d = d1*16 + d0 and
  d*e = (1-16) d0e0 + 16 (d0+d1)(e0+e1) + (256-16) d1e1:
  three stored planes (d0, d1, d0+d1), three products.
* Carry correction ("e4m3 layout envelope"): take the balanced base-16
  digits and, if d0+d1 is not exactly representable in E4M3, move one unit of
  base weight: (d0, d1) -> (d0 - 16*sgn(d0), d1 + sgn(d0)).  This keeps
  d = d0 + 16*d1 and places all three planes in E4M3 for nonsquare m <= 513.

READING: the balanced digit for base s is d0 = ((d + floor(s/2)) mod s) -
floor(s/2), i.e. d0 in [-floor(s/2), ceil(s/2)-1]; the paper says "balanced"
without fixing the tie side for even s.
"""
from __future__ import annotations

import numpy as np

from . import e4m3
from .moduli import square_root

NONSQUARE_BASE = 16

_E = np.zeros(2 * 512 + 1, dtype=bool)
for _x in e4m3.exact_integers():
    if -512 <= _x <= 512:
        _E[_x + 512] = True


def in_E(x):
    """Vectorised membership of integer array x in the E4M3-exact set."""
    x = np.asarray(x, dtype=np.int64)
    ok = (x >= -512) & (x <= 512)
    out = np.zeros(x.shape, dtype=bool)
    out[ok] = _E[x[ok] + 512]
    return out


def split(d, m):
    """Planes of centred residues d (int array) for modulus m.

    Returns a tuple of int64 arrays: (d0, d1) for a square modulus,
    (d0, d1, d0 + d1) for a nonsquare one.
    """
    d = np.asarray(d, dtype=np.int64)
    s = square_root(m)
    if s is not None:
        h = s // 2
        d0 = np.mod(d + h, s) - h
        d1 = (d - d0) // s
        return d0, d1
    B = NONSQUARE_BASE
    d0 = np.mod(d + B // 2, B) - B // 2
    d1 = (d - d0) // B
    bad = ~in_E(d0 + d1)
    sg = np.sign(d0)
    d0 = np.where(bad, d0 - B * sg, d0)
    d1 = np.where(bad, d1 + sg, d1)
    return d0, d1, d0 + d1


def products(pa, pb, m):
    """The three plane products per modulus, as the accumulators they feed.

    Square: acc0 = d0*e0, acc1 = d1*e0 + d0*e1.
    Nonsquare: acc0 = (d0+d1)*(e0+e1), acc1 = d0*e0, acc2 = d1*e1.
    Inputs may be scalars/arrays (elementwise) -- used for the exhaustive pins.
    """
    if square_root(m) is not None:
        d0, d1 = pa
        e0, e1 = pb
        return d0 * e0, d1 * e0 + d0 * e1
    d0, d1, ds = pa
    e0, e1, es = pb
    return ds * es, d0 * e0, d1 * e1


def combine(accs, m):
    """Epilogue coefficients: v == d*e (mod m); exact for nonsquare m.

    Square, Eq. (sq-shortcut): v = acc0 + s*acc1.
    Nonsquare, Eq. (kar) with b = 4: v = 16*acc0 - 15*acc1 + 240*acc2.
    """
    s = square_root(m)
    if s is not None:
        a0, a1 = accs
        return a0 + s * a1
    B = NONSQUARE_BASE
    a0, a1, a2 = accs
    return B * a0 + (1 - B) * a1 + (B * B - B) * a2


def max_term(m):
    """max |term| of each accumulator kind over all centred residue pairs."""
    d = centred_range(m)
    pl = split(d, m)
    mx = [int(np.max(np.abs(p))) for p in pl]
    if square_root(m) is not None:
        return mx[0] * mx[0], 2 * mx[0] * mx[1]
    return mx[2] * mx[2], mx[0] * mx[0], mx[1] * mx[1]


def centred_range(m):
    """All centred residues of m: [-floor(m/2), ceil(m/2) - 1]."""
    return np.arange(-(m // 2), (m + 1) // 2, dtype=np.int64)
