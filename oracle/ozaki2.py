"""Algorithm 1 (Ozaki II dense GEMM at phase level), step by step (oracle).

Test infrastructure only.  C ~= A B for float64 A (m x k), B (k x n) with r
moduli, FP8 substrate:

Phase 1 (integer scaling, Eq. (scale)):
  1. scan: E^A_i = frexp exponent of max_l |A_il|, E^B_j likewise over
     column j of B; rows/columns holding NaN or +-Inf are flagged (T1).
  2. max-magnitude pass (the trailing "+1" of alpha = 3r+1): 4-bit magnitude
     codes c = ceil(16 |x| 2^-E) in {0..16} (E4M3-exact), the code product
     G' = A^ B^ (one FP8 GEMM), row maxima R_i and column maxima K_j.
  3. widths sigma_i, tau_j and power-of-two scales s_i = sigma_i - E^A_i,
     t_j = tau_j - E^B_j (the diagonals D = diag(2^s), E = diag(2^t)).
  4. quantise A~ = RN(D A), B~ = RN(B E) (or truncation, the TZ variant of
     the numerical-contract table); rows whose nonzero entries quantise to 0
     are flagged (T2).
Phase 2 (modular GEMMs, Eq. (modgemm)): centred residues of A~, B~ per
  modulus; C^(i) = (A~ mod m_i)(B~ mod m_i) mod m_i, centred.
Phase 3 (Eq. (garner)): CRT -> exact integer C~ in [-M/2, M/2), then
  C = D^-1 C~ E^-1 rounded once to binary64.
Fallback (Alg. 1, fallback step; the contract's item (vi)): rows of A and
  columns of B the scaling cannot certify (T1/T2) are computed in native FP64
  instead.

READINGS (where the paper is silent; each is also listed in the design notes):
* The max-magnitude pass is realised with 4-bit codes relative to the row
  (column) maximum exponent; the paper only names the pass and says any valid
  bound mu serves.
* Widths: c = floor(log2 M) + 6, c_A = floor(c/2), c_B = c - c_A,
  sigma_i = min(62, c_A - ceil(ell(R_i)/2)), tau_j = min(62, c_B -
  ceil(ell(K_j)/2)), ell(x) = ceil(log2 x) (ell(0) = 0).  Then
  2^(sigma_i+tau_j-8) G'_ij <= 2^(c-8) <= M/4 and sum_l |A~||B~| <= M/4 +
  slack with slack <= k 2^max(sigma,tau) + k/4 < M/4, so Eq. (M-bound) holds
  per entry (asserted below).
* The code product is evaluated in k-slabs of 65536 (FP32-exact: a slab sum
  is at most 256 * 65536 = 2^24) and R_i is the SUM over slabs of the
  slab-wise row maxima (an upper bound of max_j G'_ij; equal to it for
  k <= 65536).  Likewise K_j.
* Fixed mode (no max pass, alpha = 3r): R_i = K_j = 256 k, the literal
  mu = k max|A~| max|B~| of Alg. 1 line "mu <- ...".
* Quantiser RN is round-half-to-even.
* Fallback trigger: T1 (non-finite entry) or T2 (a nonzero entry quantises to
  zero: the row's exponent span exceeds what the scaling certifies).  T2 is
  evaluated only on rows/columns without non-finite entries (T1 rows are not
  quantised at all).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import garner as _garner
from . import planes as _planes
from .moduli import moduli as _moduli, modulus_product, width_budget

SIGMA_CAP = 62
CODE_SLAB = 65536


@dataclass
class Result:
    C: np.ndarray                 # (len(rows), len(cols)) float64
    rows: np.ndarray
    cols: np.ndarray
    ms: list
    EA: np.ndarray
    EB: np.ndarray
    R: np.ndarray                 # row maxima of G' (all rows)
    K: np.ndarray                 # column maxima of G' (all columns)
    sA: np.ndarray                # s_i (all rows)
    tB: np.ndarray                # t_j (all columns)
    t1A: np.ndarray
    t1B: np.ndarray
    t2A: np.ndarray               # only for the rows/cols that were quantised
    t2B: np.ndarray
    residues: np.ndarray          # (r, len(rows), len(cols)) centred int64
    X: np.ndarray                 # exact integers (object), (len(rows), len(cols))
    fallback_rows: np.ndarray
    fallback_cols: np.ndarray
    extras: dict = field(default_factory=dict)


# ----------------------------------------------------------------- Phase 1

def row_exponents(A):
    """Scan of Alg. 1 Phase 1: frexp exponent of each row's max |entry|
    (0 for an all-zero row) and the non-finite flag T1 per row.
    For a column-wise scan pass A.T."""
    A = np.asarray(A, dtype=np.float64)
    finite = np.isfinite(A)
    t1 = ~np.all(finite, axis=1)
    absA = np.where(finite, np.abs(A), 0.0)
    mx = absA.max(axis=1) if A.shape[1] else np.zeros(A.shape[0])
    _, E = np.frexp(mx)
    E = np.where(mx > 0, E, 0).astype(np.int64)
    E = np.where(t1, 0, E)
    return E, t1


def magnitude_codes(A, E, t1):
    """c = ceil(16 |A_il| 2^-E_i), an integer in 0..16 (exactly 0 iff A_il = 0).

    |A_il| < 2^E_i so c <= 16, and |A_il| <= c * 2^(E_i - 4).  The scaled value
    is exact whenever it is >= 1, and any nonzero entry gets at least 1.
    Rows flagged T1 get all-zero codes (they are excluded from the pass)."""
    A = np.asarray(A, dtype=np.float64)
    a = np.where(np.isfinite(A), np.abs(A), 0.0)
    c = np.ceil(np.ldexp(a, (4 - E)[:, None]))
    c = np.where(a > 0, np.maximum(c, 1.0), 0.0)
    c = np.where(t1[:, None], 0.0, c)
    return c.astype(np.int64)


def combine_slabs(total, slab_max):
    """R_i over a k longer than one 65536-wide code slab: the SUM of the
    slab-wise row maxima (READING; an upper bound of max_j G'_ij because the
    maximum of a sum is at most the sum of the maxima)."""
    return total + slab_max


def ell(x):
    """ceil(log2 x) for integers x >= 1; 0 for x = 0."""
    x = np.asarray(x, dtype=np.int64)
    out = np.zeros(x.shape, dtype=np.int64)
    pos = x > 1
    # ceil(log2 x) = bit_length(x - 1)
    out[pos] = np.array([int(v - 1).bit_length() for v in x[pos]], dtype=np.int64)
    return out


def widths(R, cap_budget, fixed_bound=None):
    """sigma = min(62, budget - ceil(ell(R)/2)) (see READINGS)."""
    if fixed_bound is not None:
        R = np.full(np.shape(R), fixed_bound, dtype=np.int64)
    l = ell(R)
    return np.minimum(SIGMA_CAP, cap_budget - (l + 1) // 2)


def quantise(A, s, quant="rn"):
    """A~_il = RN(A_il * 2^s_i) (ties to even) or truncation toward zero.
    Exact in float64 (the result is an integer of at most 63 bits carrying at
    most 53 significant bits), returned as int64."""
    A = np.asarray(A, dtype=np.float64)
    a = np.where(np.isfinite(A), A, 0.0)
    x = np.ldexp(a, np.asarray(s, dtype=np.int64)[:, None])
    q = np.rint(x) if quant == "rn" else np.trunc(x)
    assert np.all(np.abs(q) <= 2.0 ** 62)
    return q.astype(np.int64)


def centred_residue(X, m):
    """X mod m mapped to [-floor(m/2), ceil(m/2) - 1] ([-m/2, m/2))."""
    r = np.mod(np.asarray(X, dtype=np.int64), m)
    return np.where(r >= (m + 1) // 2, r - m, r)


# ----------------------------------------------------------------- Phase 2

def modular_gemm(RA, RB, m):
    """C^(i) = centred((A~ mod m)(B~ mod m) mod m), Eq. (modgemm).
    RA (p x k) and RB (k x q) are centred residues; their fp64 product is exact
    because every partial sum is an integer below k (m/2)^2 < 2^53."""
    k = RA.shape[1]
    assert k * (m // 2 + 1) ** 2 < 2 ** 53
    P = RA.astype(np.float64) @ RB.astype(np.float64)
    return centred_residue(P.astype(np.int64), m)


# ----------------------------------------------------------------- fallback

def _two_product(a, b):
    """Error-free product a*b = p + e (Dekker/Veltkamp), exact barring
    overflow/underflow."""
    p = a * b
    sp = 134217729.0  # 2^27 + 1
    t = sp * a
    ah = t - (t - a)
    al = a - ah
    t = sp * b
    bh = t - (t - b)
    bl = b - bh
    e = ((ah * bh - p) + ah * bl + al * bh) + al * bl
    return p, e


def native_dot(a, b):
    """Reference value for a fallback entry: the exact dot product rounded once
    (finite inputs), or the IEEE class (NaN / signed Inf) of the native
    result when the inputs hold NaN or Inf."""
    import math
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if not (np.all(np.isfinite(a)) and np.all(np.isfinite(b))):
        with np.errstate(invalid="ignore", over="ignore"):
            prods = a * b
        if np.any(np.isnan(prods)):
            return float("nan")
        pos = np.any(prods == np.inf)
        neg = np.any(prods == -np.inf)
        if pos and neg:
            return float("nan")
        return float("inf") if pos else float("-inf")
    p, e = _two_product(a, b)
    return math.fsum(np.concatenate([p, e]).tolist()) + 0.0


# ----------------------------------------------------------------- driver

def dgemm(A, B, r=12, *, rows=None, cols=None, mode="bound", quant="rn",
          C_in=None, fallback=True, force_fallback=False):
    """Emulated C = A B (or C_in + A B) following Alg. 1.

    rows/cols select the output entries to compute (all by default); the
    scales are always computed from the whole matrices, as the method does.
    mode: "bound" (max-magnitude pass, alpha = 3r+1) or "fixed" (alpha = 3r).
    Returns a Result whose C has shape (len(rows), len(cols)).
    """
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    k2, n = B.shape
    assert k == k2
    ms = _moduli(r)
    M = modulus_product(ms)
    c, cA, cB = width_budget(ms)
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(n) if cols is None else np.asarray(cols)

    # Phase 1: scan + T1
    EA, t1A = row_exponents(A)
    EB, t1B = row_exponents(B.T)

    # Phase 1: max-magnitude pass (G' is formed only where it is needed:
    # rows of interest against all of B, all of A against columns of interest)
    if mode == "bound":
        cAm = magnitude_codes(A, EA, t1A).astype(np.float64)
        cBm = magnitude_codes(B.T, EB, t1B).astype(np.float64).T
        # exact: integer terms <= 256 summed over k < 2^44
        R = np.zeros(m, dtype=np.int64)
        K = np.zeros(n, dtype=np.int64)
        for l0 in range(0, max(k, 1), CODE_SLAB):
            sl = slice(l0, min(k, l0 + CODE_SLAB))
            if n:
                R[rows] = combine_slabs(R[rows], (cAm[rows, sl] @ cBm[sl]).max(axis=1).astype(np.int64))
            if m:
                K[cols] = combine_slabs(K[cols], (cAm[:, sl] @ cBm[sl, cols]).max(axis=0).astype(np.int64))
        sig = widths(R, cA)
        tau = widths(K, cB)
    elif mode == "fixed":
        R = np.full(m, 256 * k, dtype=np.int64)
        K = np.full(n, 256 * k, dtype=np.int64)
        sig = widths(R, cA)
        tau = widths(K, cB)
    else:
        raise ValueError(mode)
    sA = np.where(t1A, 0, sig - EA).astype(np.int64)
    tB = np.where(t1B, 0, tau - EB).astype(np.int64)

    # Phase 1: quantisation (only rows/cols needed for the requested block)
    Aq = quantise(np.where(t1A[rows][:, None], 0.0, A[rows]), sA[rows], quant)
    Bq = quantise(np.where(t1B[cols][:, None], 0.0, B[:, cols].T), tB[cols], quant).T
    # T2 is evaluated only on rows/columns that are quantised (not T1)
    t2A = ~t1A[rows] & np.any((A[rows] != 0) & (Aq == 0), axis=1)
    t2B = ~t1B[cols] & np.any((B[:, cols] != 0) & (Bq == 0), axis=0)

    # Eq. (M-bound) for every computed entry: sum_l |A~_il||B~_lj| < M/2.
    # Checked exactly in Python integers for small blocks.
    if Aq.shape[0] * Bq.shape[1] * k <= 1 << 16:
        for ii in range(Aq.shape[0]):
            for jj in range(Bq.shape[1]):
                tot = sum(abs(int(x)) * abs(int(y)) for x, y in zip(Aq[ii], Bq[:, jj]))
                assert 2 * tot < M, "range condition violated"
    else:
        # fp64 upper bound (relative error < 2^-40 at these sizes) with margin
        ub = np.abs(Aq).astype(np.float64) @ np.abs(Bq).astype(np.float64)
        assert np.all(ub * (1 + 2.0 ** -30) < float(M) / 2), "range condition violated"

    # Phase 2: residues and modular GEMMs
    res = np.zeros((r, len(rows), len(cols)), dtype=np.int64)
    for i, mi in enumerate(ms):
        RA = centred_residue(Aq, mi)
        RB = centred_residue(Bq, mi)
        res[i] = modular_gemm(RA, RB, mi)

    # Phase 3: Garner -> exact integer -> one rounding of X * 2^-(s_i + t_j)
    X = _garner.crt(res, ms)
    e = sA[rows][:, None] + tB[cols][None, :]
    Cv = _garner.round_scaled_array(X, e) if X.size else np.zeros(X.shape)

    # fallback rows / columns (native FP64 reference values)
    fr = np.zeros(len(rows), dtype=bool)
    fc = np.zeros(len(cols), dtype=bool)
    if fallback:
        fr = t1A[rows] | t2A
        fc = t1B[cols] | t2B
        if force_fallback:
            fr[:] = True
    for ii in np.nonzero(fr)[0]:
        for jj in range(len(cols)):
            Cv[ii, jj] = native_dot(A[rows[ii]], B[:, cols[jj]])
    for jj in np.nonzero(fc)[0]:
        for ii in range(len(rows)):
            if not fr[ii]:
                Cv[ii, jj] = native_dot(A[rows[ii]], B[:, cols[jj]])

    if C_in is not None:
        Cv = np.asarray(C_in, dtype=np.float64)[np.ix_(rows, cols)] + Cv

    return Result(C=Cv, rows=rows, cols=cols, ms=ms, EA=EA, EB=EB, R=R, K=K,
                  sA=sA, tB=tB, t1A=t1A, t1B=t1B, t2A=t2A, t2B=t2B,
                  residues=res, X=X, fallback_rows=rows[fr], fallback_cols=cols[fc],
                  extras=dict(Aq=Aq, Bq=Bq, sigma=sig, tau=tau, M=M, c=(c, cA, cB)))


def planes_of(Xq, m):
    """Digit planes of the centred residues of the integer matrix Xq."""
    return _planes.split(centred_residue(Xq, m), m)
