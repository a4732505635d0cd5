"""Seeded synthetic workloads for the emulated FP64 GEMM.

This module only draws random numbers.  It holds none of the method's
arithmetic, so both the CPU oracle and the GPU path may use it without
sharing any computation.  Every matrix is float64 in column-major (BLAS,
Fortran) order, the layout the library expects.

Recipes (numpy PCG64 via ``default_rng(seed)``; draw order is A, then B, then
any extra draws):

* ``uniform``  (256^3 correctness case): A, B iid ``2*rng.random()-1``.
* ``lognormal05`` (4096^3 accuracy/throughput case): entries
  ``(u-0.5)*exp(0.5*g)``, u ~ U(0,1), g ~ N(0,1); u for the whole matrix is
  drawn first, then g.
* ``wide`` (16384^3 wide-range case): entries ``(u-0.5)*exp(2.0*g)``, then
  ``rows = rng.random(m) < 0.01`` and ``A[rows, :] *= 1e200`` (whole rows).
* ``wide_span``: as ``wide`` but in each selected row a random half of the
  entries is scaled (``rng.random(k) < 0.5`` per selected row), so the row
  spans ~2^664 and cannot be certified by per-row scaling.
* ``rankk`` (rank-k update): A m x k, B k x n, C_in m x n, all
  ``(u-0.5)*exp(0.5*g)``; C_in drawn after A and B.
* ``gemv16384x8`` (batched GEMV): A 16384 x 16384 and X 16384 x 8, entries
  as ``lognormal05`` (seed 6).
* ``batched``: ``batch`` independent problems; A_b, B_b iid U(-1,1), each
  multiplied by its own scale ``10**rng.uniform(-8, 8)``; all A entries are
  drawn first, then all B entries, then the A scales, then the B scales.
"""
from __future__ import annotations

import numpy as np

__all__ = ["CONFIGS", "make", "uniform", "lognormal", "wide", "rankk", "batched"]


def _exp(x):
    """Elementwise exp of a float64 array.  Evaluated with torch's vectorised,
    multi-threaded CPU kernel when torch is importable (numpy's takes over a
    minute for the 2^28 entries of a 16384^2 matrix on some hosts; the two
    can differ by an ulp on some entries, so every consumer of these inputs
    draws them through this function), else with numpy."""
    try:
        import torch
    except ImportError:  # pragma: no cover
        return np.exp(x)
    return torch.exp(torch.from_numpy(np.ascontiguousarray(x))).numpy()


def _lognormal(rng, shape, spread):
    u = rng.random(shape)
    g = rng.standard_normal(shape)
    return (u - 0.5) * _exp(spread * g)


def uniform(m, n, k, seed=0):
    rng = np.random.default_rng(seed)
    A = 2.0 * rng.random((m, k)) - 1.0
    B = 2.0 * rng.random((k, n)) - 1.0
    return np.asfortranarray(A), np.asfortranarray(B)


def lognormal(m, n, k, seed=2, spread=0.5):
    rng = np.random.default_rng(seed)
    A = _lognormal(rng, (m, k), spread)
    B = _lognormal(rng, (k, n), spread)
    return np.asfortranarray(A), np.asfortranarray(B)


def wide(m, n, k, seed=3, spread=2.0, frac=0.01, big=1e200, half_rows=False):
    rng = np.random.default_rng(seed)
    A = _lognormal(rng, (m, k), spread)
    B = _lognormal(rng, (k, n), spread)
    rows = np.nonzero(rng.random(m) < frac)[0]
    for i in rows:
        if half_rows:
            sel = rng.random(k) < 0.5
            A[i, sel] *= big
        else:
            A[i, :] *= big
    return np.asfortranarray(A), np.asfortranarray(B), rows


def rankk(m, n, k, seed=4, spread=0.5):
    rng = np.random.default_rng(seed)
    A = _lognormal(rng, (m, k), spread)
    B = _lognormal(rng, (k, n), spread)
    C = _lognormal(rng, (m, n), spread)
    return np.asfortranarray(A), np.asfortranarray(B), np.asfortranarray(C)


def batched(batch, m, n, k, seed=5, decades=8.0):
    """Returns A (batch, m, k) and B (batch, k, n); each matrix column-major
    inside its own slab, slabs contiguous (stride m*k and k*n)."""
    rng = np.random.default_rng(seed)
    A = 2.0 * rng.random((batch, k, m)) - 1.0   # [b][col][row] = column-major slabs
    B = 2.0 * rng.random((batch, n, k)) - 1.0
    sa = 10.0 ** rng.uniform(-decades, decades, batch)
    sb = 10.0 ** rng.uniform(-decades, decades, batch)
    A *= sa[:, None, None]
    B *= sb[:, None, None]
    # expose as (batch, m, k) views whose per-matrix memory is column-major
    return A.transpose(0, 2, 1), B.transpose(0, 2, 1)


# name -> (description, generator call, moduli count used for acceptance)
CONFIGS = {
    "gemm256_uniform": dict(kind="uniform", m=256, n=256, k=256, seed=0, r=12),
    "gemm4096_lognormal": dict(kind="lognormal", m=4096, n=4096, k=4096, seed=2, r=12),
    "gemm16384_wide": dict(kind="wide", m=16384, n=16384, k=16384, seed=3, r=15),
    "gemm16384_wide_span": dict(kind="wide_span", m=16384, n=16384, k=16384, seed=31, r=15),
    "rankk32768x256": dict(kind="rankk", m=32768, n=32768, k=256, seed=4, r=12),
    "batched8192x64": dict(kind="batched", batch=8192, m=64, n=64, k=64, seed=5, r=12),
    # batched GEMV Y = A X (n = right-hand sides): A as the 4096^3 case's entries
    "gemv16384x8": dict(kind="lognormal", m=16384, n=8, k=16384, seed=6, r=13),
}


def make(name, **override):
    """Draw the inputs of a named workload (sizes may be overridden for
    smaller parity cases that keep the same distribution)."""
    cfg = dict(CONFIGS[name])
    cfg.update(override)
    kind = cfg["kind"]
    if kind == "uniform":
        return uniform(cfg["m"], cfg["n"], cfg["k"], cfg["seed"])
    if kind == "lognormal":
        return lognormal(cfg["m"], cfg["n"], cfg["k"], cfg["seed"])
    if kind == "wide":
        return wide(cfg["m"], cfg["n"], cfg["k"], cfg["seed"])
    if kind == "wide_span":
        return wide(cfg["m"], cfg["n"], cfg["k"], cfg["seed"], half_rows=True)
    if kind == "rankk":
        return rankk(cfg["m"], cfg["n"], cfg["k"], cfg["seed"])
    if kind == "batched":
        return batched(cfg["batch"], cfg["m"], cfg["n"], cfg["k"], cfg["seed"])
    raise KeyError(kind)
