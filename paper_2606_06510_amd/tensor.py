"""Tensor-level helpers around the C ABI (marshalling only).

Column-major (BLAS) matrices are held in torch as the transpose of a
contiguous row-major tensor: an m x k matrix with leading dimension m is the
memory of a contiguous (k, m) tensor, exposed here as its (m, k) view with
strides (1, m).
"""
from __future__ import annotations

import numpy as np

from . import _lib


def colmajor_empty(m, n, device="cuda", dtype=None):
    import torch
    return torch.empty((n, m), dtype=dtype or torch.float64, device=device).t()


def to_device_colmajor(X, device="cuda"):
    """numpy (any order) -> column-major float64 device tensor (m, n) view."""
    import torch
    Xt = np.ascontiguousarray(np.asarray(X, dtype=np.float64).T)
    return torch.from_numpy(Xt).to(device).t()


def from_device_colmajor(T):
    return T.t().contiguous().cpu().numpy().T


def _ld(T):
    if T.dim() != 2 or T.stride(0) != 1:
        raise ValueError("expected a column-major (m, n) view with stride (1, ld)")
    return max(T.stride(1), 1)


def matmul(A, B, num_moduli=12, flags=0, C=None, workspace=None, stream=None):
    """C = A B (or C += A B with OZ2_ACCUMULATE) for column-major float64
    device tensors; returns C."""
    import torch
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    if C is None:
        C = colmajor_empty(m, n, device=A.device)
    need = _lib.ozaki2_workspace_bytes(m, n, k, num_moduli, flags)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=A.device)
    _lib.ozaki2_dgemm_ex(m, n, k, A, _ld(A), B, _ld(B), C, _ld(C), num_moduli, flags,
                         workspace, workspace.numel(), stream)
    return C


class Plan:
    """The staged API over one workspace: deconstruct, residue_gemm,
    reconstruct, and the diagnostic queries (as numpy arrays)."""

    def __init__(self, m, n, k, num_moduli=12, flags=0, device="cuda"):
        import torch
        self.m, self.n, self.k, self.r, self.flags = m, n, k, num_moduli, flags
        self.ws_bytes = _lib.ozaki2_workspace_bytes(m, n, k, num_moduli, flags)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.handle = _lib.ozaki2_plan_create(m, n, k, num_moduli, flags, self.workspace,
                                              self.ws_bytes)
        self.moduli = _lib.ozaki2_moduli(num_moduli)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            try:
                _lib.ozaki2_plan_destroy(h)
            except Exception:   # interpreter shutdown: the library may be gone already
                pass
            self.handle = None

    def deconstruct(self, A, B, stream=None):
        self._A, self._B = A, B      # borrowed by the plan until reconstruct
        _lib.ozaki2_deconstruct(self.handle, A, _ld(A), B, _ld(B), stream)

    def deconstruct_a(self, A, stream=None):
        """Operand-stationary use (OZ2_SCALE_FIXED plans): new A, B's planes kept."""
        self._A = A
        _lib.ozaki2_deconstruct_a(self.handle, A, _ld(A), stream)

    def deconstruct_b(self, B, stream=None):
        """Operand-stationary use (OZ2_SCALE_FIXED plans): new B, A's planes kept."""
        self._B = B
        _lib.ozaki2_deconstruct_b(self.handle, B, _ld(B), stream)

    def residue_gemm(self, stream=None):
        _lib.ozaki2_residue_gemm(self.handle, stream)

    def reconstruct(self, C, stream=None):
        _lib.ozaki2_reconstruct(self.handle, C, _ld(C), stream)

    def query(self, what):
        m, n, k, r = self.m, self.n, self.k, self.r
        nb = _lib.ozaki2_plan_query_bytes(self.handle, what)
        raw = np.zeros(nb, dtype=np.uint8)
        _lib.ozaki2_plan_query(self.handle, what, raw)
        if what in (_lib.OZ2_Q_EXPONENTS, _lib.OZ2_Q_SCALES):
            v = raw.view(np.int32)
            return v[:m].copy(), v[m:].copy()
        if what == _lib.OZ2_Q_MAXIMA:
            v = raw.view(np.uint64)
            return v[:m].copy(), v[m:].copy()
        if what == _lib.OZ2_Q_FLAGS:
            v = raw.view(np.uint32)
            return v[:m].copy(), v[m:].copy()
        if what == _lib.OZ2_Q_CODES:
            return raw[:m * k].reshape(m, k).copy(), raw[m * k:].reshape(n, k).copy()
        if what == _lib.OZ2_Q_PLANES:
            P = nb // ((m + n) * k)
            return (raw[:P * m * k].reshape(P, m, k).copy(),
                    raw[P * m * k:].reshape(P, n, k).copy())
        if what == _lib.OZ2_Q_RESIDUES:
            return raw.view(np.int16).reshape(r, n, m).transpose(0, 2, 1).copy()
        if what == _lib.OZ2_Q_INTEGERS:
            w = raw.view(np.uint32).reshape(n, m, 5)
            out = np.empty((m, n), dtype=object)
            for j in range(n):
                for i in range(m):
                    v = 0
                    for q in range(4, -1, -1):
                        v = (v << 32) | int(w[j, i, q])
                    if v >> 159:
                        v -= 1 << 160
                    out[i, j] = v
            return out
        if what == _lib.OZ2_Q_FALLBACK_COUNT:
            v = raw.view(np.int32)
            return int(v[0]), int(v[1])
        return raw
