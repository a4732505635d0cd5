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
    """Leading dimension of a column-major (m, n) view.  A dimension of size
    1 carries no stride information (numpy and torch normalise it), so a
    single column has leading dimension max(m, 1) and a single row any
    stride."""
    if T.dim() != 2:
        raise ValueError("expected a column-major (m, n) view with stride (1, ld)")
    m, n = T.shape
    if m > 1 and T.stride(0) != 1:
        raise ValueError("expected a column-major (m, n) view with stride (1, ld)")
    if n <= 1:
        return max(m, 1)
    return max(T.stride(1), 1)


def _check_matrices(device, *items):
    """items: (name, tensor, (rows, cols)).  The C ABI sees only pointers and
    sizes, so a tensor of the wrong shape, dtype or device would be read or
    written out of bounds by the kernels: refuse it here, before any library
    call (shapes of all tensors first, then dtypes and layouts, then devices).
    Returns the leading dimensions."""
    import torch
    for name, T, shape in items:
        if not isinstance(T, torch.Tensor):
            raise TypeError(f"{name}: expected a torch tensor, got {type(T).__name__}")
        if T.dim() != 2 or tuple(T.shape) != tuple(shape):
            raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(T.shape)}")
    lds = []
    for name, T, shape in items:
        if T.dtype != torch.float64:
            raise ValueError(f"{name}: expected dtype torch.float64, got {T.dtype}")
        lds.append(_ld(T))
    want = "a CUDA device" if device is None or torch.device(device).type != "cuda" else str(device)
    for name, T, shape in items:
        if T.device.type != "cuda" or (want != "a CUDA device" and T.device != torch.device(device)):
            raise ValueError(f"{name}: expected a tensor on {want}, got one on {T.device}")
    return lds


def matmul(A, B, num_moduli=12, flags=0, C=None, workspace=None, stream=None):
    """C = A B (or C += A B with OZ2_ACCUMULATE) for column-major float64
    device tensors; returns C."""
    import torch
    if A.dim() != 2 or B.dim() != 2:
        raise ValueError("A and B must be matrices")
    m, k = A.shape
    k2, n = B.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    dev = A.device
    items = [("A", A, (m, k)), ("B", B, (k, n))] + ([("C", C, (m, n))] if C is not None else [])
    _check_matrices(dev, *items)
    if C is None:
        C = colmajor_empty(m, n, device=dev)
    lda, ldb, ldc = _check_matrices(dev, ("A", A, (m, k)), ("B", B, (k, n)), ("C", C, (m, n)))
    if workspace is None:
        need = _lib.ozaki2_workspace_bytes(m, n, k, num_moduli, flags)
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    elif workspace.device != dev:
        raise ValueError("workspace: on another device")
    # the library checks the workspace size against the route it takes
    _lib.ozaki2_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, num_moduli, flags,
                         workspace, workspace.numel() * workspace.element_size(), stream)
    return C


def gemv(A, X, num_moduli=13, flags=0, Y=None, workspace=None, stream=None):
    """Y = A X for a column-major float64 A (m x k) and X (k x nrhs), nrhs <= 16,
    through the fused batched GEMV (fixed scaling); returns Y."""
    import torch
    if A.dim() != 2 or X.dim() != 2:
        raise ValueError("A and X must be matrices")
    m, k = A.shape
    k2, nrhs = X.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    dev = A.device
    items = [("A", A, (m, k)), ("X", X, (k, nrhs))] + ([("Y", Y, (m, nrhs))] if Y is not None else [])
    _check_matrices(dev, *items)
    if Y is None:
        Y = colmajor_empty(m, nrhs, device=dev)
    lda, ldx, ldy = _check_matrices(dev, ("A", A, (m, k)), ("X", X, (k, nrhs)), ("Y", Y, (m, nrhs)))
    need = _lib.ozaki2_gemv_workspace_bytes(m, k, nrhs, num_moduli)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    elif workspace.device != dev or workspace.numel() * workspace.element_size() < need:
        raise ValueError("workspace: too small or on another device")
    _lib.ozaki2_gemv_batched(m, k, nrhs, A, lda, X, ldx, Y, ldy, num_moduli, flags, workspace,
                             workspace.numel() * workspace.element_size(), stream)
    return Y


def words_to_ints(w):
    """uint32 [..., 5] little-endian two's complement words -> Python ints
    (object array of shape w.shape[:-1])."""
    w = np.asarray(w, dtype=np.uint64)
    out = np.zeros(w.shape[:-1], dtype=object)
    for q in range(w.shape[-1] - 1, -1, -1):
        out = out * (1 << 32) + w[..., q].astype(object)
    top = 1 << (32 * w.shape[-1])
    neg = np.frompyfunc(lambda v: v - top if v >> (32 * w.shape[-1] - 1) else v, 1, 1)
    return neg(out)


class Plan:
    """The staged API over one workspace: deconstruct, residue_gemm,
    reconstruct, and the diagnostic queries (as numpy arrays)."""

    def __init__(self, m, n, k, num_moduli=12, flags=0, device="cuda", workspace=None):
        """workspace: an existing uint8 device tensor to borrow (for instance
        another plan's, used on the same stream one after the other), else a
        new one of the size the plan needs."""
        import torch
        self.m, self.n, self.k, self.r, self.flags = m, n, k, num_moduli, flags
        self.device = torch.device(device)
        if self.device.type == "cuda" and self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.ws_bytes = _lib.ozaki2_workspace_bytes(m, n, k, num_moduli, flags)
        if workspace is None:
            workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        elif workspace.device != self.device or workspace.numel() < self.ws_bytes:
            raise ValueError("workspace: too small or on another device")
        self.workspace = workspace
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
        lda, ldb = _check_matrices(self.device, ("A", A, (self.m, self.k)),
                                   ("B", B, (self.k, self.n)))
        self._A, self._B = A, B      # borrowed by the plan until reconstruct
        _lib.ozaki2_deconstruct(self.handle, A, lda, B, ldb, stream)

    def deconstruct_a(self, A, stream=None):
        """Operand-stationary use (OZ2_SCALE_FIXED plans): new A, B's planes kept."""
        lda, = _check_matrices(self.device, ("A", A, (self.m, self.k)))
        self._A = A
        _lib.ozaki2_deconstruct_a(self.handle, A, lda, stream)

    def deconstruct_b(self, B, stream=None):
        """Operand-stationary use (OZ2_SCALE_FIXED plans): new B, A's planes kept."""
        ldb, = _check_matrices(self.device, ("B", B, (self.k, self.n)))
        self._B = B
        _lib.ozaki2_deconstruct_b(self.handle, B, ldb, stream)

    def residue_gemm(self, stream=None):
        _lib.ozaki2_residue_gemm(self.handle, stream)

    def reconstruct(self, C, stream=None):
        ldc, = _check_matrices(self.device, ("C", C, (self.m, self.n)))
        _lib.ozaki2_reconstruct(self.handle, C, ldc, stream)

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
            return words_to_ints(raw.view(np.uint32).reshape(n, m, 5)).T.copy()
        if what == _lib.OZ2_Q_FALLBACK_COUNT:
            v = raw.view(np.int32)
            return int(v[0]), int(v[1])
        if what == _lib.OZ2_Q_STAGE_TIMES:
            return dict(zip(_lib.STAGE_NAMES, (float(x) for x in raw.view(np.float32))))
        return raw
