"""ctypes binding of libozaki2.so (include/ozaki2.h).

Argument marshalling only: every step of the emulated GEMM runs in the
library's gfx950 kernels.  Device pointers may be given as integers or as
torch tensors (their data_ptr is used); ``stream`` is a hipStream_t handle
(an int, a torch.cuda.Stream, or None for torch's current stream).  Error
codes become ``Ozaki2Error``.  There is no fallback: if the library is not
built, importing the functions raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libozaki2.so")

OZ2_OK = 0
OZ2_E_INVALID = -1
OZ2_E_NOMEM = -2
OZ2_E_DEVICE = -3
OZ2_E_UNSUPPORTED = -4
OZ2_E_WORKSPACE = -5

OZ2_ACCUMULATE = 1
OZ2_SCALE_FIXED = 2
OZ2_QUANT_TZ = 4
OZ2_NO_FALLBACK = 8
OZ2_FORCE_FALLBACK = 16
OZ2_KEEP_RESIDUES = 32
OZ2_TIME_STAGES = 64
OZ2_FUSED = 128
OZ2_REUSE_A_SCALES = 256

OZ2_Q_EXPONENTS = 1
OZ2_Q_MAXIMA = 2
OZ2_Q_SCALES = 3
OZ2_Q_FLAGS = 4
OZ2_Q_CODES = 5
OZ2_Q_PLANES = 6
OZ2_Q_RESIDUES = 7
OZ2_Q_INTEGERS = 8
OZ2_Q_FALLBACK_COUNT = 9
OZ2_Q_STAGE_TIMES = 10

# the six stages OZ2_Q_STAGE_TIMES reports, in its order
STAGE_NAMES = ["scan_codes", "maxmag_gemm", "split", "residue_gemm", "reconstruct", "fallback"]

EXPORTS = [
    "ozaki2_dgemm", "ozaki2_dgemm_ex", "ozaki2_dgemm_static", "ozaki2_dgemm_strided_batched",
    "ozaki2_workspace_bytes", "ozaki2_moduli", "ozaki2_plan_create",
    "ozaki2_plan_destroy", "ozaki2_deconstruct", "ozaki2_deconstruct_a", "ozaki2_deconstruct_b",
    "ozaki2_residue_gemm",
    "ozaki2_reconstruct", "ozaki2_plan_query_bytes", "ozaki2_plan_query",
    "ozaki2_status_string", "ozaki2_finalize", "ozaki2_gemv_batched", "ozaki2_gemv_workspace_bytes",
]

# include/ozaki2_probes.h
PROBE_EXPORTS = [
    "ozaki2_probe_e4m3", "ozaki2_probe_accum", "ozaki2_probe_copy", "ozaki2_probe_mfma_peak",
    "ozaki2_probe_mfma_digits", "ozaki2_probe_copy_peak", "ozaki2_probe_crt",
    "ozaki2_probe_batched_integers",
]


class Ozaki2Error(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {status} ({_status_string(status)})")


_lib = None


def load():
    """Load the shared library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(python paper_2606_06510_amd/build.py)")
    # torch first: its HIP runtime is then the one the library's
    # libamdhip64.so.7 dependency resolves to, so device pointers and streams
    # from torch and the library's launches share one runtime whatever the
    # caller imported first
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    i, u, p, sz, ll = ctypes.c_int, ctypes.c_uint, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_longlong
    sig = {
        "ozaki2_dgemm": (i, [i, i, i, p, i, p, i, p, i, i, p]),
        "ozaki2_dgemm_ex": (i, [i, i, i, p, i, p, i, p, i, i, u, p, sz, p]),
        "ozaki2_dgemm_static": (i, [i, i, i, p, i, p, i, p, i, i, p]),
        "ozaki2_dgemm_strided_batched": (i, [i, i, i, p, i, ll, p, i, ll, p, i, ll, i, i, p]),
        "ozaki2_workspace_bytes": (sz, [i, i, i, i, u]),
        "ozaki2_moduli": (i, [i, ctypes.POINTER(ctypes.c_int)]),
        "ozaki2_plan_create": (i, [ctypes.POINTER(p), i, i, i, i, u, p, sz]),
        "ozaki2_plan_destroy": (i, [p]),
        "ozaki2_deconstruct": (i, [p, p, i, p, i, p]),
        "ozaki2_deconstruct_a": (i, [p, p, i, p]),
        "ozaki2_deconstruct_b": (i, [p, p, i, p]),
        "ozaki2_residue_gemm": (i, [p, p]),
        "ozaki2_reconstruct": (i, [p, p, i, p]),
        "ozaki2_plan_query_bytes": (sz, [p, i]),
        "ozaki2_plan_query": (i, [p, i, p, sz]),
        "ozaki2_status_string": (ctypes.c_char_p, [i]),
        "ozaki2_finalize": (None, []),
        "ozaki2_gemv_batched": (i, [i, i, i, p, i, p, i, p, i, i, u, p, sz, p]),
        "ozaki2_gemv_workspace_bytes": (sz, [i, i, i, i]),
        "ozaki2_probe_e4m3": (i, [p, p, i, p]),
        "ozaki2_probe_accum": (i, [p, p, i, p, p]),
        "ozaki2_probe_copy": (i, [p, p, sz, p]),
        "ozaki2_probe_mfma_peak": (i, [i, ctypes.POINTER(ctypes.c_double)]),
        "ozaki2_probe_mfma_digits": (i, [i, ctypes.POINTER(ctypes.c_double)]),
        "ozaki2_probe_copy_peak": (i, [sz, i, ctypes.POINTER(ctypes.c_double)]),
        "ozaki2_probe_crt": (i, [i, p, p, i, p, p, p]),
        "ozaki2_probe_batched_integers": (i, [i, i, i, p, i, ll, p, i, ll, i, i, p, p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _status_string(st):
    try:
        return load().ozaki2_status_string(st).decode()
    except Exception:  # pragma: no cover - only used inside error messages
        return "?"


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, ctypes.c_void_p):
        return x.value
    raise TypeError(f"cannot take a device pointer of {type(x)}")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(fn, st):
    if st != OZ2_OK:
        raise Ozaki2Error(fn, st)
    return st


# ------------------------------------------------------------ C ABI, same names

def ozaki2_dgemm(m, n, k, A, lda, B, ldb, C, ldc, num_moduli, stream=None):
    return _check("ozaki2_dgemm", load().ozaki2_dgemm(
        m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, num_moduli, _stream(stream)))


def ozaki2_dgemm_ex(m, n, k, A, lda, B, ldb, C, ldc, num_moduli, flags, workspace, ws_bytes,
                    stream=None):
    return _check("ozaki2_dgemm_ex", load().ozaki2_dgemm_ex(
        m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, num_moduli, flags, _ptr(workspace),
        ws_bytes, _stream(stream)))


OZ2_STATIC_SCRATCH_BYTES = 64 << 20


def ozaki2_dgemm_static(m, n, k, A, lda, B, ldb, C, ldc, num_moduli, stream=None):
    return _check("ozaki2_dgemm_static", load().ozaki2_dgemm_static(
        m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, num_moduli, _stream(stream)))


def ozaki2_dgemm_strided_batched(m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC,
                                 batch, num_moduli, stream=None):
    return _check("ozaki2_dgemm_strided_batched", load().ozaki2_dgemm_strided_batched(
        m, n, k, _ptr(A), lda, strideA, _ptr(B), ldb, strideB, _ptr(C), ldc, strideC, batch,
        num_moduli, _stream(stream)))


def ozaki2_workspace_bytes(m, n, k, num_moduli, flags=0):
    return load().ozaki2_workspace_bytes(m, n, k, num_moduli, flags)


def ozaki2_gemv_batched(m, k, nrhs, A, lda, X, ldx, Y, ldy, num_moduli, flags, workspace,
                        ws_bytes, stream=None):
    return _check("ozaki2_gemv_batched", load().ozaki2_gemv_batched(
        m, k, nrhs, _ptr(A), lda, _ptr(X), ldx, _ptr(Y), ldy, num_moduli, flags, _ptr(workspace),
        ws_bytes, _stream(stream)))


def ozaki2_gemv_workspace_bytes(m, k, nrhs, num_moduli):
    return load().ozaki2_gemv_workspace_bytes(m, k, nrhs, num_moduli)


def ozaki2_moduli(num_moduli):
    out = (ctypes.c_int * max(num_moduli, 1))()
    _check("ozaki2_moduli", load().ozaki2_moduli(num_moduli, out))
    return list(out)[:num_moduli]


def ozaki2_plan_create(m, n, k, num_moduli, flags, workspace, ws_bytes):
    h = ctypes.c_void_p()
    _check("ozaki2_plan_create", load().ozaki2_plan_create(
        ctypes.byref(h), m, n, k, num_moduli, flags, _ptr(workspace), ws_bytes))
    return h


def ozaki2_plan_destroy(plan):
    return _check("ozaki2_plan_destroy", load().ozaki2_plan_destroy(plan))


def ozaki2_deconstruct(plan, A, lda, B, ldb, stream=None):
    return _check("ozaki2_deconstruct", load().ozaki2_deconstruct(
        plan, _ptr(A), lda, _ptr(B), ldb, _stream(stream)))


def ozaki2_deconstruct_a(plan, A, lda, stream=None):
    return _check("ozaki2_deconstruct_a", load().ozaki2_deconstruct_a(plan, _ptr(A), lda,
                                                                      _stream(stream)))


def ozaki2_deconstruct_b(plan, B, ldb, stream=None):
    return _check("ozaki2_deconstruct_b", load().ozaki2_deconstruct_b(plan, _ptr(B), ldb,
                                                                      _stream(stream)))


def ozaki2_residue_gemm(plan, stream=None):
    return _check("ozaki2_residue_gemm", load().ozaki2_residue_gemm(plan, _stream(stream)))


def ozaki2_reconstruct(plan, C, ldc, stream=None):
    return _check("ozaki2_reconstruct", load().ozaki2_reconstruct(plan, _ptr(C), ldc,
                                                                  _stream(stream)))


def ozaki2_plan_query_bytes(plan, what):
    return load().ozaki2_plan_query_bytes(plan, what)


def ozaki2_plan_query(plan, what, out):
    """Copy a plan quantity into the writable host buffer ``out`` (a numpy
    array or bytearray)."""
    import numpy as np
    arr = np.asarray(out) if not isinstance(out, bytearray) else out
    if isinstance(arr, np.ndarray):
        ptr, nbytes = arr.ctypes.data, arr.nbytes
    else:
        buf = (ctypes.c_char * len(arr)).from_buffer(arr)
        ptr, nbytes = ctypes.addressof(buf), len(arr)
    return _check("ozaki2_plan_query", load().ozaki2_plan_query(plan, what, ptr, nbytes))


def ozaki2_status_string(status):
    return load().ozaki2_status_string(status).decode()


def ozaki2_finalize():
    load().ozaki2_finalize()


# ------------------------------------------------------------ probes (ozaki2_probes.h)

def ozaki2_probe_e4m3(x, out, n, stream=None):
    return _check("ozaki2_probe_e4m3", load().ozaki2_probe_e4m3(_ptr(x), _ptr(out), n,
                                                                _stream(stream)))


def ozaki2_probe_accum(a, b, chain, out, stream=None):
    return _check("ozaki2_probe_accum", load().ozaki2_probe_accum(_ptr(a), _ptr(b), chain,
                                                                  _ptr(out), _stream(stream)))


def ozaki2_probe_copy(src, dst, nbytes, stream=None):
    return _check("ozaki2_probe_copy", load().ozaki2_probe_copy(_ptr(src), _ptr(dst), nbytes,
                                                                _stream(stream)))


def ozaki2_probe_mfma_peak(iters):
    """Measured dense FP8 MFMA TFLOP/s (synchronous)."""
    v = ctypes.c_double(0.0)
    _check("ozaki2_probe_mfma_peak", load().ozaki2_probe_mfma_peak(iters, ctypes.byref(v)))
    return v.value


def ozaki2_probe_mfma_digits(iters):
    """Sustained FP8 MFMA TFLOP/s of the residue GEMM's inner loop on
    plane-like digit operands read from LDS (synchronous)."""
    v = ctypes.c_double(0.0)
    _check("ozaki2_probe_mfma_digits", load().ozaki2_probe_mfma_digits(iters, ctypes.byref(v)))
    return v.value


def ozaki2_probe_copy_peak(nbytes, reps):
    """Measured HBM copy GB/s, read + write bytes (synchronous)."""
    v = ctypes.c_double(0.0)
    _check("ozaki2_probe_copy_peak", load().ozaki2_probe_copy_peak(nbytes, reps, ctypes.byref(v)))
    return v.value


def ozaki2_probe_crt(num_moduli, residues, shifts, n, words, rounded, stream=None):
    return _check("ozaki2_probe_crt", load().ozaki2_probe_crt(
        num_moduli, _ptr(residues), _ptr(shifts), n, _ptr(words), _ptr(rounded), _stream(stream)))


def ozaki2_probe_batched_integers(m, n, k, A, lda, strideA, B, ldb, strideB, batch, num_moduli,
                                  words, stream=None):
    return _check("ozaki2_probe_batched_integers", load().ozaki2_probe_batched_integers(
        m, n, k, _ptr(A), lda, strideA, _ptr(B), ldb, strideB, batch, num_moduli, _ptr(words),
        _stream(stream)))
