"""The tensor-level helpers refuse tensors whose shape, dtype, device or
storage does not match what the C ABI will be told, before any library call
(the ABI sees only pointers and sizes, so such a tensor would send the
kernels out of bounds; torch itself refuses views that run past their
storage).  Runs without a GPU: the library entry points are
replaced by functions that fail the test if reached."""
import numpy as np
import pytest
import torch

import paper_2606_06510_amd as oz
from paper_2606_06510_amd import _lib, tensor


@pytest.fixture
def no_library_calls(monkeypatch):
    def boom(*a, **k):
        raise AssertionError("a library entry point was reached")
    for name in ("ozaki2_dgemm_ex", "ozaki2_deconstruct", "ozaki2_deconstruct_a",
                 "ozaki2_deconstruct_b", "ozaki2_reconstruct"):
        monkeypatch.setattr(_lib, name, boom)


def _plan(m, n, k):
    p = object.__new__(oz.Plan)      # no workspace: nothing here reaches the device
    p.m, p.n, p.k, p.r, p.flags = m, n, k, 12, 0
    p.device = torch.device("cuda", 0)
    p.handle = None
    return p


def colmajor_cpu(m, n, dtype=torch.float64):
    return torch.zeros((n, m), dtype=dtype).t()


def test_plan_rejects_wrong_shapes(no_library_calls):
    p = _plan(8, 6, 5)
    with pytest.raises(ValueError, match="shape"):
        p.deconstruct(colmajor_cpu(8, 4), colmajor_cpu(5, 6))      # A is 8 x 4, not 8 x 5
    with pytest.raises(ValueError, match="shape"):
        p.deconstruct(colmajor_cpu(8, 5), colmajor_cpu(5, 7))      # B is 5 x 7, not 5 x 6
    with pytest.raises(ValueError, match="shape"):
        p.reconstruct(colmajor_cpu(7, 6))                          # C is 7 x 6, not 8 x 6
    with pytest.raises(ValueError, match="shape"):
        p.deconstruct_a(torch.zeros(40, dtype=torch.float64))
    with pytest.raises(ValueError, match="shape"):
        p.deconstruct_b(colmajor_cpu(6, 5))


def test_plan_rejects_wrong_dtype(no_library_calls):
    p = _plan(8, 6, 5)
    with pytest.raises(ValueError, match="dtype"):
        p.deconstruct(colmajor_cpu(8, 5, torch.float32), colmajor_cpu(5, 6))
    with pytest.raises(ValueError, match="dtype"):
        p.reconstruct(colmajor_cpu(8, 6, torch.float32))


def test_plan_rejects_host_tensors(no_library_calls):
    p = _plan(8, 6, 5)
    with pytest.raises(ValueError, match="expected a tensor on cuda:0"):
        p.deconstruct(colmajor_cpu(8, 5), colmajor_cpu(5, 6))
    with pytest.raises(ValueError, match="expected a tensor on cuda:0"):
        p.reconstruct(colmajor_cpu(8, 6))


def test_plan_rejects_row_major_views(no_library_calls):
    p = _plan(8, 6, 5)
    with pytest.raises(ValueError, match="column-major"):
        p.deconstruct(torch.zeros((8, 5), dtype=torch.float64), colmajor_cpu(5, 6))


def test_matmul_checks_before_the_library(no_library_calls):
    with pytest.raises(ValueError, match="inner dimensions"):
        oz.matmul(colmajor_cpu(4, 3), colmajor_cpu(2, 5))
    with pytest.raises(ValueError, match="dtype"):
        oz.matmul(colmajor_cpu(4, 3, torch.float32), colmajor_cpu(3, 5))
    with pytest.raises(ValueError, match="expected a tensor on a CUDA device"):
        oz.matmul(colmajor_cpu(4, 3), colmajor_cpu(3, 5))
    with pytest.raises(ValueError, match="shape"):
        oz.matmul(colmajor_cpu(4, 3), colmajor_cpu(3, 5), C=colmajor_cpu(5, 4))


def test_words_to_ints_roundtrip():
    rng = np.random.default_rng(3)
    vals = [0, 1, -1, (1 << 159) - 1, -(1 << 159), 123456789 << 70, -(987654321 << 90)]
    vals += [int(x) for x in rng.integers(-2 ** 62, 2 ** 62, 20)]
    w = np.array([[(v >> (32 * q)) & 0xFFFFFFFF for q in range(5)] for v in vals], dtype=np.uint32)
    back = oz.words_to_ints(w)
    assert [int(x) for x in back] == vals


def test_leading_dimension_of_single_columns_and_rows():
    """numpy and torch normalise the stride of a size-1 dimension (a single
    column made by to_device_colmajor has strides (1, 1)): the leading
    dimension handed to the C ABI is then max(m, 1), never below m."""
    for m, n in [(70, 1), (1, 70), (1, 1), (5, 3)]:
        X = np.asfortranarray(np.arange(m * n, dtype=np.float64).reshape(m, n))
        T = oz.to_device_colmajor(X, "cpu")
        assert tensor._ld(T) >= max(m, 1)
        assert tensor._ld(T) == (max(m, 1) if n == 1 else T.stride(1))
        assert np.array_equal(oz.from_device_colmajor(T), X)
    with pytest.raises(ValueError):
        tensor._ld(torch.zeros(4, 3))                 # row-major (stride (3, 1))
