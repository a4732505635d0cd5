"""CPU oracle for the Ozaki-II (CRT) FP64 GEMM emulated on FP8.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import
it.  The product path (``paper_2606_06510_amd``) never imports, calls or
links anything here, and this package imports nothing from it.

It is a plain, slow, obviously correct transcription of what the method
computes, written from the paper (Matsuoka, "FP8 is All You Need (Part 1)",
arXiv 2606.06510): Algorithm 1 (Ozaki II dense GEMM at phase level), the
scaling of Eq. (scale), the range condition Eq. (M-bound), the modular GEMMs of
Eq. (modgemm), Garner's reconstruction Eq. (garner) / App. A, and the FP8 plane
algebra of the section "The frozen plane kernel" (Eq. (sq-shortcut),
Eq. (kar), Eq. (envelope), Eq. (accum-exact)).  Floating point is fp64;
integers are numpy int64 where they provably fit and Python ints otherwise.

Every reading taken where the paper is silent is marked READING in the
docstring that uses it.

Parity status: every function is pinned by ``tests/test_oracle_*.py`` except
the native-FP64 fallback values, whose summation order the paper leaves to the
hardware (parity unpinned: checked against the FP64 dot-product error bound,
with NaN/Inf classes checked exactly).
"""
from . import moduli, e4m3, planes, garner, ozaki2, refgemm  # noqa: F401
from .ozaki2 import dgemm, Result  # noqa: F401
