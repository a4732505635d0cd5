"""FP64 GEMM emulated on MI355X (gfx950) FP8 matrix cores via the CRT-based
Ozaki Scheme II.  The compute path is the hand-written HIP library
``libozaki2.so`` (C ABI: include/ozaki2.h); this package is its binding plus
small tensor-level helpers.  PyTorch is used only for device memory and
streams."""
from ._lib import *  # noqa: F401,F403
from ._lib import load, Ozaki2Error, LIB_PATH  # noqa: F401
from .tensor import (colmajor_empty, to_device_colmajor, from_device_colmajor,  # noqa: F401
                     matmul, gemv, Plan, words_to_ints)
