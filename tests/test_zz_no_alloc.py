"""ozaki2_dgemm_static, the entry point for callers that cannot allocate:
its workspace is the library's static device array.  Through the C ABI, two
calls in a row (the second smaller, so the array still holds the first one's
contents) must give the results of the plain entry point ozaki2_dgemm bit for
bit (and the oracle's); a product whose workspace exceeds the array is
refused before any launch, leaving C untouched."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import bits, device

pytestmark = pytest.mark.gpu


def _run(entry, A, B, r):
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    m, k = A.shape
    n = B.shape[1]
    Ad, Bd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(B, dev)
    Cd = oz.to_device_colmajor(np.full((m, n), np.nan), dev)
    entry(m, n, k, Ad, m, Bd, k, Cd, m, r)
    torch.cuda.synchronize()
    return oz.from_device_colmajor(Cd)


@pytest.mark.parametrize("r", [12, 16])
def test_static_entry_point_matches_plain_two_calls(r):
    import paper_2606_06510_amd as oz
    cases = [((700, 650, 600), 61), ((190, 130, 100), 62)]   # the second smaller
    for (m, n, k), seed in cases:
        A, B = synth.lognormal(m, n, k, seed=seed)
        A = A.copy()
        A[3, ::2] *= 1e200                    # a fallback row: the panel is in the scratch too
        got = _run(oz.ozaki2_dgemm_static, A, B, r)
        want = _run(oz.ozaki2_dgemm, A, B, r)
        assert np.array_equal(bits(got), bits(want)), (m, n, k)
        res = oracle.dgemm(A, B, r)
        emu = ~np.isin(np.arange(m), res.fallback_rows)[:, None]
        assert np.array_equal(bits(got)[emu.repeat(n, 1)], bits(res.C)[emu.repeat(n, 1)])


def test_static_entry_point_refuses_oversized_products():
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    m = n = k = 1024                          # about 94 MiB of workspace at r = 12
    assert oz.ozaki2_workspace_bytes(m, n, k, 12) > oz.OZ2_STATIC_SCRATCH_BYTES
    Ad = oz.colmajor_empty(m, k, device=dev)
    Bd = oz.colmajor_empty(k, n, device=dev)
    Cd = oz.to_device_colmajor(np.full((m, n), 3.5), dev)
    with pytest.raises(oz.Ozaki2Error) as e:
        oz.ozaki2_dgemm_static(m, n, k, Ad, m, Bd, k, Cd, m, 12)
    assert e.value.status == oz.OZ2_E_WORKSPACE
    torch.cuda.synchronize()
    assert bool((Cd == 3.5).all())
