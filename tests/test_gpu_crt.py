"""The reconstruction's exact integers, checked on the routines the product
path runs (GPU):

* the CRT probe feeds the reconstruction's own device routines with
  residues of crafted integers -- next to +-M/2, where the quotient estimate
  is ambiguous and the exact range check decides, at the ends of the range,
  zero and random values -- given as centred residues and as other
  representatives of magnitude <= m/2 + 32 (what the residue GEMMs hand
  over); the integers must equal the oracle's Garner reconstruction
  (Eq. (garner)) and the rounded values its correctly rounded quotient;
* the single-launch batched kernel, in its integer-writing instantiation,
  must form the oracle's integers for every unflagged output;
* a plan created with OZ2_TIME_STAGES reports six stage times and its
  results stay bit-exact."""
import numpy as np
import pytest

import oracle
import synth
from oracle import garner, moduli
from tests.gpu_util import bits, device

pytestmark = pytest.mark.gpu


def _crafted(r, rng):
    ms = moduli.moduli(r)
    M = moduli.modulus_product(ms)
    lo, hi = -(M // 2), (M + 1) // 2 - 1          # the symmetric range [-M/2, M/2)
    X = [0, 1, -1, lo, hi, lo + 1, hi - 1]
    for d in range(1, 40):                        # next to +-M/2
        X += [hi - d * 997, lo + d * 991]
    for t in range(1, 30):                        # quotient estimates next to a half
        X += [hi - (t << 40), lo + (t << 37), hi - rng.integers(0, 1 << 60).item()]
    X += [int(v) for v in rng.integers(-2 ** 62, 2 ** 62, 100)]
    X += [int(rng.integers(0, 1 << 62)) * int(rng.integers(0, 1 << 50)) % M - M // 2
          for _ in range(200)]
    return ms, M, [int(x) for x in X]


def _residues(X, ms, rng, shift):
    """int16 [r][n]: centred residues, shifted by a multiple of m where the
    result stays within m/2 + 32 (shift = 0: centred)."""
    out = np.zeros((len(ms), len(X)), dtype=np.int16)
    for i, m in enumerate(ms):
        for t, x in enumerate(X):
            v = x % m
            v = v - m if v >= (m + 1) // 2 else v
            if shift and rng.random() < 0.5:
                w = v + m if v < 0 else v - m
                if abs(w) <= m // 2 + 32:
                    v = w
            out[i, t] = v
    return out


@pytest.mark.parametrize("r", range(8, 17))
@pytest.mark.parametrize("shift", [0, 1])
def test_crt_probe_crafted_integers(r, shift):
    import torch
    import paper_2606_06510_amd as oz
    rng = np.random.default_rng(100 * r + shift)
    ms, M, X = _crafted(r, rng)
    res = _residues(X, ms, rng, shift)
    n = len(X)
    e = rng.integers(-200, 400, n).astype(np.int32)
    e[:20] = 0
    e[20:40] = 1100                               # subnormal and zero results
    e[40:60] = -900                               # overflow to infinity
    dev = device()
    rd = torch.from_numpy(res).to(dev)
    ed = torch.from_numpy(e).to(dev)
    wd = torch.zeros((n, 5), dtype=torch.int32, device=dev)
    vd = torch.zeros(n, dtype=torch.float64, device=dev)
    oz.ozaki2_probe_crt(r, rd, ed, n, wd, vd)
    torch.cuda.synchronize()
    got = oz.words_to_ints(wd.cpu().numpy().view(np.uint32))
    want = garner.crt(res.astype(np.int64), ms)      # Garner, independent of the GPU's CRT sum
    assert [int(v) for v in want] == X               # the crafted residues are right
    assert [int(v) for v in got] == X
    vals = vd.cpu().numpy()
    ref = np.array([garner.round_scaled(x, int(s)) for x, s in zip(X, e)])
    assert np.array_equal(bits(vals), bits(ref))


@pytest.mark.parametrize("r", [8, 12, 15])
def test_batched_kernel_integers(r):
    import torch
    import paper_2606_06510_amd as oz
    nb, m, n, k = 5, 64, 48, 64
    Ab, Bb = synth.batched(nb, m, n, k, seed=200 + r)
    Ab = Ab.copy()
    Ab[1, 3, 5] = np.nan                               # a flagged row: left untouched
    dev = device()
    Ad = torch.from_numpy(np.ascontiguousarray(Ab.transpose(0, 2, 1))).to(dev)
    Bd = torch.from_numpy(np.ascontiguousarray(Bb.transpose(0, 2, 1))).to(dev)
    W = torch.zeros((nb, n, m, 5), dtype=torch.int32, device=dev)
    oz.ozaki2_probe_batched_integers(m, n, k, Ad, m, m * k, Bd, k, k * n, nb, r, W)
    torch.cuda.synchronize()
    got = oz.words_to_ints(W.cpu().numpy().view(np.uint32))   # [nb][n][m]
    for b in range(nb):
        res = oracle.dgemm(Ab[b], Bb[b], r)
        fr = set(res.fallback_rows.tolist())
        for j in range(n):
            for i in range(m):
                if i in fr or j in set(res.fallback_cols.tolist()):
                    assert int(got[b, j, i]) == 0
                else:
                    assert int(got[b, j, i]) == int(res.X[i, j]), (b, i, j)


def test_stage_times_query():
    import paper_2606_06510_amd as oz
    import torch
    A, B = synth.lognormal(700, 600, 900, seed=31)
    A = A.copy()
    A[7, ::2] *= 1e200                                 # one fallback row
    dev = device()
    Ad, Bd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(B, dev)
    Cd = oz.colmajor_empty(700, 600, device=dev)
    plan = oz.Plan(700, 600, 900, 12, oz.OZ2_TIME_STAGES, device=dev)
    plan.deconstruct(Ad, Bd)
    with pytest.raises(oz.Ozaki2Error):                # stages 2 and 3 not run yet
        plan.query(oz.OZ2_Q_STAGE_TIMES)
    plan.residue_gemm()
    plan.reconstruct(Cd)
    t = plan.query(oz.OZ2_Q_STAGE_TIMES)
    assert list(t) == oz.STAGE_NAMES
    assert all(v >= 0 for v in t.values()) and t["residue_gemm"] > 0
    res = oracle.dgemm(A, B, 12)
    from tests.gpu_util import compare_C
    compare_C(oz.from_device_colmajor(Cd), A, B, res)
    untimed = oz.Plan(10, 10, 10, 12, 0, device=dev)
    with pytest.raises(oz.Ozaki2Error):
        untimed.query(oz.OZ2_Q_STAGE_TIMES)
    del plan, untimed
    torch.cuda.synchronize()
