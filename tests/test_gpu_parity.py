"""GPU parity: the HIP path through the C ABI against the CPU oracle, element
by element on seeded inputs.  Integer stages (exponents, code-product maxima,
scales, flags, code and plane bytes, residues, reconstructed integers) must be
bit-exact; emulated C entries are bit-exact too (both sides round the same
exact rational once); native-FP64 fallback entries are within the FP64
dot-product error bound (their summation order is the hardware's)."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import compare_all, compare_C, run_staged, bits, device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [(1, 1, 1), (17, 33, 129), (256, 256, 256), (300, 520, 700),
                                   (513, 129, 257), (64, 700, 5)])
def test_stage_parity_shapes(shape):
    m, n, k = shape
    A, B = synth.lognormal(m, n, k, seed=m + n + k)
    res = oracle.dgemm(A, B, 12)
    plan, C = run_staged(A, B, 12)
    compare_all(plan, C, A, B, 12, res, check_integers=m * n <= 70000)


@pytest.mark.parametrize("r", range(8, 17))
def test_moduli_sweep(r):
    A, B = synth.lognormal(160, 200, 300, seed=100 + r)
    res = oracle.dgemm(A, B, r)
    plan, C = run_staged(A, B, r)
    compare_all(plan, C, A, B, r, res, check_integers=True)


def test_gemm256_uniform_full():
    A, B = synth.make("gemm256_uniform")
    res = oracle.dgemm(A, B, 12)
    plan, C = run_staged(A, B, 12)
    compare_all(plan, C, A, B, 12, res)


@pytest.mark.parametrize("flags,mode,quant", [(2, "fixed", "rn"), (4, "bound", "tz"),
                                              (6, "fixed", "tz")])
def test_modes(flags, mode, quant):
    A, B = synth.wide(200, 150, 333, seed=7, spread=1.0, frac=0.0)[:2]
    res = oracle.dgemm(A, B, 12, mode=mode, quant=quant)
    plan, C = run_staged(A, B, 12, flags=flags)
    compare_all(plan, C, A, B, 12, res, check_integers=False)


def test_accumulate():
    A, B, Cin = synth.rankk(300, 260, 256, seed=4)
    res = oracle.dgemm(A, B, 12, C_in=Cin)
    plan, C = run_staged(A, B, 12, flags=1, C_in=Cin)
    compare_C(C, A, B, res)


def test_fallback_rows_and_columns():
    rng = np.random.default_rng(9)
    A, B = synth.uniform(260, 270, 300, seed=9)
    A[3, 7] = np.nan
    A[100, 5] = np.inf
    B[11, 200] = -np.inf
    A[50, ::2] *= 1e200                       # T2: intra-row span ~2^664
    B[::3, 20] *= 1e-250                      # T2 on a column of B
    res = oracle.dgemm(A, B, 12)
    assert set(res.fallback_rows) == {3, 50, 100} and set(res.fallback_cols) == {20, 200}
    plan, C = run_staged(A, B, 12)
    compare_all(plan, C, A, B, 12, res, check_integers=False)
    import paper_2606_06510_amd as oz
    assert plan.query(oz.OZ2_Q_FALLBACK_COUNT) == (3, 2)


def test_code_bytes_edge_cases():
    """The max-magnitude codes are built per 64-wide k-block (a byte relative to
    the block's own exponent) and rebased to the row's: rows whose blocks sit
    0..6 binary orders below the row maximum, exact powers of two and
    mantissas with and without bits below the fourth, subnormal rows and
    entries, a NaN row; codes, scales and C are compared with the oracle."""
    rng = np.random.default_rng(23)
    m, n, k = 70, 66, 450                      # 8 k-blocks, the last ragged
    A, B = synth.uniform(m, n, k, seed=23)
    A, B = A.copy(), B.copy()
    for b in range(8):                         # row 0: block b lies b orders down
        A[0, 64 * b:64 * (b + 1)] *= 2.0 ** -b
    A[1] = 2.0 ** rng.integers(-30, 3, k)      # exact powers of two (sticky 0)
    A[2] = (8 + rng.integers(0, 8, k)) / 16.0 * 2.0 ** rng.integers(-6, 6, k)   # 4-bit mantissas
    A[2, ::3] *= 1.0 + 2.0 ** -40              # and some with low bits set
    A[3] = rng.integers(1, 2 ** 40, k) * 2.0 ** -1074      # a subnormal row
    A[4, ::5] = rng.integers(1, 2 ** 20, (k + 4) // 5) * 2.0 ** -1074   # subnormals in a normal row
    A[5, 10] = np.nan                          # T1 row: codes 0
    A[6] = 0.0                                 # zero row
    A[7, 300:] *= 2.0 ** 9                     # row maximum in a late block
    for b in range(8):                         # column 0 of B: block b lies 2b orders down
        B[64 * b:64 * (b + 1), 0] *= 2.0 ** (-2 * b)
    B[:, 1] = 2.0 ** rng.integers(-10, 10, k)
    B[:, 2] = rng.integers(1, 2 ** 30, k) * 2.0 ** -1074   # a subnormal column
    res = oracle.dgemm(A, B, 12)
    plan, C = run_staged(A, B, 12)
    compare_all(plan, C, A, B, 12, res, check_integers=False)


def test_whole_rows_1e200_absorbed():
    A, B, rows = synth.wide(300, 200, 256, seed=3)
    assert len(rows) > 0
    res = oracle.dgemm(A, B, 15)
    assert len(res.fallback_rows) == 0
    plan, C = run_staged(A, B, 15)
    compare_all(plan, C, A, B, 15, res, check_integers=False)


def test_no_fallback_and_force_fallback():
    A, B = synth.uniform(100, 90, 80, seed=5)
    A[2, ::2] *= 1e200
    res = oracle.dgemm(A, B, 12, fallback=False)
    plan, C = run_staged(A, B, 12, flags=8)
    assert np.array_equal(bits(C), bits(res.C))
    res2 = oracle.dgemm(A, B, 12, force_fallback=True)
    plan2, C2 = run_staged(A, B, 12, flags=16)
    compare_C(C2, A, B, res2)


def test_force_fallback_beyond_the_panel():
    """All 1300 rows flagged (and two columns of B by their values): the
    fallback reads the first 1024 listed rows of A from the panel the
    reconstruction gathered and the rest straight from A; every entry within
    the FP64 dot-product bound."""
    A, B = synth.uniform(1300, 150, 120, seed=15)
    B = B.copy()
    B[::2, 7] *= 1e-250                       # T2 on two columns of B
    B[::3, 90] *= 1e250
    res = oracle.dgemm(A, B, 12, force_fallback=True)
    assert len(res.fallback_rows) == 1300
    plan, C = run_staged(A, B, 12, flags=16)
    compare_C(C, A, B, res)


def test_multi_slab_k():
    """k above the 32768 residue slab and the 65536 code slab."""
    A, B = synth.uniform(40, 48, 70000, seed=12)
    res = oracle.dgemm(A, B, 12)
    plan, C = run_staged(A, B, 12)
    compare_all(plan, C, A, B, 12, res, check_integers=True)


def test_zero_rows_columns_and_k0():
    import paper_2606_06510_amd as oz
    import torch
    A, B = synth.uniform(70, 60, 50, seed=1)
    A[5] = 0.0
    B[:, 9] = 0.0
    res = oracle.dgemm(A, B, 12)
    plan, C = run_staged(A, B, 12)
    compare_all(plan, C, A, B, 12, res)
    assert not np.any(np.signbit(C[5])) and np.all(C[5] == 0)
    # k = 0: C = 0; with ACCUMULATE, C unchanged
    dev = device()
    Ad = oz.colmajor_empty(4, 0, device=dev)
    Bd = oz.colmajor_empty(0, 3, device=dev)
    Cd = oz.to_device_colmajor(np.full((4, 3), 7.0), dev)
    oz.ozaki2_dgemm(4, 3, 0, Ad, 4, Bd, 1, Cd, 4, 12)
    torch.cuda.synchronize()
    assert np.all(oz.from_device_colmajor(Cd) == 0.0)


def test_plain_entry_point_and_batched():
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    A, B = synth.lognormal(200, 100, 150, seed=21)
    Ad, Bd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(B, dev)
    Cd = oz.colmajor_empty(200, 100, device=dev)
    oz.ozaki2_dgemm(200, 100, 150, Ad, 200, Bd, 150, Cd, 200, 12)
    torch.cuda.synchronize()
    res = oracle.dgemm(A, B, 12)
    assert np.array_equal(bits(oz.from_device_colmajor(Cd)), bits(res.C))
    # strided batched: 5 problems of 64^3 with per-matrix scales
    Ab, Bb = synth.batched(5, 64, 64, 64, seed=5)
    Ad = torch.from_numpy(np.ascontiguousarray(Ab.transpose(0, 2, 1))).to(dev)
    Bd = torch.from_numpy(np.ascontiguousarray(Bb.transpose(0, 2, 1))).to(dev)
    Cd = torch.empty((5, 64, 64), dtype=torch.float64, device=dev)
    oz.ozaki2_dgemm_strided_batched(64, 64, 64, Ad, 64, 64 * 64, Bd, 64, 64 * 64, Cd, 64, 64 * 64,
                                    5, 12)
    torch.cuda.synchronize()
    Cb = Cd.cpu().numpy().transpose(0, 2, 1)
    for b in range(5):
        rb = oracle.dgemm(Ab[b], Bb[b], 12)
        assert np.array_equal(bits(Cb[b]), bits(rb.C))


@pytest.mark.parametrize("shape", [(100, 80, 70), (48, 40, 200)])
def test_strided_batched_beyond_the_single_launch(shape):
    """Strided-batched products larger than 64 in some dimension take the
    staged path once per problem on the internal workspace; each bit-exact."""
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    m, n, k = shape
    nb = 3
    Ab, Bb = synth.batched(nb, m, n, k, seed=m + n + k)
    Ad = torch.from_numpy(np.ascontiguousarray(Ab.transpose(0, 2, 1))).to(dev)
    Bd = torch.from_numpy(np.ascontiguousarray(Bb.transpose(0, 2, 1))).to(dev)
    Cd = torch.full((nb, n, m), float("nan"), dtype=torch.float64, device=dev)
    oz.ozaki2_dgemm_strided_batched(m, n, k, Ad, m, m * k, Bd, k, k * n, Cd, m, m * n, nb, 12)
    torch.cuda.synchronize()
    Cb = Cd.cpu().numpy().transpose(0, 2, 1)
    for b in range(nb):
        assert np.array_equal(bits(Cb[b]), bits(oracle.dgemm(Ab[b], Bb[b], 12).C)), b


def test_plain_entry_point_from_two_threads():
    """Two host threads issue plain ozaki2_dgemm calls on one stream while the
    library's internal workspace grows under them (each thread's calls get
    larger).  A thread holds the workspace from lookup to enqueue, and a grow
    synchronises before it frees, so no call's kernels run on a buffer that
    another thread's grow released; every product is bit-exact."""
    import threading
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    torch.cuda.synchronize()
    oz.ozaki2_finalize()                      # start from an empty workspace
    stream = torch.cuda.current_stream().cuda_stream
    shapes = [[(96, 80, 64), (200, 150, 260), (330, 270, 520), (420, 390, 700)],
              [(64, 72, 90), (180, 210, 300), (300, 330, 610), (450, 400, 640)]]
    jobs = []
    for t, lst in enumerate(shapes):
        row = []
        for i, (m, n, k) in enumerate(lst):
            A, B = synth.lognormal(m, n, k, seed=500 + 10 * t + i)
            row.append((A, B, oz.to_device_colmajor(A, dev), oz.to_device_colmajor(B, dev),
                        oz.colmajor_empty(m, n, device=dev)))
        jobs.append(row)
    torch.cuda.synchronize()
    errors = []

    def work(row):
        try:
            for A, B, Ad, Bd, Cd in row:
                m, k = A.shape
                n = B.shape[1]
                oz.ozaki2_dgemm(m, n, k, Ad, m, Bd, k, Cd, m, 12, stream)
        except Exception as e:               # reported after the join
            errors.append(e)

    threads = [threading.Thread(target=work, args=(row,)) for row in jobs]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for row in jobs:
        for A, B, Ad, Bd, Cd in row:
            res = oracle.dgemm(A, B, 12)
            assert np.array_equal(bits(oz.from_device_colmajor(Cd)), bits(res.C)), A.shape


def _padded(X, ld, off, dev, fill=float("nan")):
    """Column-major device view of X (m x n) with leading dimension ld, its
    first element `off` doubles into a buffer whose other entries hold fill."""
    import torch
    m, n = X.shape
    buf = torch.full((off + ld * n,), fill, dtype=torch.float64, device=dev)
    view = buf[off:].view(n, ld)[:, :m].t()
    view.copy_(torch.from_numpy(np.ascontiguousarray(X)).to(dev))
    return buf, view


@pytest.mark.parametrize("pad,off", [((2, 6, 4), 0), ((1, 3, 5), 1), ((64, 0, 0), 2)])
def test_padded_leading_dimensions(pad, off):
    """Leading dimensions above the row counts (even, odd) and base addresses
    that are not 16-byte aligned, through the staged plan, the workspace entry
    point with accumulation and the plain one: products bit-exact, padding of
    A and B (NaN, which would flag any row that read it) never used, padding
    of C untouched."""
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    m, n, k = 300, 260, 200
    A, B = synth.lognormal(m, n, k, seed=60 + off)
    C0 = synth.lognormal(m, n, 1, seed=70 + off)[0][:, :1] * np.ones((1, n))
    lda, ldb, ldc = m + pad[0], k + pad[1], m + pad[2]
    _, Ad = _padded(A, lda, off, dev)
    _, Bd = _padded(B, ldb, off, dev)
    res = oracle.dgemm(A, B, 12)
    assert len(res.fallback_rows) == 0 and len(res.fallback_cols) == 0
    sentinel = -7.25

    def check(cbuf, cview, expect):
        assert np.array_equal(bits(oz.from_device_colmajor(cview)), bits(expect))
        whole = cbuf[off:].view(n, ldc)
        assert bool((whole[:, m:] == sentinel).all()) and bool((cbuf[:off] == sentinel).all())

    # staged plan
    cbuf, Cd = _padded(np.zeros((m, n)), ldc, off, dev, fill=sentinel)
    plan = oz.Plan(m, n, k, 12, 0, device=dev)
    plan.deconstruct(Ad, Bd)
    plan.residue_gemm()
    plan.reconstruct(Cd)
    torch.cuda.synchronize()
    check(cbuf, Cd, res.C)
    # workspace entry point, C <- C0 + A B
    cbuf, Cd = _padded(C0, ldc, off, dev, fill=sentinel)
    oz.matmul(Ad, Bd, 12, oz.OZ2_ACCUMULATE, C=Cd)
    torch.cuda.synchronize()
    check(cbuf, Cd, oracle.dgemm(A, B, 12, C_in=C0).C)
    # plain entry point
    cbuf, Cd = _padded(np.zeros((m, n)), ldc, off, dev, fill=sentinel)
    oz.ozaki2_dgemm(m, n, k, Ad, lda, Bd, ldb, Cd, ldc, 12)
    torch.cuda.synchronize()
    check(cbuf, Cd, res.C)
    del plan
    torch.cuda.synchronize()


def test_batched_padded_leading_dimensions():
    """The single-launch batched path with lda, ldb, ldc above the row counts
    (odd), strides with gaps between problems and an unaligned base."""
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    nb, m, n, k = 5, 40, 50, 30
    Ab, Bb = synth.batched(nb, m, n, k, seed=88)
    lda, ldb, ldc = m + 3, k + 1, m + 5
    sA, sB, sC = lda * k + 7, ldb * n + 3, ldc * n + 9
    off = 1
    abuf = torch.full((off + sA * nb,), float("nan"), dtype=torch.float64, device=dev)
    bbuf = torch.full((off + sB * nb,), float("nan"), dtype=torch.float64, device=dev)
    cbuf = torch.full((off + sC * nb,), -7.25, dtype=torch.float64, device=dev)
    for b in range(nb):
        abuf[off + b * sA:off + b * sA + lda * k].view(k, lda)[:, :m].copy_(
            torch.from_numpy(np.ascontiguousarray(Ab[b].T)).to(dev))
        bbuf[off + b * sB:off + b * sB + ldb * n].view(n, ldb)[:, :k].copy_(
            torch.from_numpy(np.ascontiguousarray(Bb[b].T)).to(dev))
    oz.ozaki2_dgemm_strided_batched(m, n, k, abuf[off:], lda, sA, bbuf[off:], ldb, sB, cbuf[off:],
                                    ldc, sC, nb, 12)
    torch.cuda.synchronize()
    host = cbuf.cpu().numpy()
    used = np.zeros(host.shape, dtype=bool)
    for b in range(nb):
        base = off + b * sC
        Cb = host[base:base + ldc * n].reshape(n, ldc)[:, :m].T
        used[base:base + ldc * n].reshape(n, ldc)[:, :m] = True
        assert np.array_equal(bits(Cb), bits(oracle.dgemm(Ab[b], Bb[b], 12).C)), b
    assert np.all(host[~used] == -7.25)


def _batched_run(Ab, Bb, r):
    import paper_2606_06510_amd as oz
    import torch
    dev = device()
    nb, m, k = Ab.shape
    n = Bb.shape[2]
    Ad = torch.from_numpy(np.ascontiguousarray(Ab.transpose(0, 2, 1))).to(dev)
    Bd = torch.from_numpy(np.ascontiguousarray(Bb.transpose(0, 2, 1))).to(dev)
    Cd = torch.full((nb, n, m), float("nan"), dtype=torch.float64, device=dev)
    oz.ozaki2_dgemm_strided_batched(m, n, k, Ad, m, m * k, Bd, k, k * n, Cd, m, m * n, nb, r)
    torch.cuda.synchronize()
    return Cd.cpu().numpy().transpose(0, 2, 1)


@pytest.mark.parametrize("shape", [(1, 1, 1), (17, 33, 5), (64, 64, 64), (40, 64, 63), (64, 7, 64)])
def test_batched_single_launch_shapes(shape):
    m, n, k = shape
    Ab, Bb = synth.batched(6, max(m, k), max(n, k), max(k, 1), seed=m * 7 + n + k)
    Ab = np.ascontiguousarray(Ab[:, :m, :k])
    Bb = np.ascontiguousarray(Bb[:, :k, :n])
    C = _batched_run(Ab, Bb, 12)
    for b in range(Ab.shape[0]):
        rb = oracle.dgemm(Ab[b], Bb[b], 12)
        assert np.array_equal(bits(C[b]), bits(rb.C)), (shape, b)


@pytest.mark.parametrize("r", [8, 10, 13, 16])
def test_batched_single_launch_moduli(r):
    Ab, Bb = synth.batched(4, 64, 64, 64, seed=40 + r)
    C = _batched_run(Ab, Bb, r)
    for b in range(4):
        assert np.array_equal(bits(C[b]), bits(oracle.dgemm(Ab[b], Bb[b], r).C)), (r, b)


def test_batched_single_launch_fallback_and_zeros():
    from tests.gpu_util import fallback_ok
    Ab, Bb = synth.batched(4, 64, 64, 64, seed=77)
    Ab = Ab.copy()
    Bb = Bb.copy()
    Ab[0, 3, 5] = np.nan                 # T1 row of A
    Bb[1, 7, 9] = np.inf                 # T1 column of B
    Ab[2, 10, :32] *= 1e200              # T2: half a row far above the other half
    Ab[3] = 0.0                          # all-zero problem
    C = _batched_run(Ab, Bb, 12)
    for b in range(4):
        rb = oracle.dgemm(Ab[b], Bb[b], 12)
        fr = set(rb.fallback_rows.tolist())
        fc = set(rb.fallback_cols.tolist())
        for i in range(64):
            for j in range(64):
                if i in fr or j in fc:
                    assert fallback_ok(C[b], Ab[b], Bb[b], i, j), (b, i, j)
                else:
                    assert bits(C[b][i, j]) == bits(rb.C[i, j]), (b, i, j)
    assert np.all(bits(C[3]) == 0)       # exact zero is +0.0


@pytest.mark.parametrize("shape,r", [((1536, 1536, 200), 12), ((2000, 2100, 130), 12),
                                     ((2560, 2560, 96), 12), ((4096, 2048, 64), 12),
                                     ((2048, 2048, 100), 16), ((4096, 2048, 70), 13),
                                     ((4096, 4096, 2048), 12), ((4096, 4096, 1536), 13)])
def test_moduli_per_workgroup_grids(shape, r):
    """Tile counts between 1 and 2 per CU make each residue-GEMM workgroup walk
    2, 3, 4, 6 or 7 moduli (the last group shorter for r = 13); at k = 2048
    and 1536 the work per workgroup sets the split instead (8 + 4 and 10 + 3
    moduli).  Sampled outputs, including the ragged last row and column
    blocks, are bit-exact."""
    import paper_2606_06510_amd as oz
    import torch
    m, n, k = shape
    A, B = synth.lognormal(m, n, k, seed=m + 3 * n + k)
    dev = device()
    Ad = oz.to_device_colmajor(A, dev)
    Bd = oz.to_device_colmajor(B, dev)
    Cd = oz.colmajor_empty(m, n, device=dev)
    plan = oz.Plan(m, n, k, r, 0, device=dev)
    plan.deconstruct(Ad, Bd)
    plan.residue_gemm()
    plan.reconstruct(Cd)
    torch.cuda.synchronize()
    rng = np.random.default_rng(m + n)
    rows = np.unique(np.concatenate([rng.choice(m, 10, replace=False), [0, m - 1]]))
    cols = np.unique(np.concatenate([rng.choice(n, 10, replace=False), [0, n - 1]]))
    C = Cd.index_select(0, torch.as_tensor(rows, device=dev)).index_select(
        1, torch.as_tensor(cols, device=dev)).cpu().numpy()
    res = oracle.dgemm(A, B, r, rows=rows, cols=cols)
    assert len(res.fallback_rows) == 0 and len(res.fallback_cols) == 0
    assert np.array_equal(bits(C), bits(res.C))
    del plan, Ad, Bd, Cd
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("shape,r,acc", [((1024, 512, 200), 12, False), ((1000, 500, 448), 15, False),
                                         ((1024, 512, 256), 12, True), ((2048, 1024, 512), 9, False)])
def test_short_k_two_workgroups_per_cu(shape, r, acc):
    """Short k (at most 8 K-stages per product) on a tile count divisible by
    8: the residue GEMMs run as two workgroups per CU, each on one 256 x 128
    half of a tile.  Every stage is compared with the oracle (codes, scales,
    planes, residue representatives, C), including the accumulate route and
    ragged m, n and k."""
    m, n, k = shape
    if acc:
        A, B, Cin = synth.rankk(m, n, k, seed=m + n + k)
        res = oracle.dgemm(A, B, r, C_in=Cin)
        plan, C = run_staged(A, B, r, flags=1, C_in=Cin)
        compare_C(C, A, B, res, C_in=Cin)
        return
    A, B = synth.lognormal(m, n, k, seed=m + n + k + r)
    res = oracle.dgemm(A, B, r)
    plan, C = run_staged(A, B, r)
    compare_all(plan, C, A, B, r, res, check_integers=m * n <= 600000)


def test_subnormal_and_overflowing_results():
    """Rows and columns scaled so that one block of C lies in the subnormal
    range and another overflows: the GPU's gradual-underflow rounding path and
    the overflow to infinity are bit-exact against the oracle."""
    m, n, k = 96, 80, 200
    A, B = synth.lognormal(m, n, k, seed=321)
    A = A.copy()
    B = B.copy()
    A[:32] *= 2.0 ** -560
    A[64:] *= 2.0 ** 520
    B[:, :24] *= 2.0 ** -500
    B[:, 56:] *= 2.0 ** 520
    res = oracle.dgemm(A, B, 12)
    assert ((res.C != 0) & (np.abs(res.C) < 2.0 ** -1022)).sum() == 32 * 24
    assert np.isinf(res.C).sum() == 32 * 24
    plan, C = run_staged(A, B, 12)
    compare_all(plan, C, A, B, 12, res)


@pytest.mark.parametrize("r", [12, 15])
def test_batched_subnormal_and_overflowing_results(r):
    """The single-launch path rounds into the subnormal range and overflows
    to infinity bit-exactly: problem 0 has rows and columns scaled so that
    one block of C is subnormal and another overflows; problem 1 stays in
    range (r = 12 takes the three-limb CRT, r = 15 the 32-bit words)."""
    Ab, Bb = synth.batched(2, 64, 64, 64, seed=90 + r)
    Ab = Ab.copy()
    Bb = Bb.copy()
    Ab[0] /= np.abs(Ab[0]).max()          # undo the per-matrix scale of the workload
    Bb[0] /= np.abs(Bb[0]).max()
    Ab[0, :16] *= 2.0 ** -560
    Ab[0, 48:] *= 2.0 ** 520
    Bb[0, :, :12] *= 2.0 ** -500
    Bb[0, :, 40:] *= 2.0 ** 520
    C = _batched_run(Ab, Bb, r)
    r0 = oracle.dgemm(Ab[0], Bb[0], r)
    assert ((r0.C != 0) & (np.abs(r0.C) < 2.0 ** -1022)).sum() == 16 * 12
    assert np.isinf(r0.C).sum() == 16 * 24
    for b in range(2):
        rb = r0 if b == 0 else oracle.dgemm(Ab[b], Bb[b], r)
        assert not len(rb.fallback_rows) and not len(rb.fallback_cols)
        assert np.array_equal(bits(C[b]), bits(rb.C)), b


def test_repeated_reconstruct_keeps_fallback_lists():
    """A plan may reconstruct its residues more than once; the flagged-row
    lists the deconstruction built stay as they are (more than half the rows
    are flagged here, so lists that grew per reconstruction would overrun
    their m entries)."""
    import paper_2606_06510_amd as oz
    import torch
    m, n, k = 200, 150, 100
    A, B = synth.uniform(m, n, k, seed=77)
    A = A.copy()
    A[:140, ::2] *= 1e200                     # T2: intra-row span ~2^664 on 140 rows
    res = oracle.dgemm(A, B, 12)
    assert len(res.fallback_rows) == 140 and len(res.fallback_cols) == 0
    plan, C = run_staged(A, B, 12)
    compare_C(C, A, B, res)
    assert plan.query(oz.OZ2_Q_FALLBACK_COUNT) == (140, 0)
    C2d = oz.to_device_colmajor(np.full((m, n), np.nan), device())
    plan.reconstruct(C2d)
    torch.cuda.synchronize()
    C2 = oz.from_device_colmajor(C2d)
    assert np.array_equal(bits(C2), bits(C))
    assert plan.query(oz.OZ2_Q_FALLBACK_COUNT) == (140, 0)


def test_operand_stationary_planes():
    """Mode P on a fixed-scale plan: A's planes are kept across a product with a
    new B, then B's across a new A; every product equals the oracle's
    fixed-scale result on its pair, bit for bit.  One-operand deconstruction
    is refused without OZ2_SCALE_FIXED and before both operands exist."""
    import paper_2606_06510_amd as oz
    import torch
    m, n, k = 300, 260, 200
    A, B1 = synth.lognormal(m, n, k, seed=41)
    A2, B2 = synth.lognormal(m, n, k, seed=43)
    dev = device()
    Ad, B1d, A2d, B2d = (oz.to_device_colmajor(X, dev) for X in (A, B1, A2, B2))
    plan = oz.Plan(m, n, k, 12, oz.OZ2_SCALE_FIXED, device=dev)
    with pytest.raises(oz.Ozaki2Error):
        plan.deconstruct_a(Ad)
        plan.residue_gemm()                   # B was never deconstructed

    def product():
        Cd = oz.colmajor_empty(m, n, device=dev)
        plan.residue_gemm()
        plan.reconstruct(Cd)
        torch.cuda.synchronize()
        return oz.from_device_colmajor(Cd)

    plan.deconstruct(Ad, B1d)
    C1 = product()
    plan.deconstruct_b(B2d)
    C2 = product()
    plan.deconstruct_a(A2d)
    C3 = product()
    for C, X, Y in ((C1, A, B1), (C2, A, B2), (C3, A2, B2)):
        compare_C(C, X, Y, oracle.dgemm(X, Y, 12, mode="fixed"))
    adaptive = oz.Plan(m, n, k, 12, 0, device=dev)
    adaptive.deconstruct(Ad, B1d)
    with pytest.raises(oz.Ozaki2Error):
        adaptive.deconstruct_b(B2d)


def test_side_streams_and_concurrent_plans():
    """Work is enqueued on the stream it is given: two plans of different
    shapes run interleaved on two side streams, ozaki2_dgemm_ex on a third;
    the first plan's A is overwritten on its own stream just before its
    deconstruction, so a library that ignored the stream could read stale
    data.  Every result is bit-exact against the oracle."""
    import torch
    import paper_2606_06510_amd as oz
    dev = device()
    A1, B1 = synth.lognormal(300, 260, 500, seed=41)
    A1b = synth.lognormal(300, 260, 500, seed=43)[0]
    A2, B2 = synth.uniform(257, 129, 700, seed=42)
    res1 = oracle.dgemm(A1b, B1, 12)
    res2 = oracle.dgemm(A2, B2, 12)
    res3 = oracle.dgemm(A2, B2, 13)
    Ad1, Bd1 = oz.to_device_colmajor(A1, dev), oz.to_device_colmajor(B1, dev)
    Anew = oz.to_device_colmajor(A1b, dev)
    Ad2, Bd2 = oz.to_device_colmajor(A2, dev), oz.to_device_colmajor(B2, dev)
    C1 = oz.colmajor_empty(300, 260, device=dev)
    C2 = oz.colmajor_empty(257, 129, device=dev)
    C3 = oz.colmajor_empty(257, 129, device=dev)
    p1 = oz.Plan(300, 260, 500, 12, 0, device=dev)
    p2 = oz.Plan(257, 129, 700, 12, 0, device=dev)
    torch.cuda.synchronize()
    s1, s2, s3 = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s1):
        Ad1.copy_(Anew)                     # ordered before the deconstruction on s1
    p1.deconstruct(Ad1, Bd1, stream=s1)
    p2.deconstruct(Ad2, Bd2, stream=s2)
    oz.matmul(Ad2, Bd2, num_moduli=13, C=C3, stream=s3)
    p1.residue_gemm(stream=s1)
    p2.residue_gemm(stream=s2)
    p1.reconstruct(C1, stream=s1)
    p2.reconstruct(C2, stream=s2)
    torch.cuda.synchronize()
    compare_C(oz.from_device_colmajor(C1), A1b, B1, res1)
    compare_C(oz.from_device_colmajor(C2), A2, B2, res2)
    compare_C(oz.from_device_colmajor(C3), A2, B2, res3)
