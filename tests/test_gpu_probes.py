"""gfx950 probes through the C ABI (include/ozaki2_probes.h): the hardware
facts the exactness argument rests on -- the E4M3 encoding of the split's
conversion instruction and exact FP32 accumulation of FP8 MFMA products up to
2^24 (Eq. (accum-exact)) -- checked against the format's definition and exact
integer sums; plus sanity of the measured peaks."""
import numpy as np
import pytest

import paper_2606_06510_amd as oz
from oracle import e4m3

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def test_e4m3_encoding_of_every_finite_value(torch_cuda):
    torch = torch_cuda
    codes = [b for b in range(256) if e4m3.decode(b) == e4m3.decode(b)]     # drop the two NaNs
    vals = np.array([e4m3.decode(b) for b in codes], dtype=np.float32)
    x = torch.from_numpy(vals).cuda()
    out = torch.empty(len(vals), dtype=torch.uint8, device="cuda")
    oz.ozaki2_probe_e4m3(x, out, len(vals))
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert list(got) == codes


def test_e4m3_exact_integers_used_by_the_planes(torch_cuda):
    torch = torch_cuda
    ints = [v for v in e4m3.exact_integers() if -33 <= v <= 33]
    x = torch.tensor(ints, dtype=torch.float32, device="cuda")
    out = torch.empty(len(ints), dtype=torch.uint8, device="cuda")
    oz.ozaki2_probe_e4m3(x, out, len(ints))
    torch.cuda.synchronize()
    assert list(out.cpu().numpy()) == [e4m3.encode_int(v) for v in ints]


def _operands(rng, lo, hi):
    vals = [v for v in e4m3.exact_integers() if lo <= v <= hi]
    a = rng.choice(vals, size=(64, 32))
    b = rng.choice(vals, size=(64, 32))
    return a, b


def _run_accum(torch, a, b, chain):
    enc = np.vectorize(e4m3.encode_int)
    ad = torch.from_numpy(enc(a).astype(np.uint8)).cuda()
    bd = torch.from_numpy(enc(b).astype(np.uint8)).cuda()
    out = torch.empty((64, 16), dtype=torch.float32, device="cuda")
    oz.ozaki2_probe_accum(ad, bd, chain, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    # lane L holds row / column L%32 and k bytes 32(L/32)..: A[row][k], B[col][k]
    A = np.zeros((32, 64), dtype=np.int64)
    B = np.zeros((32, 64), dtype=np.int64)
    for lane in range(64):
        A[lane % 32, 32 * (lane // 32):32 * (lane // 32) + 32] = a[lane]
        B[lane % 32, 32 * (lane // 32):32 * (lane // 32) + 32] = b[lane]
    C = A @ B.T * chain
    want = np.zeros((64, 16))
    for lane in range(64):
        for e in range(16):
            want[lane, e] = C[8 * (e // 4) + 4 * (lane // 32) + e % 4, lane % 32]
    return got, want


def test_fp32_accumulation_exact_to_2_pow_24(torch_cuda):
    # every product 16*16 = 256 (the largest plane term), 64 per MFMA: after
    # 1024 chained MFMAs each output is exactly 2^24
    a = np.full((64, 32), 16)
    b = np.full((64, 32), 16)
    got, want = _run_accum(torch_cuda, a, b, 1024)
    assert np.all(want == 2 ** 24)
    assert np.array_equal(got, want)


def test_fp32_accumulation_exact_mixed_signs(torch_cuda):
    rng = np.random.default_rng(11)
    a, b = _operands(rng, -16, 16)
    # each MFMA adds at most 64 * 256 per output, so 1024 of them stay within 2^24
    got, want = _run_accum(torch_cuda, a, b, 1024)
    assert np.abs(want).max() <= 2 ** 24
    assert np.array_equal(got, want)


def test_copy_probe_and_peaks(torch_cuda):
    torch = torch_cuda
    n = 64 << 20
    src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    dst = torch.zeros(n, dtype=torch.uint8, device="cuda")
    oz.ozaki2_probe_copy(src, dst, n)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    gbs = oz.ozaki2_probe_copy_peak(256 << 20, 3)
    tf = oz.ozaki2_probe_mfma_peak(200)
    td = oz.ozaki2_probe_mfma_digits(2000)
    assert 500 < gbs < 8200          # at most the 8 TB/s datasheet figure
    assert 500 < tf < 5100           # at most the 5 PF dense FP8 figure
    assert 500 < td < 5100
