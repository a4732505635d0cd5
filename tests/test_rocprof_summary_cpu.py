"""The arithmetic of the profile summaries (paper_2606_06510_amd.rocprof_summary)
on small synthetic rocprofv3 CSV files: which dispatches count as timed steps,
the copy-kernel scaling of FETCH_SIZE / WRITE_SIZE, the FP8 operation count,
busy share and clock of the MFMA summary, the algorithmic bytes of the
memory-bound kernels and the SQ counter ratios."""
import csv
import hashlib

import pytest

from paper_2606_06510_amd import rocprof_summary as rs


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)
    return str(path)


def _kv(path):
    out = {}
    for line in open(path):
        if ": " in line and not line.startswith(("#", "|")):
            k, v = line.split(": ", 1)
            out[k] = v.split()[0]
    return out


def _table(path):
    rows = {}
    for line in open(path):
        if line.startswith("| ") and not line.startswith(("| kernel", "| counter")):
            cells = [c.strip() for c in line.strip().strip("|").split("|")]
            rows[cells[0]] = cells[1:]
    return rows


def _counter_rows(kernel, dispatch, start, end, counters):
    return [[dispatch, kernel, name, value, start, end] for name, value in counters.items()]


CC_HEADER = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
             "End_Timestamp"]


def test_trace_keeps_the_timed_steps_only(tmp_path):
    # kernel A: 2 launches per step over 5 steps, launch j lasting 10 + j us;
    # kernel B: once per plan (dropped: not a whole number per step)
    rows, t = [], 0
    for j in range(10):
        rows.append(["void k_a<1>(int)", t, t + 10000 + 1000 * j])
        t += 50000
    rows.append(["k_b(float)", t, t + 777])
    src = _write(tmp_path / "trace.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"], rows)
    dst = tmp_path / "trace.md"
    rs.trace(src, dst, "t", "cmd", skip=2, count=2, steps=5)
    tab = _table(dst)
    assert set(tab) == {"void k_a<1>"}
    L, calls, avg, lo, hi, per_step, share = tab["void k_a<1>"]
    # dispatches 4 .. 7 (L = 2): 14, 15, 16, 17 us
    assert (L, calls) == ("2", "4")
    assert float(avg) == pytest.approx(15.5)
    assert float(lo) == pytest.approx(14.0) and float(hi) == pytest.approx(17.0)
    assert float(per_step) == pytest.approx(31.0)   # the sum over 2 launches per step
    assert share == "100.0%"


def test_trace_without_steps_skips_dispatches(tmp_path):
    rows = [["k_c", 10 ** 5 * i, 10 ** 5 * i + (5000 if i < 3 else 9000)] for i in range(6)]
    src = _write(tmp_path / "trace.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"], rows)
    dst = tmp_path / "trace.md"
    rs.trace(src, dst, "t", "cmd", skip=3, count=3)
    calls, avg = _table(dst)["k_c"][:2]
    assert calls == "3" and float(avg) == pytest.approx(9.0)


def test_traffic_scales_by_the_copy_kernel(tmp_path):
    copy_bytes = 1 << 30
    fetch_rows, write_rows = [], []
    d = 0
    # the copy reads 1 GiB and writes 1 GiB; its counters read half the fetch
    for _ in range(2):
        fetch_rows += _counter_rows("k_copy(double const*)", d, 0, 1, {"FETCH_SIZE": 524288.0})
        write_rows += _counter_rows("k_copy(double const*)", d, 0, 1, {"WRITE_SIZE": 1048576.0})
        d += 1
    for j in range(3):   # three steps, one launch each; the value is split over two rows
        fetch_rows += [[d, "void k_res<0>(int)", "FETCH_SIZE", 60.0 + j, 0, 1],
                       [d, "void k_res<0>(int)", "FETCH_SIZE", 40.0 - j, 0, 1]]
        write_rows += [[d, "void k_res<0>(int)", "WRITE_SIZE", 50.0, 0, 1]]
        d += 1
    f = _write(tmp_path / "f.csv", CC_HEADER, fetch_rows)
    w = _write(tmp_path / "w.csv", CC_HEADER, write_rows)
    src = tmp_path / "k.hip"
    src.write_text("kernel source\n")
    dst = tmp_path / "traffic.txt"
    rs.traffic(f, w, dst, "void k_res<0>", copy_bytes, str(src), "cf", "cw", steps=5)
    kv = _kv(dst)
    assert float(kv["fetch_scale"]) == pytest.approx(2.0)
    assert float(kv["write_scale"]) == pytest.approx(1.0)
    assert int(kv["fetch_bytes_per_launch"]) == 100 * 1024 * 2
    assert int(kv["write_bytes_per_launch"]) == 50 * 1024
    assert int(kv["traffic_bytes_per_launch"]) == 100 * 1024 * 2 + 50 * 1024
    assert "launches_per_step" not in kv          # 3 dispatches are not a whole number of 5 steps
    assert kv["kernel_source_sha256"] == hashlib.sha256(b"kernel source\n").hexdigest()
    rs.traffic(f, w, dst, "void k_res<0>", copy_bytes, str(src), "cf", "cw", steps=3)
    kv = _kv(dst)
    assert int(kv["launches_per_step"]) == 1
    assert int(kv["traffic_bytes_per_step"]) == 100 * 1024 * 2 + 50 * 1024


def test_mfma_ops_busy_share_and_clock(tmp_path):
    rows = []
    # 3 launches of 1 ms; the first (warm-up) is left out with skip=1
    for d in range(3):
        rows += _counter_rows("k_gemm", d, d * 10 ** 7, d * 10 ** 7 + 10 ** 6, {
            "SQ_INSTS_VALU_MFMA_MOPS_F8": 1.0e9 * (1 + 9 * (d == 0)),
            "SQ_VALU_MFMA_BUSY_CYCLES": 0.5 * 2.0e6 * 1024,      # half of every SIMD's cycles
            "GRBM_GUI_ACTIVE": 8 * 2.0e6})                       # 2e6 cycles per XCD: 2 GHz
    src_csv = _write(tmp_path / "m.csv", CC_HEADER, rows)
    src = tmp_path / "k.hip"
    src.write_text("x")
    dst = tmp_path / "mfma.txt"
    rs.mfma(src_csv, dst, str(src), "cmd", skip=1)
    n, avg, ops, tflops, busy, clock = _table(dst)["k_gemm"]
    assert n == "2" and float(avg) == pytest.approx(1000.0)
    assert float(ops) == pytest.approx(512e9)                  # MOPS x 512
    assert float(tflops) == pytest.approx(512.0, abs=1)        # 512e9 FLOP in 1 ms
    assert busy == "50.0%" and float(clock) == pytest.approx(2.0)


def test_algorithmic_bytes():
    m, n, k, r, p = 300, 200, 100, 12, 30
    alg = rs._algorithmic(m, n, k, r, p)
    assert alg["k_scan_codes_rows"] == 9 * m * k and alg["k_scan_codes_cols"] == 9 * k * n
    assert alg["k_rebase"] == 2 * (m * k + k * n)
    assert alg["k_split"] == (8 + p) * (m * k + k * n)
    for pair in ("false", "true"):
        assert alg[f"void k_reconstruct<12, false, {pair}>"] == 18 * m * n + 8 * m * n
    acc = rs._algorithmic(m, n, k, 15, p, acc=True)
    assert acc["void k_reconstruct<15, true, true>"] == 3 * 15 * m * n // 2 + 16 * m * n


def test_hbm_rates_against_the_peak(tmp_path):
    m = n = k = 1024
    r, p = 12, 30
    alg = rs._algorithmic(m, n, k, r, p)
    split_t = alg["k_split"] / 4.0e12           # an achieved 4 TB/s
    stats = _write(tmp_path / "s.csv", ["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "Percentage"],
                   [["k_split", 1, split_t * 1e9, 0, 0, 100.0],
                    ["k_copy", 1, 1000.0, 0, 0, 0.0]])
    f = _write(tmp_path / "f.csv", CC_HEADER,
               _counter_rows("k_copy", 0, 0, 1, {"FETCH_SIZE": 512.0})
               + _counter_rows("k_split", 1, 0, 1, {"FETCH_SIZE": 8 * 2 * m * k / 2048.0}))
    w = _write(tmp_path / "w.csv", CC_HEADER,
               _counter_rows("k_copy", 0, 0, 1, {"WRITE_SIZE": 1024.0})
               + _counter_rows("k_split", 1, 0, 1, {"WRITE_SIZE": p * 2 * m * k / 1024.0}))
    dst = tmp_path / "hbm.md"
    rs.hbm(stats, f, w, dst, 1 << 20, m, n, k, r, p, "ct", "cf", "cw")
    row = _table(dst)["k_split"]
    assert float(row[3]) == pytest.approx(1.0, abs=1e-3)       # measured = algorithmic bytes
    assert row[4] == "4.00 TB/s" and row[5] == "50%"


def test_counter_ratios(tmp_path):
    cyc = 1.0e6                                   # per XCD, GRBM sums 8
    rows = []
    for d in range(3):
        rows += _counter_rows("void k_b<12, false>", d, 0, 500_000, {
            "SQ_INSTS_VALU": 1024 * cyc / 4 * 0.5,        # issuing on half the SIMD cycles
            "SQ_LDS_BANK_CONFLICT": 256 * cyc * 0.25,
            "SQ_WAVE_CYCLES": 1024 * cyc / 4 * 2,         # two resident waves per SIMD
            "SQ_WAIT_ANY": 1024 * cyc / 4 * 2 * 0.3,
            "GRBM_GUI_ACTIVE": 8 * cyc})
    rows += _counter_rows("other", 9, 0, 1, {"SQ_INSTS_VALU": 1.0, "GRBM_GUI_ACTIVE": 1.0})
    src_csv = _write(tmp_path / "c.csv", CC_HEADER, rows)
    src = tmp_path / "k.hip"
    src.write_text("y")
    dst = tmp_path / "sq.txt"
    rs.counters(str(dst), "void k_b<12, false>", str(src), 1, 4096, [(src_csv, "cmd")])
    kv = _kv(dst)
    assert float(kv["clock_ghz"]) == pytest.approx(2.0)          # 1e6 cycles in 0.5 ms
    assert float(kv["valu_issue_share"]) == pytest.approx(0.5)
    assert float(kv["lds_bank_conflict_share"]) == pytest.approx(0.25)
    assert float(kv["waves_per_simd"]) == pytest.approx(2.0)
    assert float(kv["sq_wait_any_over_wave_cycles"]) == pytest.approx(0.3)
    per_unit = _table(dst)["SQ_INSTS_VALU"][1]
    assert float(per_unit) == pytest.approx(1024 * cyc / 8 / 4096, rel=1e-3)
