"""Render rocprofv3 output into the short text summaries kept under profiles/.

    python -m paper_2606_06510_amd.rocprof_summary stats STATS_CSV OUT_MD TITLE COMMAND
    python -m paper_2606_06510_amd.rocprof_summary trace TRACE_CSV OUT_MD TITLE COMMAND SKIP COUNT \\
        [STEPS]
    python -m paper_2606_06510_amd.rocprof_summary traffic FETCH_CSV WRITE_CSV OUT_TXT \\
        KERNEL COPY_BYTES SOURCE CMD_FETCH CMD_WRITE [STEPS]
    python -m paper_2606_06510_amd.rocprof_summary mfma COUNTER_CSV OUT_TXT SOURCE CMD [SKIP [STEPS]]
    python -m paper_2606_06510_amd.rocprof_summary hbm STATS_CSV FETCH_CSV WRITE_CSV OUT_MD \
        COPY_BYTES M N K R PSTORE CMD_TRACE CMD_FETCH CMD_WRITE [SKIP COUNT [ACC]]
    python -m paper_2606_06510_amd.rocprof_summary counters OUT_TXT KERNEL SOURCE SKIP UNITS \
        CSV CMD [CSV CMD ...]

``stats`` turns a ``--kernel-trace --stats`` kernel_stats.csv into a markdown
table.  ``trace`` does the same from the per-dispatch kernel_trace.csv, keeping
only dispatches SKIP .. SKIP+COUNT-1 of each kernel (in launch order): with
SKIP = the bench's warm-up steps and COUNT = its timed steps, the averages
cover the timed steps alone (kernels launched once per plan, not per step,
drop out).  With STEPS (every step the traced program ran), a kernel
dispatched L times per step (L = its dispatches / STEPS, a whole number)
keeps dispatches L*SKIP .. L*(SKIP+COUNT)-1, and the table adds L and the
kernel's time per step (the sum of its L launches).  ``traffic`` reads two ``--pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE``
counter_collection.csv files (KiB per dispatch), takes the mean per launch of
KERNEL and of the plain copy kernel (COPY_BYTES read and written), and scales
the kernel's figures by copy_bytes / copy_reading; the result carries the
sha256 of SOURCE so that bench.py uses it only for the kernel it was taken on.
``mfma`` reads one ``--pmc SQ_INSTS_VALU_MFMA_MOPS_F8 SQ_VALU_MFMA_BUSY_CYCLES
GRBM_GUI_ACTIVE`` counter_collection.csv and reports, per FP8-MFMA kernel,
the FP8 operations per launch (MOPS x 512), the share of SIMD cycles the MFMA
unit was busy and the shader clock the launch ran at (GRBM_GUI_ACTIVE is
summed over the XCDs: cycles = sum / XCDs, clock = cycles / duration).
With SKIP, ``mfma`` leaves out the first SKIP dispatches of each kernel (the
warm-up launches, which run while the clock settles); with SKIP COUNT,
``hbm`` takes its mean durations from a kernel_trace.csv given in place of
STATS_CSV, over dispatches SKIP .. SKIP+COUNT-1 as ``trace`` does.
``hbm`` puts the memory-bound kernels of an m x n x k product at r moduli
(PSTORE plane bytes per input element) side by side: mean duration from the
kernel trace, algorithmic bytes, the copy-scaled FETCH_SIZE + WRITE_SIZE
bytes, and the achieved rate (algorithmic bytes / mean duration) against
the 8 TB/s HBM peak.
``counters`` gathers the SQ counters of KERNEL from one or more ``--pmc``
passes (each a counter_collection.csv with the command that made it; every
pass also collects GRBM_GUI_ACTIVE for the clock), leaves out the first SKIP
dispatches of the kernel, and writes the mean per launch of each counter,
per unit of work (UNITS per launch, e.g. problems of a batch), and the
ratios that read directly against the chip: VALU instructions x 4 cycles
(a wave64 VALU instruction occupies its SIMD's 16 lanes for 4 cycles) over
the SIMD cycles, LDS bank-conflict cycles over the CU cycles, and the
resident waves per SIMD (SQ_WAVE_CYCLES, counted in 4-cycle units).
"""
from __future__ import annotations

import collections
import csv
import hashlib
import sys


def _short(name):
    if name.startswith("Cijk_"):
        return "rocBLAS DGEMM " + name.split("_")[3] + " (torch.matmul float64, baseline)"
    return name.replace("(anonymous namespace)::", "").split("(")[0]


def stats(src, dst, title, cmd):
    rows = list(csv.DictReader(open(src)))
    with open(dst, "w") as f:
        f.write(f"# {title}\n\nCommand (from the repository root, on one MI355X):\n\n```\n{cmd}\n```\n\n")
        f.write("| kernel | calls | avg (us) | min (us) | max (us) | share |\n|---|---|---|---|---|---|\n")
        for r in rows:
            f.write(f"| {_short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                    f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                    f"{float(r['Percentage']):.1f}% |\n")


def _per_step(n, steps):
    """Launches per step of a kernel dispatched n times in `steps` steps
    (0 when it is not a whole number: launched per plan, not per step)."""
    if not steps or n % steps:
        return 0
    return n // steps


def trace(src, dst, title, cmd, skip, count, steps=None):
    by = collections.defaultdict(list)
    for r in csv.DictReader(open(src)):
        by[_short(r["Kernel_Name"])].append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    rows = []
    for name, ds in by.items():
        ds.sort()
        L = _per_step(len(ds), steps) if steps else 1
        if steps and not L:
            continue
        sel = [(e - b) * 1e-3 for b, e in ds[L * skip:L * (skip + count)]]
        if sel:
            rows.append((name, L, len(sel), sum(sel) / len(sel), min(sel), max(sel), sum(sel)))
    tot = sum(r[6] for r in rows) or 1.0
    rows.sort(key=lambda r: -r[6])
    with open(dst, "w") as f:
        f.write(f"# {title}\n\nCommand (from the repository root, on one MI355X):\n\n```\n{cmd}\n```\n\n")
        if steps:
            f.write(f"The timed steps only ({count} steps after {skip} warm-up steps, of {steps} "
                    f"steps the program ran): for a kernel launched L times per step, its "
                    f"dispatches L*{skip} .. L*{skip + count}-1 in launch order.\n\n")
            f.write("| kernel | launches per step | calls | avg (us) | min (us) | max (us) | "
                    "per step (us) | share |\n|---|---|---|---|---|---|---|---|\n")
            for name, L, n, avg, lo, hi, t in rows:
                f.write(f"| {name} | {L} | {n} | {avg:.1f} | {lo:.1f} | {hi:.1f} | "
                        f"{t / count:.1f} | {100 * t / tot:.1f}% |\n")
            return
        f.write(f"Dispatches {skip} .. {skip + count - 1} of each kernel (launch order), i.e. the "
                f"timed steps only; warm-up launches excluded.\n\n")
        f.write("| kernel | calls | avg (us) | min (us) | max (us) | share |\n|---|---|---|---|---|---|\n")
        for name, L, n, avg, lo, hi, t in rows:
            f.write(f"| {name} | {n} | {avg:.1f} | {lo:.1f} | {hi:.1f} | {100 * t / tot:.1f}% |\n")


def _per_launch(path, counter, counts=None):
    """{kernel short name: mean over dispatches of the summed counter value};
    `counts`, if given, receives the dispatches per kernel."""
    per = collections.defaultdict(float)
    names = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        key = r["Dispatch_Id"]
        per[key] += float(r["Counter_Value"])
        names[key] = _short(r["Kernel_Name"])
    by = collections.defaultdict(list)
    for key, v in per.items():
        by[names[key]].append(v)
    if counts is not None:
        counts.update({k: len(v) for k, v in by.items()})
    return {k: sum(v) / len(v) for k, v in by.items()}


def traffic(fetch_csv, write_csv, dst, kernel, copy_bytes, source, cmd_fetch, cmd_write,
            steps=None):
    counts = {}
    fetch = _per_launch(fetch_csv, "FETCH_SIZE", counts)
    write = _per_launch(write_csv, "WRITE_SIZE")
    copy = next(k for k in fetch if k.startswith("k_copy"))
    sf = copy_bytes / (fetch[copy] * 1024.0)
    sw = copy_bytes / (write[copy] * 1024.0)
    kf, kw = fetch[kernel] * 1024.0 * sf, write[kernel] * 1024.0 * sw
    sha = hashlib.sha256(open(source, "rb").read()).hexdigest()
    with open(dst, "w") as f:
        f.write(f"# HBM traffic per launch of {kernel}: rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per\n"
                f"# dispatch), each scaled by the reading of a plain copy kernel of {copy_bytes} bytes.\n")
        f.write(f"command_fetch: {cmd_fetch}\ncommand_write: {cmd_write}\n")
        f.write(f"kernel: {kernel}\nkernel_source: {source}\nkernel_source_sha256: {sha}\n")
        f.write(f"copy_fetch_kib: {fetch[copy]:.1f}\ncopy_write_kib: {write[copy]:.1f}\n")
        f.write(f"fetch_scale: {sf:.4f}\nwrite_scale: {sw:.4f}\n")
        f.write(f"kernel_fetch_kib_per_launch: {fetch[kernel]:.1f}\n"
                f"kernel_write_kib_per_launch: {write[kernel]:.1f}\n")
        f.write(f"fetch_bytes_per_launch: {kf:.0f}\nwrite_bytes_per_launch: {kw:.0f}\n")
        f.write(f"traffic_bytes_per_launch: {kf + kw:.0f}\n")
        L = _per_step(counts.get(kernel, 0), steps)
        if L:
            f.write(f"launches_per_step: {L}\ntraffic_bytes_per_step: {L * (kf + kw):.0f}\n")
        f.write("# all kernels (KiB per launch, unscaled): fetch / write\n")
        for k in sorted(fetch):
            f.write(f"#   {k}: {fetch[k]:.1f} / {write.get(k, float('nan')):.1f}\n")


def mfma(src, dst, source, cmd, skip=0, steps=None, xcds=8, simds=1024):
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    names, dur, start = {}, {}, {}
    for r in csv.DictReader(open(src)):
        key = r["Dispatch_Id"]
        per[key][r["Counter_Name"]] += float(r["Counter_Value"])
        names[key] = _short(r["Kernel_Name"])
        dur[key] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
        start[key] = int(r["Start_Timestamp"])
    order = collections.defaultdict(list)
    for key in per:
        order[names[key]].append((start[key], key))
    keep = set()
    for name, ks in order.items():
        # SKIP counts steps when STEPS is given: L launches per step each
        L = (_per_step(len(ks), steps) or 1) if steps else 1
        keep.update(key for _, key in sorted(ks)[L * skip:])
    by = collections.defaultdict(list)
    for key, v in per.items():
        if key not in keep:
            continue
        if v.get("SQ_INSTS_VALU_MFMA_MOPS_F8", 0.0) <= 0.0:
            continue
        cycles = v["GRBM_GUI_ACTIVE"] / xcds
        by[names[key]].append((dur[key], v["SQ_INSTS_VALU_MFMA_MOPS_F8"] * 512.0,
                               v["SQ_VALU_MFMA_BUSY_CYCLES"], cycles))
    sha = hashlib.sha256(open(source, "rb").read()).hexdigest()
    with open(dst, "w") as f:
        f.write("# FP8 MFMA activity per launch: rocprofv3 SQ_INSTS_VALU_MFMA_MOPS_F8 (x 512 = FP8\n"
                "# operations), SQ_VALU_MFMA_BUSY_CYCLES over the SIMD cycles, GRBM_GUI_ACTIVE over\n"
                f"# the {xcds} XCDs for the clock.\n")
        f.write(f"command: {cmd}\nkernel_source: {source}\nkernel_source_sha256: {sha}\n")
        if skip:
            f.write(f"# the first {skip} {'steps' if steps else 'launches'} of each kernel "
                    "(warm-up) are left out\n")
        f.write("# busy share and clock are summed over the launches (weighted by their cycles)\n")
        f.write("| kernel | launches | avg (us) | FP8 ops per launch | TFLOP/s | MFMA busy | clock (GHz) |\n")
        f.write("|---|---|---|---|---|---|---|\n")
        for k in sorted(by):
            xs = by[k]
            n = len(xs)
            d = sum(x[0] for x in xs) / n
            fl = sum(x[1] for x in xs) / n
            cyc = sum(x[3] for x in xs)
            f.write(f"| {k} | {n} | {d * 1e6:.1f} | {fl:.4g} | {fl / d / 1e12:.0f} | "
                    f"{100 * sum(x[2] for x in xs) / (cyc * simds):.1f}% | "
                    f"{cyc / sum(x[0] for x in xs) / 1e9:.2f} |\n")


def _algorithmic(m, n, k, r, pstore, acc=False):
    """Algorithmic bytes per launch of the memory-bound kernels: each operand
    read once per pass, each code, plane, residue and output written once
    (and C read once more when accumulating)."""
    ea, eb = m * k, k * n
    return {
        "k_scan_codes_rows": 9 * ea,              # A read (8 B), code byte written (1 B)
        "k_scan_codes_cols": 9 * eb,
        "k_rebase": 2 * (ea + eb),                # code bytes read and rewritten in place
        "k_split": (8 + pstore) * (ea + eb),      # operand read, plane bytes written
        # 12-bit residues read, FP64 written (and read when accumulating);
        # one instantiation per residue layout (lane-major, pair-major)
        **{f"void k_reconstruct<{r}, {'true' if acc else 'false'}, {pair}>":
           3 * r * m * n // 2 + (16 if acc else 8) * m * n for pair in ("false", "true")},
    }


def _trace_avg(path, skip, count):
    by = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        by[_short(r["Kernel_Name"])].append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    out = {}
    for name, ds in by.items():
        sel = [(e - b) * 1e-9 for b, e in sorted(ds)[skip:skip + count]]
        if sel:
            out[name] = sum(sel) / len(sel)
    return out


def hbm(stats_csv, fetch_csv, write_csv, dst, copy_bytes, m, n, k, r, pstore, cmd_t, cmd_f, cmd_w,
        skip=None, count=None, acc=False, peak=8.0e12):
    if skip is None:
        avg = {_short(x["Name"]): float(x["AverageNs"]) * 1e-9
               for x in csv.DictReader(open(stats_csv))}
    else:
        avg = _trace_avg(stats_csv, skip, count)
    fetch = _per_launch(fetch_csv, "FETCH_SIZE")
    write = _per_launch(write_csv, "WRITE_SIZE")
    copy = next(x for x in fetch if x.startswith("k_copy"))
    sf = copy_bytes / (fetch[copy] * 1024.0)
    sw = copy_bytes / (write[copy] * 1024.0)
    alg = _algorithmic(m, n, k, r, pstore, acc)
    with open(dst, "w") as f:
        f.write(f"# Memory-bound kernels of the emulated DGEMM {m}x{n}x{k}, r = {r}: achieved HBM "
                f"rate against the {peak / 1e12:.0f} TB/s peak\n\n")
        f.write("Commands (from the repository root, on one MI355X): the kernel trace for the mean "
                "durations, then one counter pass each for FETCH_SIZE and WRITE_SIZE (each scaled "
                f"by its reading for a plain copy of {copy_bytes} bytes: x{sf:.4f} and x{sw:.4f}).\n\n")
        f.write(f"```\n{cmd_t}\n{cmd_f}\n{cmd_w}\n```\n\n")
        f.write("| kernel | avg (us) | algorithmic bytes | measured bytes (fetch + write) | "
                "measured / algorithmic | achieved (algorithmic / avg) | of peak |\n")
        f.write("|---|---|---|---|---|---|---|\n")
        tot_t = tot_a = 0.0
        for name, ab in alg.items():
            if name not in avg or name not in fetch:
                continue
            t = avg[name]
            mb = fetch[name] * 1024.0 * sf + write.get(name, 0.0) * 1024.0 * sw
            tot_t += t
            tot_a += ab
            f.write(f"| {name} | {t * 1e6:.1f} | {ab / 1e6:.1f} MB | {mb / 1e6:.1f} MB | "
                    f"{mb / ab:.3f} | {ab / t / 1e12:.2f} TB/s | {100 * ab / t / peak:.0f}% |\n")
        f.write(f"| all of the above | {tot_t * 1e6:.1f} | {tot_a / 1e6:.1f} MB | | | "
                f"{tot_a / tot_t / 1e12:.2f} TB/s | {100 * tot_a / tot_t / peak:.0f}% |\n")


def counters(dst, kernel, source, skip, units, passes, xcds=8, cus=256, simds=1024):
    vals = collections.defaultdict(list)
    cyc, dur = [], []
    for path, _ in passes:
        per = collections.defaultdict(lambda: collections.defaultdict(float))
        meta = {}
        for r in csv.DictReader(open(path)):
            if _short(r["Kernel_Name"]) != kernel:
                continue
            key = r["Dispatch_Id"]
            per[key][r["Counter_Name"]] += float(r["Counter_Value"])
            meta[key] = (int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
        keys = [k for _, k in sorted((meta[k][0], k) for k in per)][skip:]
        for key in keys:
            for name, v in per[key].items():
                if name == "GRBM_GUI_ACTIVE":
                    cyc.append(v / xcds)
                    dur.append((meta[key][1] - meta[key][0]) * 1e-9)
                else:
                    vals[name].append(v)
    mean = {k: sum(v) / len(v) for k, v in vals.items()}
    cycles = sum(cyc) / len(cyc)
    d = sum(dur) / len(dur)
    sha = hashlib.sha256(open(source, "rb").read()).hexdigest()
    with open(dst, "w") as f:
        f.write(f"# SQ counters of {kernel} per launch (mean over launches after the first {skip}"
                f" of each pass)\n")
        for _, cmd in passes:
            f.write(f"command: {cmd}\n")
        f.write(f"kernel_source: {source}\nkernel_source_sha256: {sha}\n")
        f.write(f"launch_us: {d * 1e6:.1f}\ncycles_per_launch: {cycles:.0f}\n"
                f"clock_ghz: {cycles / d / 1e9:.2f}\nunits_per_launch: {units}\n")
        f.write("| counter | per launch | per unit |\n|---|---|---|\n")
        for k in sorted(mean):
            f.write(f"| {k} | {mean[k]:.4g} | {mean[k] / units:.4g} |\n")
        simd_cycles = cycles * simds
        if "SQ_INSTS_VALU" in mean:
            f.write(f"valu_issue_share: {4 * mean['SQ_INSTS_VALU'] / simd_cycles:.3f}"
                    "  (VALU instructions x 4 cycles / SIMD cycles)\n")
        if "SQ_INSTS_LDS" in mean:
            f.write(f"lds_insts_per_cu_cycle: {mean['SQ_INSTS_LDS'] / (cycles * cus):.3f}\n")
        if "SQ_LDS_BANK_CONFLICT" in mean:
            f.write(f"lds_bank_conflict_share: {mean['SQ_LDS_BANK_CONFLICT'] / (cycles * cus):.3f}"
                    "  (bank-conflict cycles / CU cycles)\n")
        if "SQ_WAVE_CYCLES" in mean:
            f.write(f"waves_per_simd: {4 * mean['SQ_WAVE_CYCLES'] / simd_cycles:.2f}\n")
        for k in ("SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_LDS",
                  "SQ_WAIT_INST_ANY", "SQ_WAIT_ANY", "SQ_ACTIVE_INST_ANY"):
            if k in mean and "SQ_WAVE_CYCLES" in mean:
                f.write(f"{k.lower()}_over_wave_cycles: {mean[k] / mean['SQ_WAVE_CYCLES']:.3f}\n")


def main(argv):
    if argv[0] == "stats":
        stats(*argv[1:5])
    elif argv[0] == "trace":
        trace(*argv[1:5], int(argv[5]), int(argv[6]), *(int(x) for x in argv[7:8]))
    elif argv[0] == "traffic":
        traffic(argv[1], argv[2], argv[3], argv[4], int(argv[5]), argv[6], argv[7], argv[8],
                *(int(x) for x in argv[9:10]))
    elif argv[0] == "mfma":
        mfma(*argv[1:5], *(int(x) for x in argv[5:7]))
    elif argv[0] == "hbm":
        hbm(argv[1], argv[2], argv[3], argv[4], int(argv[5]), *map(int, argv[6:11]),
            argv[11], argv[12], argv[13], *(int(x) for x in argv[14:16]),
            *(bool(int(x)) for x in argv[16:17]))
    elif argv[0] == "counters":
        rest = argv[6:]
        counters(argv[1], argv[2], argv[3], int(argv[4]), int(argv[5]),
                 [(rest[i], rest[i + 1]) for i in range(0, len(rest), 2)])
    else:
        raise SystemExit(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
