#!/usr/bin/env python3
"""Throughput of the FP64 GEMM emulated on MI355X FP8 MFMA (Ozaki-II, CRT).

One step = one whole pass of the path over one batch of input already
resident in HBM: deconstruct (scan, max-magnitude code GEMM, scales, residue
planes) -> residue GEMMs -> reconstruction (+ fallback).  The default
workload is the largest single-GPU one: the 16384^3 GEMM with entries
(u-0.5)*exp(2 g) and 1% of the rows of A scaled by 1e200, at r = 15 moduli
(the FP64-grade count for that range).  Prints ONE JSON line (rank 0, one
GPU).

Extra fields beside the contract: the residue GEMMs' launch times (HIP
events around them on the launch stream, in the timed steps themselves), the
six-way stage split (a plan created with OZ2_TIME_STAGES, in extra steps
after the timed ones), the native FP64 DGEMM (torch.matmul float64) on the
same inputs, and the CPU oracle on a bounded sample of the same workload
(with bit-parity and exact-error checks of that sample).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP8_PEAK_TFLOPS = 5000.0      # MI355X dense FP8 (E4M3) MFMA
HBM_PEAK_GBS = 8000.0
MIN_WARMUP = 10


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # the clock takes some 20 ms of work to settle after the device idles:
    # fewer warm-up steps than MIN_WARMUP are raised to it
    ap.add_argument("--warmup", type=int, default=MIN_WARMUP)
    ap.add_argument("--config", default="gemm16384_wide")
    ap.add_argument("--moduli", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="sampled rows and columns of the CPU-oracle baseline (default: 512 at "
                         "k = 16384, 2304 at k = 4096; 10-30 s of oracle work on the GPU hosts)")
    ap.add_argument("--route", choices=["staged", "fused"], default="staged",
                    help="residue GEMMs and reconstruction as separate stages (the library's "
                         "default), or fused into one kernel (OZ2_FUSED: r <= 12, k <= 32768)")
    ap.add_argument("--stage-steps", type=int, default=3,
                    help="extra steps on a stage-timed plan for the six-way split")
    ap.add_argument("--no-probes", action="store_true", help="skip the measured-peak probes")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 1 GiB copy kernel (rocprofv3 counter calibration)")
    ap.add_argument("--stationary", action="store_true",
                    help="operand-stationary use (Mode P): A deconstructed once under fixed "
                         "scaling, each step deconstructs a new B and runs the residue GEMMs "
                         "and the reconstruction")
    ap.add_argument("--accuracy-sweep", action="store_true",
                    help="instead of the bench line: max componentwise error of a sampled set "
                         "of outputs against the exact product for r = 8..16")
    return ap.parse_args()


def log(msg):
    """Progress on stderr (the JSON line alone goes to stdout)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def source_sha256(rel):
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def pmc_traffic(kernel_src, tag):
    """HBM traffic per step of the dominant kernel (all its launches in one
    step) from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary, scaled
    by the plain copy kernel's reading; None unless the summary was taken on
    the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{tag}_pmc_traffic.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            key, val = line.split(":", 1)
            vals[key.strip()] = val.strip()
    if vals.get("kernel_source_sha256") != source_sha256(kernel_src):
        return None
    try:
        return float(vals.get("traffic_bytes_per_step", vals["traffic_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def pmc_mfma(kernel_src, tag):
    """MFMA busy share and clock of the residue GEMM from the committed rocprofv3
    counter summary; None unless it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{tag}_pmc_mfma.txt")
    if not os.path.exists(path):
        return None
    lines = open(path).read().splitlines()
    sha = [x.split(":", 1)[1].strip() for x in lines if x.startswith("kernel_source_sha256:")]
    if not sha or sha[0] != source_sha256(kernel_src):
        return None
    for x in lines:
        cells = [c.strip() for c in x.strip("|").split("|")]
        if len(cells) == 7 and ("k_resgemm" in cells[0]):
            return {"mfma_busy": cells[5], "clock_ghz": float(cells[6]),
                    "fp8_ops_per_launch": float(cells[3]), "source": os.path.relpath(path, ROOT)}
    return None


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the emulated GEMM runs on one GPU (a single-GPU kernel path; "
              "its sharding over several GPUs is not implemented). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2606_06510_amd as oz

    cfg = dict(synth.CONFIGS[args.config])
    r = args.moduli or cfg["r"]
    dev = torch.device("cuda:0")
    if cfg["kind"] == "batched":
        batched_line(args, cfg, r, dev)
        return
    if args.config.startswith("gemv"):
        gemv_line(args, cfg, r, dev)
        return
    t_in = time.perf_counter()
    drawn = synth.make(args.config)
    A, B = drawn[0], drawn[1]
    log(f"inputs of {args.config} drawn in {time.perf_counter() - t_in:.1f} s")
    m, k = A.shape
    n = B.shape[1]
    if args.accuracy_sweep:
        accuracy_sweep(A, B, dev)
        return
    if args.stationary:
        stationary_line(args, cfg, r, dev, A, B)
        return
    Ad = oz.to_device_colmajor(A, dev)
    Bd = oz.to_device_colmajor(B, dev)
    flags = 0
    if cfg["kind"] == "rankk":
        Cd = oz.to_device_colmajor(drawn[2], dev)      # C += A B on the drawn C_in
        flags = oz.OZ2_ACCUMULATE
    else:
        Cd = oz.colmajor_empty(m, n, device=dev)
    if args.route == "fused":
        flags |= oz.OZ2_FUSED
    plan = oz.Plan(m, n, k, r, flags, device=dev)
    stream = torch.cuda.current_stream()
    warmup = max(args.warmup, MIN_WARMUP)

    def step(p, ev=None):
        p.deconstruct(Ad, Bd)
        if ev is not None:
            ev[0].record(stream)
        p.residue_gemm()
        if ev is not None:
            ev[1].record(stream)
        p.reconstruct(Cd)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(warmup):
        step(plan)
    torch.cuda.synchronize()
    log(f"{warmup} warm-up steps done")

    # timed steps: HIP events around the residue GEMMs (the dominant kernel:
    # one launch per modulus group, chunk of tiles and k-slab) on the stream
    # they are launched on
    gev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(plan, gev[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    fused = bool(flags & oz.OZ2_FUSED)
    # the dominant kernel: the residue GEMMs, or the fused kernel that runs
    # them inside the reconstruction
    gem = float(np.mean([(e[1].elapsed_time(e[2]) if fused else e[0].elapsed_time(e[1]))
                         for e in gev]))
    slabs = (k + 32767) // 32768
    log(f"{args.steps} timed steps: {ms_step:.3f} ms per step, residue GEMMs {gem:.3f} ms")

    # six-way split: a stage-timed plan on the same workspace, extra steps
    split = {}
    if args.stage_steps > 0:
        tplan = oz.Plan(m, n, k, r, flags | oz.OZ2_TIME_STAGES, device=dev,
                        workspace=plan.workspace)
        acc = []
        for _ in range(args.stage_steps):
            step(tplan)
            acc.append(tplan.query(oz.OZ2_Q_STAGE_TIMES))
        split = {name: round(float(np.mean([a[name] for a in acc])), 4) for name in acc[0]}
        del tplan
    nfb = plan.query(oz.OZ2_Q_FALLBACK_COUNT)

    flop = 2.0 * m * n * k
    tflops = flop / (ms_step * 1e-3) / 1e12
    fp8_flop = 3 * r * flop                     # 3 plane products per modulus
    achieved = fp8_flop / (gem * 1e-3) / 1e12

    # native FP64 DGEMM on the same inputs (baseline only)
    native = None
    try:
        At = torch.from_numpy(np.ascontiguousarray(A)).to(dev)
        Bt = torch.from_numpy(np.ascontiguousarray(B)).to(dev)
        for _ in range(2):
            torch.matmul(At, Bt)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(5):
            torch.matmul(At, Bt)
        torch.cuda.synchronize()
        native = flop / ((time.perf_counter() - t) / 5) / 1e12
        del At, Bt
    except Exception as e:  # pragma: no cover
        native = f"error: {e}"

    peaks = None
    if not args.no_probes:
        peaks = {"fp8_mfma_tflops": round(oz.ozaki2_probe_mfma_peak(2000), 1),
                 "fp8_mfma_digits_tflops": round(oz.ozaki2_probe_mfma_digits(20000), 1),
                 "hbm_copy_gbs": round(oz.ozaki2_probe_copy_peak(1 << 30, 5), 1),
                 "how": "gfx950 probes: independent 32x32x64 FP8 MFMAs on every SIMD "
                        "(near-constant operands; and digit-plane operands read from LDS "
                        "each step, the residue GEMM's inner loop); "
                        "1 GiB device copy (read + write bytes)"}
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        oz.ozaki2_probe_copy(src, dst, 1 << 30)
        torch.cuda.synchronize()
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        nsamp = args.cpu_sample or (512 if k > 8192 else 2304)
        log(f"CPU oracle on {nsamp} x {nsamp} sampled outputs ...")
        C_in = None
        if cfg["kind"] == "rankk":
            # one step from the drawn C_in, so that C = C_in + A B
            C_in = drawn[2]
            Cd.copy_(oz.to_device_colmajor(C_in, dev))
            step(plan)
            torch.cuda.synchronize()
        cpu = cpu_baseline(A, B, r, Cd, nsamp, C_in=C_in)

    tag = f"{'fused' if fused else 'resgemm'}_{args.config}_r{r}"
    ksrc = "paper_2606_06510_amd/csrc/" + ("fused.hip" if fused else "gemm.hip")
    traffic = pmc_traffic(ksrc, tag)
    mfma_pmc = pmc_mfma(ksrc, tag)
    pstore = plan_pstore(r)
    # algorithmic bytes: A, B read once, code bytes and planes written once;
    # residues (12 bits per output and modulus) read and C written (C also
    # read when accumulating)
    dec_bytes = (m * k + k * n) * (8 + 1 + pstore)
    rec_bytes = m * n * (1.5 * r + 8 + (8 if flags & oz.OZ2_ACCUMULATE else 0))
    out = {
        "metric": "effective FP64 TFLOPS of emulated DGEMM (Ozaki-II on FP8 MFMA)",
        "value": round(tflops, 3),
        "unit": "TFLOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8-e4m3 MFMA -> exact int -> f64",
        "data": "synthetic (seeded numpy PCG64)",
        "config": {"workload": f"{args.config}: C {'+' if flags & oz.OZ2_ACCUMULATE else ''}= "
                               f"A B, m={m} n={n} k={k}, {cfg['kind']} entries, r={r} moduli "
                               f"(alpha={3 * r + 1})"
                               f"{', residue GEMMs fused with the reconstruction' if flags & oz.OZ2_FUSED else ''}",
                   "m": m, "n": n, "k": k, "num_moduli": r},
        "roofline": {"bound": "mfma",
                     "kernel": ("k_resgemm_crt (residue GEMMs fused with the reconstruction)"
                                if fused else "k_resgemm (residue GEMMs, 3r FP8 products)"),
                     "achieved": round(achieved, 2), "peak": FP8_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / FP8_PEAK_TFLOPS, 4),
                     "traffic": None if traffic is None else round(traffic),
                     "per_step": f"{fp8_flop:.4g} FP8 FLOP (3r plane products x 2mnk)"
                                 + ("" if fused else ", over all residue-GEMM launches of the "
                                    "step (one per modulus group, chunk of 256 or 1024 tiles and "
                                    f"k-slab; {slabs} k-slab{'s' if slabs > 1 else ''})"),
                     "timing": f"HIP events around the {'fused kernel' if fused else 'residue GEMMs'}"
                               f" in each of the {args.steps} timed steps (first launch start "
                               f"to last launch end), mean {gem:.3f} ms per step"},
        "stages_ms": split,
        "fallback_rows_cols": list(nfb),
        "fp8_mfma_util_residue_gemm": round(achieved / FP8_PEAK_TFLOPS, 4),
        "fp8_mfma_rocprof_residue_gemm": mfma_pmc,
        "measured_peak": peaks,
        "native_fp64_tflops": native if not isinstance(native, float) else round(native, 3),
        "cpu_baseline": cpu,
    }
    if split:
        dec = split["scan_codes"] + split["maxmag_gemm"] + split["split"]
        rec = split["reconstruct"]
        if fused:   # the reconstruction reads no residues; its kernel is the MFMA-bound one
            rec_bytes = m * n * (8 + (8 if flags & oz.OZ2_ACCUMULATE else 0))
        out["deconstruct_gbs_algorithmic"] = round(dec_bytes / (dec * 1e-3) / 1e9, 1)
        out["deconstruct_frac_hbm"] = round(dec_bytes / (dec * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        out["deconstruct_streaming_frac_hbm"] = round(
            dec_bytes / ((split["scan_codes"] + split["split"]) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        out["reconstruct_gbs_algorithmic"] = round(rec_bytes / (rec * 1e-3) / 1e9, 1)
        out["reconstruct_frac_hbm"] = round(rec_bytes / (rec * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        if peaks:
            out["frac_of_measured_peak"] = {
                "residue_gemm_fp8": round(achieved / peaks["fp8_mfma_tflops"], 4),
                "residue_gemm_fp8_digits": round(achieved / peaks["fp8_mfma_digits_tflops"], 4),
                "deconstruct_hbm": round(out["deconstruct_gbs_algorithmic"] / peaks["hbm_copy_gbs"], 4),
                "reconstruct_hbm": round(out["reconstruct_gbs_algorithmic"] / peaks["hbm_copy_gbs"], 4)}
    print(json.dumps(out))


def stationary_line(args, cfg, r, dev, A, B):
    """Operand-stationary workload (the paper's Mode P for a dense operand):
    a fixed-scale plan keeps A's planes; each timed step deconstructs a new B
    (two B matrices alternate), then runs the residue GEMMs and the
    reconstruction."""
    import torch
    import paper_2606_06510_amd as oz
    m, k = A.shape
    n = B.shape[1]
    B2 = np.ascontiguousarray(B[:, ::-1])
    Ad = oz.to_device_colmajor(A, dev)
    Bds = [oz.to_device_colmajor(B, dev), oz.to_device_colmajor(B2, dev)]
    Cd = oz.colmajor_empty(m, n, device=dev)
    plan = oz.Plan(m, n, k, r, oz.OZ2_SCALE_FIXED, device=dev)
    plan.deconstruct(Ad, Bds[0])
    stream = torch.cuda.current_stream()

    def step(i, ev=None):
        if ev is not None:
            ev[0].record(stream)
        plan.deconstruct_b(Bds[i & 1])
        if ev is not None:
            ev[1].record(stream)
        plan.residue_gemm()
        if ev is not None:
            ev[2].record(stream)
        plan.reconstruct(Cd)
        if ev is not None:
            ev[3].record(stream)

    warmup = max(args.warmup, MIN_WARMUP)
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(warmup + i)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    # per-stage split from as many further, instrumented steps
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(warmup + args.steps + i, events[i])
    torch.cuda.synchronize()
    dec = float(np.mean([e[0].elapsed_time(e[1]) for e in events]))
    gem = float(np.mean([e[1].elapsed_time(e[2]) for e in events]))
    rec = float(np.mean([e[2].elapsed_time(e[3]) for e in events]))
    flop = 2.0 * m * n * k
    fp8_flop = 3 * r * flop
    achieved = fp8_flop / (gem * 1e-3) / 1e12
    Blast = B if ((warmup + 2 * args.steps - 1) & 1) == 0 else B2
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(A, Blast, r, Cd, min(args.cpu_sample or 256, 256), mode="fixed")
    print(json.dumps({
        "metric": "effective FP64 TFLOPS of emulated DGEMM, operand-stationary "
                  "(A's planes kept, fixed scaling)",
        "value": round(flop / (ms_step * 1e-3) / 1e12, 3), "unit": "TFLOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp8-e4m3 MFMA -> exact int -> f64", "data": "synthetic (seeded numpy PCG64)",
        "config": {"workload": f"{args.config} operand-stationary: C = A B_t, m={m} n={n} k={k}, "
                               f"r={r} moduli (alpha={3 * r}), new B each step",
                   "m": m, "n": n, "k": k, "num_moduli": r},
        "roofline": {"bound": "mfma",
                     "kernel": "k_resgemm (residue GEMMs, 3r FP8 products)",
                     "achieved": round(achieved, 2), "peak": FP8_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / FP8_PEAK_TFLOPS, 4),
                     "traffic": None},
        "stages_ms": {"deconstruct_b": round(dec, 4), "residue_gemm": round(gem, 4),
                      "reconstruct": round(rec, 4)},
        "cpu_baseline": cpu}))


def accuracy_sweep(A, B, dev):
    """Max componentwise error |C - AB| / (|A||B|) over 256 sampled outputs
    (exact error by compensated summation) for every moduli count."""
    import torch
    import paper_2606_06510_amd as oz
    from oracle import refgemm
    m, k = A.shape
    n = B.shape[1]
    rng = np.random.default_rng(4321)
    rows = rng.integers(0, m, 256)
    cols = rng.integers(0, n, 256)
    Ad = oz.to_device_colmajor(A, dev)
    Bd = oz.to_device_colmajor(B, dev)
    Cd = oz.colmajor_empty(m, n, device=dev)
    chart = {}
    for r in range(8, 17):
        plan = oz.Plan(m, n, k, r, 0, device=dev)
        plan.deconstruct(Ad, Bd)
        plan.residue_gemm()
        plan.reconstruct(Cd)
        torch.cuda.synchronize()
        C = oz.from_device_colmajor(Cd)[rows, cols]
        chart[r] = {"alpha": 3 * r + 1,
                    "max_componentwise_err": refgemm.componentwise_ratio(C, A, B, rows, cols)}
        del plan
    print(json.dumps({"accuracy_vs_moduli": chart, "sample": "256 random outputs",
                      "m": m, "n": n, "k": k}))


def batched_line(args, cfg, r, dev):
    """Strided-batched workload: one ozaki2_dgemm_strided_batched call per step."""
    import torch
    import synth
    import paper_2606_06510_amd as oz
    Ab, Bb = synth.make(args.config)
    nb, m, k = Ab.shape
    n = Bb.shape[2]
    Ad = torch.from_numpy(np.ascontiguousarray(Ab.transpose(0, 2, 1))).to(dev)
    Bd = torch.from_numpy(np.ascontiguousarray(Bb.transpose(0, 2, 1))).to(dev)
    Cd = torch.empty((nb, n, m), dtype=torch.float64, device=dev)

    def step():
        oz.ozaki2_dgemm_strided_batched(m, n, k, Ad, m, m * k, Bd, k, k * n, Cd, m, m * n, nb, r)

    warmup = max(args.warmup, MIN_WARMUP)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    flop = 2.0 * m * n * k * nb
    At = Ad.transpose(1, 2)
    Bt = Bd.transpose(1, 2)
    for _ in range(2):
        torch.bmm(At.contiguous(), Bt.contiguous())
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(5):
        torch.bmm(At.contiguous(), Bt.contiguous())
    torch.cuda.synchronize()
    native = flop / ((time.perf_counter() - t) / 5) / 1e12
    print(json.dumps({
        "metric": "effective FP64 TFLOPS of emulated DGEMM (Ozaki-II on FP8 MFMA)",
        "value": round(flop / (ms * 1e-3) / 1e12, 4), "unit": "TFLOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp8-e4m3 MFMA -> exact int -> f64", "data": "synthetic (seeded numpy PCG64)",
        "config": {"workload": f"{args.config}: {nb} strided-batched {m}x{n}x{k} products, r={r}",
                   "batch": nb, "m": m, "n": n, "k": k, "num_moduli": r},
        "native_fp64_tflops": round(native, 3)}))


def gemv_line(args, cfg, r, dev):
    """Batched GEMV Y = A X (the fused kernel of Alg. 2, fixed scaling): one
    ozaki2_gemv_batched call per step on resident inputs and a preallocated
    workspace; native FP64 torch.matmul on the same inputs beside it."""
    import torch
    import synth
    import paper_2606_06510_amd as oz
    A, X = synth.make(args.config)
    m, k = A.shape
    nrhs = X.shape[1]
    log(f"inputs of {args.config} drawn")
    Ad, Xd = oz.to_device_colmajor(A, dev), oz.to_device_colmajor(X, dev)
    Yd = oz.colmajor_empty(m, nrhs, device=dev)
    ws = torch.empty(oz.ozaki2_gemv_workspace_bytes(m, k, nrhs, r), dtype=torch.uint8, device=dev)
    warmup = max(args.warmup, MIN_WARMUP)

    def step():
        oz.gemv(Ad, Xd, num_moduli=r, Y=Yd, workspace=ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    flop = 2.0 * m * k * nrhs
    At = torch.from_numpy(np.ascontiguousarray(A)).to(dev)
    Xt = torch.from_numpy(np.ascontiguousarray(X)).to(dev)
    for _ in range(3):
        torch.matmul(At, Xt)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(20):
        torch.matmul(At, Xt)
    torch.cuda.synchronize()
    ms_native = (time.perf_counter() - t) * 1e3 / 20
    # operand-stationary A (an iterative method): each call after the first
    # reuses A's row scales from the workspace (OZ2_REUSE_A_SCALES)
    for _ in range(3):
        oz.gemv(Ad, Xd, num_moduli=r, Y=Yd, workspace=ws, flags=oz.OZ2_REUSE_A_SCALES)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(args.steps):
        oz.gemv(Ad, Xd, num_moduli=r, Y=Yd, workspace=ws, flags=oz.OZ2_REUSE_A_SCALES)
    torch.cuda.synchronize()
    ms_reuse = (time.perf_counter() - t) * 1e3 / args.steps
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        rng = np.random.default_rng(1234)
        rows = np.sort(rng.choice(m, size=min(args.cpu_sample or 512, m), replace=False))
        tc = time.perf_counter()
        res = oracle.dgemm(A, X, r, rows=rows, mode="fixed")
        dt = time.perf_counter() - tc
        Y = Yd.index_select(0, torch.as_tensor(rows, device=dev)).cpu().numpy()
        hi = host_info()
        cpu = {"value": round(2.0 * k * nrhs * len(rows) / dt / 1e12, 9), "unit": "TFLOPS",
               "cores": hi["cores"], "blas": hi["blas"], "cpu_model": hi["cpu_model"],
               "kind": "oracle", "sample": f"{len(rows)} sampled rows x {nrhs} columns, full k; "
                                           f"{dt:.2f} s",
               "sample_bitexact": f"{int(np.sum(Y.view(np.uint64) == res.C.view(np.uint64)))}/{Y.size}"}
    abytes = 8.0 * m * k
    print(json.dumps({
        "metric": "effective FP64 TFLOPS of the emulated batched GEMV (fused Ozaki-II, Alg. 2)",
        "value": round(flop / (ms * 1e-3) / 1e12, 4), "unit": "TFLOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp8-e4m3 MFMA -> exact int -> f64", "data": "synthetic (seeded numpy PCG64)",
        "config": {"workload": f"{args.config}: Y = A X, A {m}x{k}, {nrhs} right-hand sides, "
                               f"r={r} moduli, fixed scaling", "m": m, "k": k, "nrhs": nrhs,
                   "num_moduli": r},
        "operational_intensity_flop_per_byte": round(flop / abytes, 3),
        "a_stream_gbs": round(abytes / (ms * 1e-3) / 1e9, 1),
        "native_fp64_tflops": round(flop / (ms_native * 1e-3) / 1e12, 4),
        "native_ms": round(ms_native, 4),
        "emulated_over_native": round(ms_native / ms, 4),
        "reuse_a_scales": {"ms_per_call": round(ms_reuse, 4),
                           "tflops": round(flop / (ms_reuse * 1e-3) / 1e12, 4),
                           "over_native": round(ms_native / ms_reuse, 4)},
        "cpu_baseline": cpu}))


def plan_pstore(r):
    import paper_2606_06510_amd as oz
    ms = oz.ozaki2_moduli(r)
    return sum(2 if int(round(x ** 0.5)) ** 2 == x else 3 for x in ms)


def host_info():
    """Threads of the host BLAS, its name and version, and the CPU model: the
    oracle's products run on them."""
    cores, blas = os.cpu_count(), None
    try:
        from threadpoolctl import threadpool_info
        pools = [t for t in threadpool_info() if t.get("user_api") == "blas"] or threadpool_info()
        cores = max([t.get("num_threads", 1) for t in pools] + [1])
        if pools:
            blas = f"{pools[0].get('internal_api', '?')} {pools[0].get('version', '')}".strip()
    except Exception:  # pragma: no cover
        pass
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return {"cores": cores, "blas": blas, "cpu_model": model}


def cpu_baseline(A, B, r, Cd, nsamp, mode="bound", C_in=None):
    """The oracle, as it stands, on a bounded sample: nsamp sampled rows x nsamp
    sampled columns of the same workload (the scales of a sampled row need its
    code product against all of B, as the method does).  With C_in (C += A B)
    the device C must hold C_in + A B of one step."""
    import torch
    import oracle
    from oracle import refgemm
    import paper_2606_06510_amd as oz
    hi = host_info()
    m, k = A.shape
    n = B.shape[1]
    rng = np.random.default_rng(1234)
    rows = np.sort(rng.choice(m, size=min(nsamp, m), replace=False))
    cols = np.sort(rng.choice(n, size=min(nsamp, n), replace=False))
    t = time.perf_counter()
    res = oracle.dgemm(A, B, r, rows=rows, cols=cols, mode=mode, C_in=C_in)
    dt = time.perf_counter() - t
    C = Cd.index_select(0, torch.as_tensor(rows, device=Cd.device)).index_select(
        1, torch.as_tensor(cols, device=Cd.device)).cpu().numpy()
    same = int(np.sum(C.view(np.uint64) == res.C.view(np.uint64)))
    rr, cc = np.meshgrid(rows, cols, indexing="ij")
    # exact componentwise error on the first 1024 sampled entries (fsum per
    # entry) of the product itself (not defined for C_in + A B)
    ratio = None if C_in is not None else refgemm.componentwise_ratio(
        C.ravel()[:1024], A, B, rr.ravel()[:1024], cc.ravel()[:1024])
    return {"value": round(2.0 * k * len(rows) * len(cols) / dt / 1e12, 9), "unit": "TFLOPS",
            "cores": hi["cores"], "kind": "oracle", "blas": hi["blas"], "cpu_model": hi["cpu_model"],
            "sample": f"{len(rows)}x{len(cols)} output entries (sampled rows x cols) of the same "
                      f"workload, full k={k}; {dt:.2f} s",
            "sample_bitexact": f"{same}/{C.size}",
            "sample_max_componentwise_err": ratio,
            "sample_err_entries": min(1024, C.size)}


if __name__ == "__main__":
    main()
