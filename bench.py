#!/usr/bin/env python3
"""Throughput of the FP64 GEMM emulated on MI355X FP8 MFMA (Ozaki-II, CRT).

One step = one whole pass of the path over one batch of input already
resident in HBM: deconstruct (scan, max-magnitude code GEMM, scales, residue
planes) -> residue GEMMs -> reconstruction (+ fallback).  The default
workload is the 4096^3 GEMM with entries (u-0.5)*exp(0.5 g) at r = 12
moduli.  Prints ONE JSON line (rank 0, one GPU).

Extra fields beside the contract: per-stage times (HIP events on the launch
stream), the native FP64 DGEMM (torch.matmul float64) on the same inputs, and
the CPU oracle on a bounded sample of the same workload (with bit-parity and
exact-error checks of that sample).
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="gemm4096_lognormal")
    ap.add_argument("--moduli", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=16, help="sampled rows and columns")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs on exactly one GPU (the emulated GEMM is a "
              "single-GPU kernel path; see the sharding design notes). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2606_06510_amd as oz

    cfg = dict(synth.CONFIGS[args.config])
    r = args.moduli or cfg["r"]
    if cfg["kind"] in ("batched",):
        print("bench.py: the batched workload is not a bench line", file=sys.stderr)
        sys.exit(2)
    drawn = synth.make(args.config)
    A, B = drawn[0], drawn[1]
    m, k = A.shape
    n = B.shape[1]
    dev = torch.device("cuda:0")
    Ad = oz.to_device_colmajor(A, dev)
    Bd = oz.to_device_colmajor(B, dev)
    Cd = oz.colmajor_empty(m, n, device=dev)
    plan = oz.Plan(m, n, k, r, 0, device=dev)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        plan.deconstruct(Ad, Bd)
        if ev is not None:
            ev[1].record(stream)
        plan.residue_gemm()
        if ev is not None:
            ev[2].record(stream)
        plan.reconstruct(Cd)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    ms_step = (t1 - t0) * 1e3 / args.steps
    dec = float(np.mean([e[0].elapsed_time(e[1]) for e in events]))
    gem = float(np.mean([e[1].elapsed_time(e[2]) for e in events]))
    rec = float(np.mean([e[2].elapsed_time(e[3]) for e in events]))
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

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(A, B, r, Cd, args.cpu_sample)

    pm, pn, pk = [((x + 255) // 256) * 256 for x in (m, n)] + [((k + 127) // 128) * 128]
    out = {
        "metric": "effective FP64 TFLOPS of emulated DGEMM (Ozaki-II on FP8 MFMA)",
        "value": round(tflops, 3),
        "unit": "TFLOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8-e4m3 MFMA -> exact int -> f64",
        "data": "synthetic (seeded numpy PCG64)",
        "config": {"workload": f"{args.config}: C = A B, m={m} n={n} k={k}, "
                               f"{cfg['kind']} entries, r={r} moduli (alpha={3 * r + 1})",
                   "m": m, "n": n, "k": k, "num_moduli": r},
        "roofline": {"bound": "mfma", "kernel": "k_resgemm (residue GEMMs, 3r FP8 products)",
                     "achieved": round(achieved, 2), "peak": FP8_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / FP8_PEAK_TFLOPS, 4), "traffic": None},
        "stages_ms": {"deconstruct": round(dec, 4), "residue_gemm": round(gem, 4),
                      "reconstruct": round(rec, 4)},
        "fp8_mfma_util_residue_gemm": round(achieved / FP8_PEAK_TFLOPS, 4),
        "deconstruct_gbs_algorithmic": round(((m * k + k * n) * (8 + 1 + plan_pstore(r)))
                                             / (dec * 1e-3) / 1e9, 1),
        "reconstruct_gbs_algorithmic": round((m * n * (2 * r + 8)) / (rec * 1e-3) / 1e9, 1),
        "native_fp64_tflops": native if not isinstance(native, float) else round(native, 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


def plan_pstore(r):
    import paper_2606_06510_amd as oz
    ms = oz.ozaki2_moduli(r)
    return sum(2 if int(round(x ** 0.5)) ** 2 == x else 3 for x in ms)


def cpu_baseline(A, B, r, Cd, nsamp):
    """The oracle, as it stands, on a bounded sample: nsamp sampled rows x nsamp
    sampled columns of the same workload (the scales of a sampled row need its
    code product against all of B, as the method does)."""
    import oracle
    from oracle import refgemm
    import paper_2606_06510_amd as oz
    try:
        from threadpoolctl import threadpool_info
        cores = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count()
    m, k = A.shape
    n = B.shape[1]
    rng = np.random.default_rng(1234)
    rows = np.sort(rng.choice(m, size=min(nsamp, m), replace=False))
    cols = np.sort(rng.choice(n, size=min(nsamp, n), replace=False))
    t = time.perf_counter()
    res = oracle.dgemm(A, B, r, rows=rows, cols=cols)
    dt = time.perf_counter() - t
    C = oz.from_device_colmajor(Cd)[np.ix_(rows, cols)]
    same = int(np.sum(C.view(np.uint64) == res.C.view(np.uint64)))
    rr, cc = np.meshgrid(rows, cols, indexing="ij")
    ratio = refgemm.componentwise_ratio(C.ravel(), A, B, rr.ravel(), cc.ravel())
    return {"value": round(2.0 * k * len(rows) * len(cols) / dt / 1e12, 9), "unit": "TFLOPS",
            "cores": cores, "kind": "oracle",
            "sample": f"{len(rows)}x{len(cols)} output entries (sampled rows x cols) of the same "
                      f"workload, full k={k}; {dt:.2f} s",
            "sample_bitexact": f"{same}/{C.size}",
            "sample_max_componentwise_err": ratio}


if __name__ == "__main__":
    main()
