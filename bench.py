"""Benchmark of the cross-validated kernel-machine path on one MI355X.

A step is one kmp_fit_path call over the whole hot path: Gram + fold gather,
per-fold factorisation, per-stage precompute, the batched (fold x lambda)
iterations and the finalize, for the kernel-logistic workload
(n = 2000, d = 50, sigma in {0.5, 1, 2} x median distance, 5-fold CV,
50 lambdas log-spaced in [1e-5, 1e1]: 750 cells). Inputs are seeded
synthetic data already resident in device memory.

Prints one JSON line: fits/sec (cells per second) over the timed steps, the
roofline of the dominant kernel measured with HIP events on the library's
stream, and a CPU baseline (the oracle, on a bounded sample of cells).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "(fold x lambda) fits/sec for full CV path; Gram+solver FP64 MFMA utilisation"
HBM_PEAK_GBS = 8000.0
FP64_PEAK_TFS = 78.6


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="C2")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-cells", type=int, default=48)
    ap.add_argument("--timing-every", type=int, default=16)
    ap.add_argument("--refit", action="store_true",
                    help="time the full-data refit of the workload instead (every sigma and "
                         "lambda on all n points); no CPU baseline, no counter traffic")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device-to-device three times (a plain copy of known "
                         "size, the reference for the HBM byte counters) and exit")
    return ap.parse_args()


def copy_calibration(mib):
    """Three plain device copies of `mib` MiB: under the counter profiler they
    give the FETCH_SIZE / WRITE_SIZE readings of a known byte count."""
    import torch
    dev = torch.device("cuda:0")
    n = mib * (1 << 20) // 8
    src = torch.ones(n, dtype=torch.float64, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize(dev)
    print(json.dumps({"copy_bytes_per_launch": n * 8, "launches": 3}), flush=True)


def profiled_traffic(kernel_class, workload):
    """HBM bytes per launch of `kernel_class` on `workload` from the committed
    counter summary profiles/pmc_<class>_<workload>.txt, or None when there is
    none or when a source file it lists has changed since the counters were
    taken (its recorded sha256 no longer matches)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"pmc_{kernel_class}_{workload}.txt")
    if not os.path.exists(path):
        return None
    traffic = None
    for line in open(path):
        parts = line.split()
        if len(parts) == 4 and parts[0] == "source" and parts[2] == "sha256":
            src = os.path.join(ROOT, parts[1])
            if not os.path.exists(src):
                return None
            if hashlib.sha256(open(src, "rb").read()).hexdigest() != parts[3]:
                return None
        elif len(parts) == 2 and parts[0] == "traffic_bytes_per_launch:":
            traffic = float(parts[1])
    return traffic


def cpu_baseline(inp, w, ncells):
    """The oracle, untuned, on a bounded sample of the workload's cells."""
    import oracle
    from oracle import gram as OG
    try:
        from threadpoolctl import threadpool_info
        cores = max([int(p.get("num_threads", 1)) for p in threadpool_info()] + [1])
    except Exception:
        cores = 1
    X, y, fold = inp["X"], inp["y"], inp["fold_id"]
    rng = np.random.default_rng(7)
    picks = sorted({(int(rng.integers(len(inp["sigmas"]))), int(rng.integers(w.V)),
                     int(rng.integers(w.L))) for _ in range(ncells)})
    tau = inp["taus"][0] if w.loss == "check" else None
    delta = None if w.loss == "logistic" else 2.0 ** -6
    t0 = time.perf_counter()
    blocks = {}
    for (s, v, l) in picks:
        if (s, v) not in blocks:
            blocks[(s, v)] = OG.fold_blocks(X, fold, v, inp["sigmas"][s])
        Kv, Kc, T, H = blocks[(s, v)]
        oracle.solve_cell(Kv, y[T], inp["lambdas"][l], w.loss, delta, tau)
    dt = time.perf_counter() - t0
    return {"value": len(picks) / dt, "unit": "fits/s", "cores": cores, "kind": "oracle",
            "sample": f"{len(picks)} random cells of {w.name} (sigma, fold, lambda drawn with "
                      f"seed 7), fold Gram blocks included, {dt:.1f} s"}


# Kernel classes that run on the matrix cores. One of them is priced against
# the fp64 MFMA peak when its algorithmic intensity (flops per HBM byte) is
# above the ridge point of the two peaks, otherwise against HBM bandwidth;
# every other class is priced against HBM bandwidth.
MFMA_CLASSES = ("gemm_f", "gemm_zhat", "panel_wy", "trail_update", "q_form", "gram")
RIDGE = FP64_PEAK_TFS * 1e12 / (HBM_PEAK_GBS * 1e9)


def roofline(kt, workload):
    """Roofline object of the dominant timed kernel class."""
    if not kt:
        return None
    # dominant = largest estimated total time (sampled mean x all launches)
    name = max(kt, key=lambda k: kt[k][0] / kt[k][1] * kt[k][2])
    ms, launches, seen, nbytes, flops = kt[name]
    sec = 1e-3 * ms
    if name in MFMA_CLASSES and nbytes > 0 and flops / nbytes >= RIDGE:
        achieved = flops / sec / 1e12
        return {"kernel": name, "bound": "mfma", "achieved": achieved, "peak": FP64_PEAK_TFS,
                "unit": "TFLOP/s", "frac": achieved / FP64_PEAK_TFS,
                "traffic": profiled_traffic(name, workload),
                "algorithmic_flops_per_launch": flops / launches,
                "avg_launch_us": 1e3 * ms / launches, "timed_launches": launches}
    achieved = nbytes / sec / 1e9
    return {"kernel": name, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": profiled_traffic(name, workload),
            "algorithmic_bytes_per_launch": nbytes / launches,
            "algorithmic_flops_per_launch": flops / launches,
            "avg_launch_us": 1e3 * ms / launches, "timed_launches": launches}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; --gpus must be 1",
                          "requested_gpus": args.gpus}))
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    import torch
    import workloads as W
    from paper_2606_06742_amd import kmpath as km

    w = W.get(args.workload)
    inp = W.make_inputs(w)
    dev = torch.device("cuda:0")
    runner = km.PathRunner(inp["X"], inp["y"], w.loss, inp["sigmas"], inp["lambdas"],
                           inp["fold_id"], w.V, taus=inp["taus"] if w.loss == "check" else None,
                           device=dev, refit=args.refit)
    # every kernel class is timed live in the timed region, one launch in
    # TIMING_EVERY bracketed by HIP events on the library's stream
    runner.set_kernel_timing(km.KERNEL_CLASSES, every=args.timing_every)
    stream = torch.cuda.current_stream(dev)
    for _ in range(args.warmup):
        runner.run(stream)
    torch.cuda.synchronize(dev)
    phases = {k: 0.0 for k in ("gram_ms", "factor_ms", "precompute_ms", "path_ms", "finalize_ms")}
    kt = {}
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        runner.run(stream)
        for k in phases:
            phases[k] += getattr(runner.timings, k)
        for name, (ms, cnt, seen, nbytes, flops) in runner.kernel_times().items():
            a = kt.setdefault(name, [0.0, 0, 0, 0.0, 0.0])
            a[0] += ms
            a[1] += cnt
            a[2] += seen
            a[3] += nbytes
            a[4] += flops
    torch.cuda.synchronize(dev)
    elapsed = time.perf_counter() - t0
    ms_step = 1e3 * elapsed / args.steps
    value = runner.cells * args.steps / elapsed
    res = runner.results()
    assert np.all(res["status"] == 0), "some cells did not converge"

    # the counter summaries are of the CV run: none matches a refit
    roof = roofline(kt, f"{w.name}-refit" if args.refit else w.name)
    metric = "(sigma x lambda) fits/sec for the full-data refit" if args.refit else METRIC
    shape = (f"{len(w.sigma_mults)} sigmas x {w.L} lambdas on all {w.n} points"
             if args.refit else f"{len(w.sigma_mults)} sigmas x {w.V} folds x {w.L} lambdas")
    out = {
        "metric": metric, "value": value, "unit": "fits/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{w.name}{' refit' if args.refit else ''}: {w.description}; "
                               f"n={w.n}, d={w.d}, {shape} = {runner.cells} cells, loss={w.loss}",
                   "cells": runner.cells, "n": w.n, "d": w.d, "folds": 1 if args.refit else w.V,
                   "lambdas": w.L, "sigmas": len(w.sigma_mults)},
        "phases_ms_per_step": {k: v / args.steps for k, v in phases.items()},
        "path_fits_per_s": runner.cells / (1e-3 * (phases["precompute_ms"] + phases["path_ms"]
                                                   + phases["finalize_ms"]) / args.steps),
        "iterations_per_step": int(runner.timings.iterations),
        "cell_iterations_per_step": int(runner.timings.cell_iterations),
        "kernels": {k: {"est_ms_per_step": v[0] / v[1] * v[2] / args.steps,
                        "launches_per_step": v[2] / args.steps,
                        "avg_launch_us": 1e3 * v[0] / v[1],
                        "GB_per_s": v[3] / (1e-3 * v[0]) / 1e9 if v[0] else None,
                        "TFLOP_per_s": v[4] / (1e-3 * v[0]) / 1e12 if v[0] else None}
                    for k, v in kt.items()},
        "kernel_timing": f"HIP events around 1 in {args.timing_every} launches of each class",
        "roofline": roof,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline and not args.refit:
        out["cpu_baseline"] = cpu_baseline(inp, w, args.cpu_sample_cells)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
