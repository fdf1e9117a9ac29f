"""Benchmark of the cross-validated kernel-machine path on one MI355X.

A step is one kmp_fit_path call over the whole hot path: Gram + fold gather,
per-fold factorisation, per-stage precompute, the batched (fold x lambda)
iterations and the finalize. The default workload is the smoothed-hinge SVM
with n = 10000, d = 100, sigma = median distance, 10-fold CV and 100 lambdas
in [1e-6, 1e1] (1000 cells; 9000 training points per fold), the largest
configuration whose timed steps fit a few minutes on one GPU. Inputs are
seeded synthetic data already resident in device memory.

Prints one JSON line: fits/sec (cells per second) over the timed steps, the
roofline of the dominant kernel class measured with HIP events on the
library's stream, a CPU baseline (the oracle, on a fixed sample of cells, in
a process pool on the host's cores), and, timed separately as context, one
call on the largest workload's unit of work (n = 40000, one bandwidth, 5 folds
of 32000 training points, 20 lambdas) and the same default workload in the
shared-factor exact-CV mode. Progress goes to stderr.
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


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="C3")
    ap.add_argument("--sigma-index", type=int, default=None,
                    help="time only this bandwidth of the workload (e.g. 1: sigma = median "
                         "distance for the five-bandwidth n = 40000 workload, one GPU's unit)")
    ap.add_argument("--shared", action="store_true",
                    help="time the shared-factor exact-CV mode instead of the per-fold mode")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=16,
                    help="oracle cells in the CPU baseline's fixed sample")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the separately timed context calls (largest unit, shared mode)")
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


# ------------------------------------------------------------ CPU baseline
def _host_facts():
    model, ram = None, None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal"):
                ram = f"{int(line.split()[1]) / 2 ** 20:.0f} GiB"
                break
    except OSError:
        pass
    return model, ram


def _oracle_cell(task):
    """One sampled cell: the fold's Gram blocks by direct differences and the
    oracle's cell solve, on one BLAS thread."""
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:
        pass
    import oracle
    from oracle import gram as OG
    X, y, fold, v, sigma, lam, loss, delta, tau = task
    t0 = time.perf_counter()
    Kv, Kc, T, H = OG.fold_blocks(X, fold, v, sigma)
    _, _, info = oracle.solve_cell(Kv, y[T], lam, loss, delta, tau)
    return time.perf_counter() - t0, bool(info["converged"])


def cpu_baseline(inp, w, ncells):
    """The oracle, untuned, on a fixed sample of the workload's cells: cell k
    is fold k mod V at lambda index L/4 + k (mod L), sigma 0, tau 0; each in
    its own process of a pool of min(16, usable cores) workers, one BLAS
    thread each (the oracle includes that fold's Gram blocks). Cells at the
    smallest lambdas take minutes each on the CPU and are left out of the
    sample, so the rate is, if anything, favourable to the CPU."""
    from concurrent.futures import ProcessPoolExecutor
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    workers = max(1, min(16, avail, ncells))
    tau = float(inp["taus"][0]) if w.loss == "check" else None
    delta = None if w.loss == "logistic" else 2.0 ** -6
    picks = [(k % w.V, (w.L // 4 + k) % w.L) for k in range(ncells)]
    tasks = [(inp["X"], inp["y"], inp["fold_id"], v, float(inp["sigmas"][0]),
              float(inp["lambdas"][l]), w.loss, delta, tau) for v, l in picks]
    t0 = time.perf_counter()
    with ProcessPoolExecutor(max_workers=workers) as ex:
        res = list(ex.map(_oracle_cell, tasks))
    wall = time.perf_counter() - t0
    model, ram = _host_facts()
    return {"value": ncells / wall, "unit": "fits/s", "cores": workers, "kind": "oracle",
            "sample": f"{ncells} cells of {w.name} (cell k: fold k mod {w.V}, lambda index "
                      f"{w.L // 4}+k mod {w.L}), each with its fold's Gram blocks, one per "
                      f"process in a pool of {workers} single-BLAS-thread workers; "
                      f"{wall:.1f} s wall, {sum(t for t, _ in res):.1f} s of cell time, "
                      f"all converged: {all(c for _, c in res)}",
            "cpu_model": model, "host_ram": ram, "host_cores_visible": avail}


# ---------------------------------------------------------------- roofline
# Kernel classes that run on the matrix cores. One of them is priced against
# the fp64 MFMA peak when its algorithmic intensity (flops per HBM byte) is
# above the ridge point of the two peaks, otherwise against HBM bandwidth;
# every other class is priced against HBM bandwidth.
MFMA_CLASSES = ("gemm_f", "gemm_zhat", "panel_wy", "trail_update", "q_form", "gram", "finalize")
RIDGE = FP64_PEAK_TFS * 1e12 / (HBM_PEAK_GBS * 1e9)


def roofline(kt, workload, name=None):
    """Roofline object of kernel class `name` (default: the dominant timed
    class, the largest estimated total time)."""
    if not kt:
        return None
    if name is None:
        name = max(kt, key=lambda k: kt[k][0] / kt[k][1] * kt[k][2])
    ms, launches, seen, nbytes, flops = kt[name][:5]
    sec = 1e-3 * ms
    common = {"kernel": name, "algorithmic_bytes_per_launch": nbytes / launches,
              "algorithmic_flops_per_launch": flops / launches,
              "avg_launch_us": 1e3 * ms / launches, "timed_launches": launches,
              "traffic": profiled_traffic(name, workload)}
    if name in MFMA_CLASSES:
        common["regimes"] = regimes(kt[name])
    if name in MFMA_CLASSES and nbytes > 0 and flops / nbytes >= RIDGE:
        achieved = flops / sec / 1e12
        return {"bound": "mfma", "achieved": achieved, "peak": FP64_PEAK_TFS, "unit": "TFLOP/s",
                "frac": achieved / FP64_PEAK_TFS, **common}
    achieved = nbytes / sec / 1e9
    return {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, **common}


def regimes(v):
    """The bracketed launches of one class split at the ridge point by their
    own algorithmic intensity, each part priced against its own roof: the
    launches above it against the fp64 matrix peak (flops), the others
    against HBM bandwidth (bytes)."""
    ms, launches, _, nbytes, flops, ms_mb, n_mb, bytes_mb, flops_mb = v
    out = {}
    if n_mb > 0 and ms_mb > 0:
        a = flops_mb / (1e-3 * ms_mb) / 1e12
        out["mfma"] = {"launches": n_mb, "ms": ms_mb, "achieved": a, "peak": FP64_PEAK_TFS,
                       "unit": "TFLOP/s", "frac": a / FP64_PEAK_TFS}
    if launches - n_mb > 0 and ms - ms_mb > 0:
        a = (nbytes - bytes_mb) / (1e-3 * (ms - ms_mb)) / 1e9
        out["hbm"] = {"launches": launches - n_mb, "ms": ms - ms_mb, "achieved": a,
                      "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": a / HBM_PEAK_GBS}
    return out


def sigma_batch_that_fits(km, w, inp, args, dev):
    """The largest number of bandwidths per batch whose workspace fits in
    90 % of the device memory free now (all of them when that fits)."""
    import torch
    free = torch.cuda.mem_get_info(dev)[0]
    S = len(inp["sigmas"])
    spec = km.kmp_default_spec(w.loss)
    if args.refit:
        spec.flags |= km.KMP_FLAG_REFIT
    if args.shared:
        spec.flags |= km.KMP_FLAG_SHARED_FACTOR
    n, d = inp["X"].shape
    Q = len(inp["taus"]) if w.loss == "check" else 1
    # the refit runs every cell on all n points: one fold (as PathRunner does)
    fold_id, V = (np.zeros(n, dtype=np.int32), 1) if args.refit else (inp["fold_id"], w.V)
    for sb in range(S, 0, -1):
        b = km.kmp_workspace_bytes(spec, n, d, len(inp["lambdas"]), fold_id, V, S, Q, sb)
        if 0 < b <= 0.9 * free:
            return sb
    return 1


def kernel_table(kt, steps):
    return {k: {"est_ms_per_step": v[0] / v[1] * v[2] / steps,
                "launches_per_step": v[2] / steps,
                "avg_launch_us": 1e3 * v[0] / v[1],
                "GB_per_s": v[3] / (1e-3 * v[0]) / 1e9 if v[0] else None,
                "TFLOP_per_s": v[4] / (1e-3 * v[0]) / 1e12 if v[0] else None}
            for k, v in kt.items()}


PHASES = ("gram_ms", "factor_ms", "precompute_ms", "path_ms", "finalize_ms")


def run_steps(runner, stream, steps, dev):
    """Times `steps` calls; returns (seconds, phase ms summed, kernel table)."""
    import torch
    phases = {k: 0.0 for k in PHASES}
    kt = {}
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for i in range(steps):
        runner.run(stream)
        for k in phases:
            phases[k] += getattr(runner.timings, k)
        for name, vals in runner.kernel_times().items():
            a = kt.setdefault(name, [0.0, 0, 0, 0.0, 0.0, 0.0, 0, 0.0, 0.0])
            for j, v in enumerate(vals):
                a[j] += v
        log(f"step {i + 1}/{steps} done")
    torch.cuda.synchronize(dev)
    return time.perf_counter() - t0, phases, kt


def context_call(name, inp, w, dev, stream, every, shared=False):
    """One separately timed call as context (no warm-up call of its own: the
    timed steps before it have loaded every kernel)."""
    import torch
    from paper_2606_06742_amd import kmpath as km
    runner = km.PathRunner(inp["X"], inp["y"], w.loss, inp["sigmas"], inp["lambdas"],
                           inp["fold_id"], w.V, taus=inp["taus"] if w.loss == "check" else None,
                           device=dev, shared=shared)
    runner.set_kernel_timing(km.KERNEL_CLASSES, every=every)
    sec, phases, kt = run_steps(runner, stream, 1, dev)
    res = runner.results()
    out = {"workload": name, "cells": runner.cells, "wall_s": sec, "fits_per_s": runner.cells / sec,
           "phases_ms": phases, "iterations": int(runner.timings.iterations),
           "all_converged": bool(np.all(res["status"] == 0)),
           "kernels": kernel_table(kt, 1), "dominant": roofline(kt, None),
           "gemm_f": roofline(kt, None, "gemm_f") if "gemm_f" in kt else None}
    del runner
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU (a multi-GPU run is not part "
                                   "of this build); --gpus must be 1",
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
    if args.sigma_index is not None:
        inp["sigmas"] = inp["sigmas"][args.sigma_index:args.sigma_index + 1]
    dev = torch.device("cuda:0")
    log(f"inputs of {w.name} ready")
    sb = sigma_batch_that_fits(km, w, inp, args, dev)
    runner = km.PathRunner(inp["X"], inp["y"], w.loss, inp["sigmas"], inp["lambdas"],
                           inp["fold_id"], w.V, taus=inp["taus"] if w.loss == "check" else None,
                           device=dev, refit=args.refit, shared=args.shared, sigma_batch=sb)
    # every kernel class is timed live in the timed region, one launch in
    # TIMING_EVERY bracketed by HIP events on the library's stream
    runner.set_kernel_timing(km.KERNEL_CLASSES, every=args.timing_every)
    stream = torch.cuda.current_stream(dev)
    for i in range(args.warmup):
        runner.run(stream)
        log(f"warmup {i + 1}/{args.warmup} done")
    torch.cuda.synchronize(dev)
    elapsed, phases, kt = run_steps(runner, stream, args.steps, dev)
    ms_step = 1e3 * elapsed / args.steps
    value = runner.cells * args.steps / elapsed
    res = runner.results()
    assert np.all(res["status"] == 0), "some cells did not converge"

    # the counter summaries are of the per-fold CV run: none matches another mode
    tag = (w.name + ("-refit" if args.refit else "") + ("-shared" if args.shared else "") +
           (f"-sigma{args.sigma_index}" if args.sigma_index is not None else ""))
    roof = roofline(kt, tag)
    metric = "(sigma x lambda) fits/sec for the full-data refit" if args.refit else METRIC
    nsig = len(inp["sigmas"])
    shape = (f"{nsig} sigmas x {w.L} lambdas on all {w.n} points"
             if args.refit else f"{nsig} sigmas x {w.V} folds x {w.L} lambdas")
    mode = "refit" if args.refit else ("shared-factor exact CV" if args.shared else "per-fold factors")
    out = {
        "metric": metric, "value": value, "unit": "fits/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.description}; n={w.n}, d={w.d}, {shape} = "
                               f"{runner.cells} cells, loss={w.loss}, {mode}",
                   "cells": runner.cells, "n": w.n, "d": w.d, "folds": 1 if args.refit else w.V,
                   "lambdas": w.L, "sigmas": nsig, "sigma_batch": sb, "mode": mode},
        "phases_ms_per_step": {k: v / args.steps for k, v in phases.items()},
        "path_fits_per_s": runner.cells / (1e-3 * (phases["precompute_ms"] + phases["path_ms"]
                                                   + phases["finalize_ms"]) / args.steps),
        "iterations_per_step": int(runner.timings.iterations),
        "cell_iterations_per_step": int(runner.timings.cell_iterations),
        "kernels": kernel_table(kt, args.steps),
        "kernel_timing": f"HIP events around 1 in {args.timing_every} launches of each class",
        "roofline": roof,
        "mfma_classes": {k: roofline(kt, tag, k) for k in ("gram", "gemm_f", "gemm_zhat", "q_form")
                         if k in kt},
        "cpu_baseline": None,
    }
    del runner
    torch.cuda.empty_cache()
    log(f"timed steps done: {value:.1f} fits/s")
    if not args.no_extra and not args.refit and not args.shared:
        w5 = W.get("C5")
        inp5 = W.make_inputs(w5)
        inp5["sigmas"] = inp5["sigmas"][1:2]          # sigma = 1 x median
        out["largest_unit"] = context_call("C5 unit: n=40000, d=28, sigma = median, 5 folds x 20 "
                                           "lambdas (100 cells, 32000 training points per fold)",
                                           inp5, w5, dev, stream, args.timing_every)
        log("largest unit done")
        out["shared_factor"] = context_call(f"{w.name} in the shared-factor exact-CV mode", inp, w,
                                            dev, stream, args.timing_every, shared=True)
        log("shared-factor call done")
    if not args.no_cpu_baseline and not args.refit:
        out["cpu_baseline"] = cpu_baseline(inp, w, args.cpu_sample)
        log("cpu baseline done")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
