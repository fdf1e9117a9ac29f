"""Writes the oracle-computed expected values the large GPU parity tests use.

Every value stored here comes from ``oracle/`` (cell solves, certificates,
selection) on the seeded inputs of ``workloads``; nothing is read from the
GPU library. The large workloads take minutes to hours of CPU time per cell
at their smallest penalties, which is why their expected values are stored
rather than recomputed by the tests.

Fixtures (numpy .npz, one per job):

* c3_cells.npz   smoothed-hinge workload n = 10000, d = 100, fold 0: the four
                 smallest penalties (1e-6 .. 2.3e-6) and three more across the
                 grid; noise-floor probe (the smallest penalty re-solved with
                 the norm-expansion Gram) on the first.
* c5_cells.npz   smoothed-hinge workload n = 40000, d = 28, sigma = 1 x median,
                 fold 0 (32000 training points): penalties 0, 5, 10, 19 of the
                 20-point grid; noise-floor probe on the smallest.
* c3_selection.npz, c2_selection.npz   the held-out loss sums of every cell
                 and the selected penalty per bandwidth (and the joint
                 (sigma, lambda) choice).

Per cell: the training-point coefficients alpha_T, beta, the optimal
intercept interval, the objective at delta = 2^-6, the held-out loss sum and
error count, the oracle's own KKT residual (extended precision), convergence
flag and certificate (duality gap, feasibility, zone counts).

Usage (from the repository root):
    python tests/golden/make_oracle_fixtures.py c3_cells c5_cells c3_selection c2_selection \\
        [--workers 4]
"""
from __future__ import annotations

import argparse
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as W  # noqa: E402
from oracle import gram as OG  # noqa: E402
from oracle import losses as OL  # noqa: E402

DELTA = 2.0 ** -6


def _limit_threads(n=1):
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(n)
    except Exception:
        pass


def _log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def solve_fold_cells(X, y, fold, v, sigma, lambdas, ls, loss, delta, tau=None, probe=(),
                     on_cell=None):
    """Oracle solves of cells ls of fold v; returns a dict of per-cell arrays
    (on_cell, if given, receives that dict after every cell)."""
    Kv, Kc, T, H = OG.fold_blocks(X, fold, v, sigma)
    yT, yH = y[T], y[H]
    out = {k: [] for k in ("l", "alpha_T", "beta", "beta_lo", "beta_hi", "objective", "cv_sum",
                           "cv_err", "kkt", "converged", "gap", "rel_gap", "box", "zone",
                           "noise_floor", "seconds")}
    for l in ls:
        lam = float(lambdas[l])
        t0 = time.time()
        a, b, info = oracle.solve_cell(Kv, yT, lam, loss, delta, tau)
        dt = time.time() - t0
        cert = oracle.certify_cell(Kv, yT, a, b, lam, loss, delta, tau)
        lo, hi = oracle.beta_interval(Kv, yT, a, b, loss, delta, tau)
        fH = Kc @ a + b
        floor = np.nan
        if l in probe:
            K2 = OG.rbf_gram_expansion(X[T], X[T], sigma)
            a2, _, _ = oracle.solve_cell(K2, yT, lam, loss, delta, tau)
            floor = float(np.abs(a2 - a).max() / np.abs(a).max())
            del K2
        out["l"].append(l)
        out["alpha_T"].append(a)
        out["beta"].append(b)
        out["beta_lo"].append(lo)
        out["beta_hi"].append(hi)
        out["objective"].append(oracle.objective(Kv, yT, a, b, lam, loss, delta, tau))
        out["cv_sum"].append(float(OL.eval_loss(loss, yH, fH, tau).sum()))
        out["cv_err"].append(int(np.count_nonzero(yH * fH <= 0.0)) if loss != "check" else 0)
        out["kkt"].append(info["kkt"])
        out["converged"].append(info["converged"])
        out["gap"].append(cert["gap"])
        out["rel_gap"].append(cert["rel_gap"])
        out["box"].append(cert["box"])
        out["zone"].append(cert["zone"])
        out["noise_floor"].append(floor)
        out["seconds"].append(dt)
        if on_cell is not None:
            on_cell({k: np.array(v) for k, v in out.items()})
        _log(f"fold {v} l={l} lambda={lam:.3e}: {dt:.0f} s, kkt {info['kkt']:.2e} "
             f"(fp64 loop {info['kkt_fp64']:.2e}), gap {cert['rel_gap']:.1e}, zone {cert['zone']}"
             f"{'' if np.isnan(floor) else f', noise floor {floor:.1e}'}")
    return {k: np.array(v) for k, v in out.items()}


def job_c3_cells(args):
    w = W.get("C3")
    inp = W.make_inputs(w)
    ls = (0, 1, 2, 3, 10, 45, 99)
    r = solve_fold_cells(inp["X"], inp["y"], inp["fold_id"], 0, inp["sigmas"][0],
                         inp["lambdas"], ls, "hinge", DELTA, probe=(0,))
    np.savez_compressed(os.path.join(HERE, "c3_cells.npz"), sigma=inp["sigmas"][0],
                        lambdas=inp["lambdas"], fold=0, delta=DELTA, **r)


def job_c5_cells(args):
    w = W.get("C5")
    X, y = W.make_data(w)
    fold = W.make_folds(w.n, w.V, w.fold_seed)
    lambdas = W.lambda_grid(w.lam_lo, w.lam_hi, w.L)
    _log("C5 median pairwise distance")
    med = W.median_pairwise_distance(X)
    sigma = 1.0 * med
    _log(f"sigma {sigma!r}")

    def save(r):
        np.savez_compressed(os.path.join(HERE, "c5_cells.npz"), sigma=sigma, sigma_median=med,
                            lambdas=lambdas, fold=0, delta=DELTA, **r)

    solve_fold_cells(X, y, fold, 0, sigma, lambdas, (19, 10, 5, 0), "hinge", DELTA,
                     probe=(0,) if args.probe_c5 else (), on_cell=save)


CACHE = os.path.join(ROOT, "_build", "fixture_cache")


def _sel_task(t):
    X, y, fold, v, sigma, lambdas, ls, loss, delta, tau, s, path = t
    if os.path.exists(path):                       # finished by an earlier run
        return s, v, dict(np.load(path, allow_pickle=False))
    r = solve_fold_cells(X, y, fold, v, sigma, lambdas, ls, loss, delta, tau)
    np.savez(path + ".tmp.npz", **r)
    os.replace(path + ".tmp.npz", path)
    return s, v, r


def _selection(name, loss, delta, chunks, workers):
    w = W.get(name)
    inp = W.make_inputs(w)
    S, V, L = len(inp["sigmas"]), w.V, w.L
    tasks = []
    # each task's cells are kept under _build/fixture_cache until the job
    # ends, so an interrupted job resumes where it stopped
    cache = os.path.join(CACHE, name)
    os.makedirs(cache, exist_ok=True)
    for s in range(S):
        for v in range(V):
            for c in range(chunks):
                ls = tuple(range(c, L, chunks))
                tasks.append((inp["X"], inp["y"], inp["fold_id"], v, float(inp["sigmas"][s]),
                              inp["lambdas"], ls, loss, delta, None, s,
                              os.path.join(cache, f"s{s}_v{v}_c{c}.npz")))
    # the longest tasks (smallest lambdas first in chunk 0) go first
    tasks.sort(key=lambda t: t[6][0])
    cv = np.zeros((S, V, L))
    err = np.zeros((S, V, L), dtype=np.int64)
    kkt = np.zeros((S, V, L))
    conv = np.zeros((S, V, L), dtype=bool)
    with ProcessPoolExecutor(max_workers=workers, initializer=_limit_threads) as ex:
        for s, v, r in ex.map(_sel_task, tasks):
            cv[s, v, r["l"]] = r["cv_sum"]
            err[s, v, r["l"]] = r["cv_err"]
            kkt[s, v, r["l"]] = r["kkt"]
            conv[s, v, r["l"]] = r["converged"]
    n = w.n
    sel = np.array([oracle.select(cv[s], inp["lambdas"], n)[0] for s in range(S)])
    joint = np.array(oracle.select_joint(cv, inp["lambdas"], inp["sigmas"], n))
    np.savez_compressed(os.path.join(HERE, f"{name.lower()}_selection.npz"), sigmas=inp["sigmas"],
                        lambdas=inp["lambdas"], cv_sum=cv, cv_err=err, kkt=kkt, converged=conv,
                        selected=sel, selected_joint=joint, delta=-1.0 if delta is None else delta)
    _log(f"{name}: selected {sel}, joint {joint}, worst oracle kkt {kkt.max():.2e}, "
         f"all converged {bool(conv.all())}")


def job_c3_selection(args):
    _selection("C3", "hinge", DELTA, 4, args.workers)


def job_c2_selection(args):
    _selection("C2", "logistic", None, 1, args.workers)


JOBS = {"c3_cells": job_c3_cells, "c5_cells": job_c5_cells, "c3_selection": job_c3_selection,
        "c2_selection": job_c2_selection}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("jobs", nargs="+", choices=sorted(JOBS))
    ap.add_argument("--workers", type=int, default=oracle.path.default_workers())
    ap.add_argument("--probe-c5", action="store_true",
                    help="also re-solve the smallest C5 penalty with the norm-expansion Gram")
    args = ap.parse_args()
    for j in args.jobs:
        _log(f"job {j}")
        JOBS[j](args)


if __name__ == "__main__":
    main()
