"""The whole cross-validated regularisation path, one cell at a time.

Oracle (test infrastructure only). For every kernel bandwidth sigma, quantile
level tau (check loss only), fold v and lambda on the grid, the fold-restricted
problem of Appendix A.2 is solved independently from a cold start by
``oracle.cell.solve_cell`` at the final smoothing level delta. Then:

* alpha is scattered to length n with zeros on the held-out fold (the layout
  of the exact-CV formula, Appendix A.2);
* objective = F(alpha, beta) at delta (training loss, 1/n_v normalisation);
* cv_sum = sum over held-out points of the unsmoothed loss at
  f = K[H_v, T_v] alpha + beta, and cv_err counts y f <= 0 (classifiers);
* the selected index minimises sum_v cv_sum / n over lambda (the fold-wise
  validation losses of Appendix A.4, pooled), ties to the larger lambda;
  the joint (sigma, lambda) choice breaks ties by larger lambda, then larger
  sigma.
"""
from __future__ import annotations

import os
from concurrent.futures import ProcessPoolExecutor

import numpy as np

from . import losses as Ls
from .cell import objective, solve_cell, beta_interval
from .gram import fold_blocks


def _fold_task(args):
    X, y, loss, sigma, tau, lambdas, fold_id, v, delta, tol = args
    Kv, Kc, T, H = fold_blocks(X, fold_id, v, sigma)
    yT, yH = y[T], y[H]
    L = len(lambdas)
    n = y.shape[0]
    out = {"alpha": np.zeros((L, n)), "beta": np.zeros(L), "objective": np.zeros(L),
           "cv_sum": np.zeros(L), "cv_err": np.zeros(L, dtype=np.int64),
           "kkt": np.zeros(L), "converged": np.zeros(L, dtype=bool),
           "iters": np.zeros(L, dtype=np.int64),
           "beta_lo": np.zeros(L), "beta_hi": np.zeros(L)}
    for l, lam in enumerate(lambdas):
        a, b, info = solve_cell(Kv, yT, lam, loss, delta, tau, tol=tol)
        out["alpha"][l, T] = a
        out["beta"][l] = b
        out["objective"][l] = objective(Kv, yT, a, b, lam, loss, delta, tau)
        fH = Kc @ a + b
        out["cv_sum"][l] = Ls.eval_loss(loss, yH, fH, tau).sum()
        out["cv_err"][l] = int(np.count_nonzero(yH * fH <= 0.0)) if loss != "check" else 0
        out["kkt"][l] = info["kkt"]
        out["converged"][l] = info["converged"]
        out["iters"][l] = info["iters"]
        lo, hi = beta_interval(Kv, yT, a, b, loss, delta, tau)
        out["beta_lo"][l], out["beta_hi"][l] = lo, hi
    return out


def _limit_threads():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:
        pass


def select(cv_sum, lambdas, n):
    """argmin_l sum_v cv_sum[v, l]/n, ties to the larger lambda."""
    score = cv_sum.sum(axis=0) / n
    best = score.min()
    cand = np.flatnonzero(score == best)
    return int(cand[np.argmax(np.asarray(lambdas)[cand])]), score


def select_joint(cv_sum_s, lambdas, sigmas, n):
    """Joint (sigma, lambda) choice over cv_sum_s[s, v, l]; ties: larger lambda, then sigma."""
    score = cv_sum_s.sum(axis=1) / n            # [S, L]
    best = score.min()
    cands = [(lambdas[l], sigmas[s], s, l) for s, l in zip(*np.nonzero(score == best))]
    cands.sort()
    _, _, s, l = cands[-1]
    return int(s), int(l)


def fit_path(X, y, loss, sigmas, lambdas, fold_id, V, taus=None, delta=2.0 ** -6,
             tol=1e-13, workers=1):
    """All cells of the CV path. Arrays are indexed [sigma, tau, fold, lambda, ...]."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    y = np.ascontiguousarray(y, dtype=np.float64)
    fold_id = np.asarray(fold_id, dtype=np.int64)
    sigmas = np.atleast_1d(np.asarray(sigmas, dtype=np.float64))
    lambdas = np.asarray(lambdas, dtype=np.float64)
    tau_list = list(taus) if (loss == "check") else [None]
    if loss == "logistic":
        delta = None
    S, Q, L, n = len(sigmas), len(tau_list), len(lambdas), y.shape[0]
    tasks = [(X, y, loss, float(sigmas[s]), tau_list[q], lambdas, fold_id, v, delta, tol)
             for s in range(S) for q in range(Q) for v in range(V)]
    if workers > 1:
        with ProcessPoolExecutor(max_workers=workers, initializer=_limit_threads) as ex:
            results = list(ex.map(_fold_task, tasks))
    else:
        results = [_fold_task(t) for t in tasks]
    res = {k: np.stack([r[k] for r in results]).reshape((S, Q, V) + results[0][k].shape)
           for k in results[0]}
    res["selected"] = np.zeros((S, Q), dtype=np.int64)
    for s in range(S):
        for q in range(Q):
            res["selected"][s, q], _ = select(res["cv_sum"][s, q], lambdas, n)
    res["selected_joint"] = np.zeros((Q, 2), dtype=np.int64)
    for q in range(Q):
        res["selected_joint"][q] = select_joint(res["cv_sum"][:, q], lambdas, sigmas, n)
    return res


def default_workers(cap=16):
    """Worker processes for the cell pool: the usable cores, at most ``cap``."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(cap, n))
