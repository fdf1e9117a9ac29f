"""Seeded synthetic inputs for the cross-validated kernel-machine path.

This module is shared by the CPU oracle and the GPU library's harness, so it
holds no arithmetic of the method itself: only data generators, fold ids,
regularisation grids and the kernel bandwidth recipe (median pairwise
distance). Everything is deterministic given the seed.

Workloads C1..C5 follow the five synthetic configurations this project is
measured on (hinge, logistic and quantile losses; RBF kernels; V-fold CV;
log-spaced lambda grids). They stand in for the paper's own benchmark data
(Table 2 synthetic rows, the LIBSVM sets of Appendix B), which are not
reproduced here.

Fold assignment uses SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014) to drive a Fisher-Yates shuffle;
sample i of the shuffled order goes to fold (i mod V). It is integer-only so
that the C library's ``kmp_make_folds`` reproduces it bit for bit.
"""
from __future__ import annotations

import json
import os
from dataclasses import dataclass, field
from typing import Tuple

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "get", "splitmix64_next", "splitmix64_stream",
    "make_folds", "lambda_grid", "median_pairwise_distance", "make_data",
    "make_inputs", "small_problem",
]

_MASK64 = (1 << 64) - 1
_SM64_GAMMA = 0x9E3779B97F4A7C15
_SM64_M1 = 0xBF58476D1CE4E5B9
_SM64_M2 = 0x94D049BB133111EB


def splitmix64_next(state: int) -> Tuple[int, int]:
    """One SplitMix64 step: returns (new_state, output), both uint64 ints."""
    state = (state + _SM64_GAMMA) & _MASK64
    z = state
    z = ((z ^ (z >> 30)) * _SM64_M1) & _MASK64
    z = ((z ^ (z >> 27)) * _SM64_M2) & _MASK64
    return state, z ^ (z >> 31)


def splitmix64_stream(seed: int, count: int):
    """First ``count`` outputs of SplitMix64 seeded with ``seed``."""
    out = []
    s = seed & _MASK64
    for _ in range(count):
        s, v = splitmix64_next(s)
        out.append(v)
    return out


def make_folds(n: int, V: int, seed: int) -> np.ndarray:
    """Random V-fold assignment of n samples (int32 array of fold ids).

    Fisher-Yates from the top: for i = n-1 .. 1 draw j uniform on [0, i] as
    the high 64 bits of (SplitMix64 output) * (i + 1), swap perm[i], perm[j].
    Then fold[perm[i]] = i mod V, so fold sizes differ by at most one.
    """
    if n <= 0 or V <= 0:
        raise ValueError("n and V must be positive")
    perm = list(range(n))
    s = seed & _MASK64
    for i in range(n - 1, 0, -1):
        s, r = splitmix64_next(s)
        j = (r * (i + 1)) >> 64
        perm[i], perm[j] = perm[j], perm[i]
    fold = np.empty(n, dtype=np.int32)
    for i in range(n):
        fold[perm[i]] = i % V
    return fold


def lambda_grid(lo_exp: float, hi_exp: float, L: int) -> np.ndarray:
    """L values log-spaced on [10**lo_exp, 10**hi_exp] (increasing)."""
    return 10.0 ** np.linspace(lo_exp, hi_exp, L)


def median_pairwise_distance(X: np.ndarray) -> float:
    """Median of {||x_i - x_j|| : i < j}, distances by direct differences.

    For an even number of pairs this is the mean of the two middle order
    statistics. Squared distances are ranked (same order as distances) and
    the two middle ones are square-rooted before averaging.
    """
    X = np.ascontiguousarray(X, dtype=np.float64)
    n, d = X.shape
    N = n * (n - 1) // 2
    if N == 0:
        raise ValueError("need at least two points")
    out = np.empty(N, dtype=np.float64)
    pos = 0
    chunk = max(1, int(4_000_000 // max(1, n * d)))
    for i0 in range(0, n - 1, chunk):
        i1 = min(n - 1, i0 + chunk)
        for i in range(i0, i1):
            diff = X[i + 1:] - X[i]
            sq = np.einsum("ij,ij->i", diff, diff)
            out[pos:pos + sq.size] = sq
            pos += sq.size
    assert pos == N
    if N % 2 == 1:
        k = N // 2
        out.partition(k)
        return float(np.sqrt(out[k]))
    k = N // 2
    out.partition((k - 1, k))
    return float(0.5 * (np.sqrt(out[k - 1]) + np.sqrt(out[k])))


@dataclass(frozen=True)
class Workload:
    name: str
    loss: str                 # "hinge", "logistic" or "check"
    n: int
    d: int
    V: int
    L: int
    lam_lo: float             # log10 of smallest lambda
    lam_hi: float             # log10 of largest lambda
    sigma_mults: Tuple[float, ...]
    taus: Tuple[float, ...] = field(default=())
    index: int = 0            # k: data seed 1000+k, fold seed 2000+k
    description: str = ""

    @property
    def data_seed(self) -> int:
        return 1000 + self.index

    @property
    def fold_seed(self) -> int:
        return 2000 + self.index

    @property
    def cells(self) -> int:
        return len(self.sigma_mults) * max(1, len(self.taus)) * self.V * self.L


WORKLOADS = {
    "C1": Workload("C1", "hinge", 200, 10, 5, 10, -4.0, 1.0, (1.0,), (), 1,
                   "smoothed-hinge SVM, two Gaussian classes N(+-0.5*1, I), 100 each"),
    "C2": Workload("C2", "logistic", 2000, 50, 5, 50, -5.0, 1.0, (0.5, 1.0, 2.0), (), 2,
                   "kernel logistic, N(0,I) features, Bernoulli(sigmoid(sin x1 + x2 x3 + 0.5 x4))"),
    "C3": Workload("C3", "hinge", 10000, 100, 10, 100, -6.0, 1.0, (1.0,), (), 3,
                   "smoothed-hinge SVM, mean shift 0.3 in 20 coords, 10% label noise"),
    "C4": Workload("C4", "check", 5000, 20, 5, 40, -5.0, 0.0, (1.0,), (0.1, 0.5, 0.9), 4,
                   "kernel quantile, U(-1,1) features, heteroscedastic t3 noise"),
    "C5": Workload("C5", "hinge", 40000, 28, 5, 20, -6.0, 0.0, (0.5, 1.0, 2.0, 4.0, 8.0), (), 5,
                   "smoothed-hinge SVM, Gaussian + log-normal features, tanh-net labels"),
    # the mixture-of-Gaussians simulation of the paper's appendix (Fig. 1):
    # p = 10, 5-fold CV over 50 lambdas, n = 1000 and 10000
    "H1": Workload("H1", "hinge", 1000, 10, 5, 50, -5.0, 0.0, (1.0,), (), 6,
                   "smoothed-hinge SVM, two 10-centre Gaussian mixtures (mu = 2, sigma = 3)"),
    "H2": Workload("H2", "hinge", 10000, 10, 5, 50, -5.0, 0.0, (1.0,), (), 7,
                   "smoothed-hinge SVM, two 10-centre Gaussian mixtures (mu = 2, sigma = 3)"),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def make_data(w: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """(X, y) for workload w: X is n x d row-major float64, y float64."""
    rng = np.random.default_rng(w.data_seed)
    n, d = w.n, w.d
    if w.name == "C1":
        h = n // 2
        Xp = rng.standard_normal((h, d)) + 0.5
        Xn = rng.standard_normal((n - h, d)) - 0.5
        X = np.vstack([Xp, Xn])
        y = np.concatenate([np.ones(h), -np.ones(n - h)])
    elif w.name == "C2":
        X = rng.standard_normal((n, d))
        eta = np.sin(X[:, 0]) + X[:, 1] * X[:, 2] + 0.5 * X[:, 3]
        p = 1.0 / (1.0 + np.exp(-eta))
        u = rng.random(n)
        y = np.where(u < p, 1.0, -1.0)
    elif w.name == "C3":
        h = n // 2
        y0 = np.concatenate([np.ones(h), -np.ones(n - h)])
        X = rng.standard_normal((n, d))
        X[:, :20] += 0.15 * y0[:, None]
        flip = rng.choice(n, size=n // 10, replace=False)
        y = y0.copy()
        y[flip] = -y[flip]
    elif w.name == "C4":
        X = rng.uniform(-1.0, 1.0, size=(n, d))
        t = rng.standard_t(3, size=n)
        y = np.sin(2.0 * np.pi * X[:, 0]) + X[:, 1] ** 2 + (0.5 + np.abs(X[:, 2])) * t
    elif w.name == "C5":
        X = np.empty((n, d))
        X[:, :21] = rng.standard_normal((n, 21))
        X[:, 21:] = np.exp(0.5 * rng.standard_normal((n, d - 21)))
        H = 32
        W1 = rng.normal(0.0, np.sqrt(1.0 / d), size=(H, d))
        w2 = rng.normal(0.0, np.sqrt(1.0 / H), size=H)
        o = np.tanh(X @ W1.T) @ w2
        e = rng.normal(0.0, 0.5, size=n)
        y = np.where(o + e >= 0.0, 1.0, -1.0)
    elif w.name in ("H1", "H2"):
        # class means: mu on one half of the coordinates (first half for +1,
        # second for -1), zero elsewhere; ten centres per class drawn from
        # N(mean, I); a point takes one of its class's centres uniformly and
        # adds N(0, sigma I) with sigma = 3 read as the variance; half the
        # points in each class
        mu, var, K = 2.0, 3.0, 10
        half = d // 2
        mean_p = np.zeros(d)
        mean_p[:half] = mu
        mean_n = np.zeros(d)
        mean_n[half:] = mu
        cen_p = mean_p + rng.standard_normal((K, d))
        cen_n = mean_n + rng.standard_normal((K, d))
        h = n // 2
        Xp = cen_p[rng.integers(0, K, size=h)] + np.sqrt(var) * rng.standard_normal((h, d))
        Xn = cen_n[rng.integers(0, K, size=n - h)] + np.sqrt(var) * rng.standard_normal((n - h, d))
        X = np.vstack([Xp, Xn])
        y = np.concatenate([np.ones(h), -np.ones(n - h)])
    else:
        raise KeyError(w.name)
    return np.ascontiguousarray(X, dtype=np.float64), np.ascontiguousarray(y, dtype=np.float64)


MEDIANS_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "medians.json")


def stored_median(name: str):
    """The median pairwise distance of workload `name` as stored in
    medians.json (written by ``python -m workloads.make_medians``, which calls
    median_pairwise_distance on make_data's output), or None."""
    try:
        with open(MEDIANS_PATH) as fh:
            return float.fromhex(json.load(fh)[name])
    except (OSError, KeyError, ValueError):
        return None


def make_inputs(w: Workload, with_sigma: bool = True, stored: bool = True) -> dict:
    """All inputs of one workload: X, y, fold ids, lambdas, sigmas, taus.

    The bandwidths are multiples of the median pairwise distance; with
    stored=True the value stored for the workload is used when there is one
    (the n = 40000 workload's median takes minutes to recompute), else it is
    computed here."""
    X, y = make_data(w)
    fold = make_folds(w.n, w.V, w.fold_seed)
    lam = lambda_grid(w.lam_lo, w.lam_hi, w.L)
    out = {"X": X, "y": y, "fold_id": fold, "V": w.V, "lambdas": lam,
           "loss": w.loss, "taus": np.array(w.taus, dtype=np.float64)}
    if with_sigma:
        med = stored_median(w.name) if stored else None
        if med is None:
            med = median_pairwise_distance(X)
        out["sigma_median"] = med
        out["sigmas"] = np.array([m * med for m in w.sigma_mults])
    return out


def small_problem(loss: str, n: int, d: int, seed: int, V: int = 5,
                  L: int = 6, lam_lo: float = -3.0, lam_hi: float = 0.0,
                  sigma_mults=(1.0,), taus=(0.3, 0.7)) -> dict:
    """A small seeded problem of any size, for tests (ragged n allowed)."""
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d))
    if loss == "check":
        y = np.sin(2.0 * X[:, 0]) + 0.3 * rng.standard_normal(n)
        tau_arr = np.array(taus, dtype=np.float64)
    else:
        s = X[:, 0] + 0.5 * X[:, 1] ** 2 - 0.5 + 0.5 * rng.standard_normal(n)
        y = np.where(s >= 0.0, 1.0, -1.0)
        # keep both classes present in every training fold
        if np.all(y > 0) or np.all(y < 0):
            y[: n // 2] = -y[: n // 2]
        tau_arr = np.zeros(0)
    fold = make_folds(n, V, seed + 7)
    med = median_pairwise_distance(X)
    return {"X": np.ascontiguousarray(X), "y": np.ascontiguousarray(y),
            "fold_id": fold, "V": V, "lambdas": lambda_grid(lam_lo, lam_hi, L),
            "loss": loss, "taus": tau_arr, "sigma_median": med,
            "sigmas": np.array([m * med for m in sigma_mults])}
