"""Finite smoothing to the exact hinge SVM (KMP_FLAG_EXACT_HINGE; Appendix
A.1, Algorithm 1's outer loop): every cell's exact minimiser of eq.
(kernelsvm) on its fold against the oracle's (oracle.hinge, pinned by brute
force, zero duality gap and libsvm).

Bars: hinge objectives 1e-8 relative, coefficients 1e-6 of max |alpha|,
intercepts inside the oracle's optimal interval (a point when a point lies
on the margin) to 1e-6, held-out sums 1e-6 (at the GPU's intercept where the
intercept is an interval), status 0 (solution verified) for every cell.
"""
import numpy as np
import pytest

import workloads as W
from oracle import gram as OG
from oracle import losses as OL
from oracle.hinge import hinge_objective, solve_exact_hinge
from tests.gpu_common import ALPHA_RTOL, CV_RTOL, OBJ_RTOL, announce, device

pytestmark = pytest.mark.gpu


def _gpu(inp):
    from paper_2606_06742_amd import kmpath as km
    device()
    r = km.PathRunner(inp["X"], inp["y"], "hinge", inp["sigmas"], inp["lambdas"], inp["fold_id"],
                      inp["V"], device="cuda", exact_hinge=True, max_iter=20000)
    code = r.run()
    g = r.results()
    assert code == 0, code
    assert np.all(g["status"] == 0), np.argwhere(g["status"] != 0)[:5]
    return g


def _compare(g, inp, cells):
    X, y, fold = inp["X"], inp["y"], inp["fold_id"]
    worst = {"obj": 0.0, "alpha": 0.0, "cv": 0.0}
    blocks = {}
    for (s, v, l) in cells:
        if (s, v) not in blocks:
            blocks[(s, v)] = OG.fold_blocks(X, fold, v, inp["sigmas"][s])
        Kv, Kc, T, H = blocks[(s, v)]
        lam = inp["lambdas"][l]
        a, b, info = solve_exact_hinge(Kv, y[T], lam)
        assert info["converged"], ((s, v, l), info)
        Po = hinge_objective(Kv, y[T], a, b, lam)
        Pg = g["objective"][s, 0, v, l]
        assert abs(Pg - Po) <= OBJ_RTOL * Po, ((s, v, l), Pg, Po)
        ag = g["alpha"][s, 0, v, l]
        assert np.all(ag[H] == 0.0)
        err = np.abs(ag[T] - a).max()
        assert err <= ALPHA_RTOL * np.abs(a).max() + 1e-15, ((s, v, l), err)
        bg = g["beta"][s, 0, v, l]
        tol = ALPHA_RTOL * max(1.0, abs(b))
        assert info["beta_lo"] - tol <= bg <= info["beta_hi"] + tol, ((s, v, l), bg, info)
        co = float(OL.eval_loss("hinge", y[H], Kc @ a + bg).sum())
        cg = g["cv_sum"][s, 0, v, l]
        assert abs(cg - co) <= CV_RTOL * max(1.0, abs(co)), ((s, v, l), cg, co)
        worst["obj"] = max(worst["obj"], abs(Pg - Po) / Po)
        worst["alpha"] = max(worst["alpha"], err / np.abs(a).max())
        worst["cv"] = max(worst["cv"], abs(cg - co) / max(1.0, abs(co)))
    return worst


def test_exact_hinge_c1_all_cells():
    """The n = 200 workload, all 50 cells."""
    inp = W.make_inputs(W.get("C1"))
    announce("exact hinge C1 (n=200, 5 folds, 10 lambdas)")
    g = _gpu(inp)
    S, _, V, L = g["objective"].shape
    worst = _compare(g, inp, [(s, v, l) for s in range(S) for v in range(V) for l in range(L)])
    print("C1 exact hinge worst", worst, "finalize_ms", g["timings"]["finalize_ms"])


def test_exact_hinge_ragged_two_bandwidths():
    """Ragged n = 203 (unequal folds), two bandwidths, six lambdas."""
    inp = W.small_problem("hinge", 203, 5, seed=41, V=5, L=6, lam_lo=-4.0, lam_hi=0.5,
                          sigma_mults=(0.6, 1.5))
    announce("exact hinge ragged n=203, 2 sigmas")
    g = _gpu(inp)
    S, _, V, L = g["objective"].shape
    worst = _compare(g, inp, [(s, v, l) for s in range(S) for v in range(V) for l in range(L)])
    print("ragged exact hinge worst", worst)


def test_exact_hinge_h1_sampled():
    """The appendix's mixture at n = 1000 (5 folds, 50 lambdas): ten sampled
    cells (800 training points per fold)."""
    w = W.get("H1")
    inp = W.make_inputs(w)
    announce("exact hinge H1 (n=1000, 5 folds, 50 lambdas)")
    g = _gpu(inp)
    rng = np.random.default_rng(8)
    cells = sorted({(0, int(rng.integers(w.V)), int(rng.integers(w.L))) for _ in range(10)})
    worst = _compare(g, inp, cells)
    print("H1 exact hinge worst", worst, "finalize_ms", g["timings"]["finalize_ms"])
