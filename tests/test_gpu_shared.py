"""Exact CV on one factor of the full kernel matrix per bandwidth
(KMP_FLAG_SHARED_FACTOR; Appendix A.2's exact cross-validation formula and
Algorithm 1's single decomposition), and exact leave-one-out CV (V = n).

The fold problem is solved as the n-point problem whose held-out points
carry no loss (the paper's Lemma 2): its minimiser is the fold solution
with zero coefficients on the held-out points. Bars as for the per-fold
path (objectives 1e-8 relative, coefficients 1e-6 of max |alpha|, intercepts
1e-6 or inside the oracle's interval, held-out sums 1e-6, selection equal),
against the oracle's per-fold solves and, cell by cell, against the
per-fold mode on the GPU.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_common import (ALPHA_RTOL, CV_RTOL, OBJ_RTOL, announce, compare_cells, device,
                              expected_selection, oracle_cells)

pytestmark = pytest.mark.gpu


def _gpu(inp, loss, shared, **spec):
    from paper_2606_06742_amd import kmpath as km
    device()
    taus = inp["taus"] if loss == "check" else None
    r = km.PathRunner(inp["X"], inp["y"], loss, inp["sigmas"], inp["lambdas"], inp["fold_id"],
                      inp["V"], taus=taus, device="cuda", shared=shared,
                      **{"max_iter": 50000, **spec})
    code = r.run()
    out = r.results()
    assert code == 0, code
    assert np.all(out["status"] == 0)
    return out


def _oracle(inp, loss):
    return oracle.fit_path(inp["X"], inp["y"], loss, inp["sigmas"], inp["lambdas"], inp["fold_id"],
                           inp["V"], taus=inp["taus"] if loss == "check" else None,
                           workers=oracle.path.default_workers())


def _modes_agree(a, b, what):
    """Lemma 2 on the GPU: shared-factor and per-fold results cell by cell."""
    rel = np.abs(a["objective"] - b["objective"]) / np.abs(b["objective"])
    assert rel.max() <= OBJ_RTOL, (what, "objective", rel.max())
    scale = np.abs(b["alpha"]).max(axis=-1, keepdims=True)
    ra = (np.abs(a["alpha"] - b["alpha"]) / scale).max()
    assert ra <= ALPHA_RTOL, (what, "alpha", ra)
    rc = np.abs(a["cv_sum"] - b["cv_sum"]) / np.maximum(1.0, np.abs(b["cv_sum"]))
    assert rc.max() <= CV_RTOL, (what, "cv", rc.max())
    assert np.array_equal(a["selected"], b["selected"]), (what, a["selected"], b["selected"])
    return float(rel.max()), float(ra), float(rc.max())


def test_shared_c1_full_parity_and_lemma2():
    """All 50 cells of the n = 200 smoothed-hinge workload against the
    oracle; the same cells from the per-fold mode."""
    inp = W.make_inputs(W.get("C1"))
    announce("shared factor C1 (hinge, n=200, 5 folds, 10 lambdas)")
    g = _gpu(inp, "hinge", True)
    o = _oracle(inp, "hinge")
    cv = np.array(o["cv_sum"])
    worst = compare_cells(g, o, inp, "hinge", cv_expected=cv)
    assert np.array_equal(g["selected"], expected_selection(o, cv, inp["lambdas"], inp["X"].shape[0]))
    p = _gpu(inp, "hinge", False)
    agree = _modes_agree(g, p, "C1")
    print("C1 shared worst", worst, "shared vs per-fold", agree, "iterations",
          g["timings"]["cell_iterations"], "per-fold", p["timings"]["cell_iterations"])


@pytest.mark.parametrize("loss", ["hinge", "logistic", "check"])
def test_shared_small_ragged(loss):
    """n = 203 with unequal folds (each column keeps its own n_v), two
    bandwidths, two tau levels for the check loss: every cell."""
    inp = W.small_problem(loss, 203, 5, seed=41, V=5, L=6, lam_lo=-4.0, lam_hi=0.5,
                          sigma_mults=(0.6, 1.5), taus=(0.25, 0.75))
    announce(f"shared factor ragged n=203 loss={loss}")
    g = _gpu(inp, loss, True)
    o = _oracle(inp, loss)
    cv = np.array(o["cv_sum"])
    worst = compare_cells(g, o, inp, loss, cv_expected=cv)
    assert np.array_equal(g["selected"], expected_selection(o, cv, inp["lambdas"], inp["X"].shape[0]))
    print(loss, "shared worst", worst)


def test_shared_c4_lemma2_sampled():
    """Kernel quantile regression at full size (n = 5000, 3 tau x 5 folds x
    40 lambdas = 600 columns on one factor of order 5000): every cell
    against the per-fold mode, eight cells against independent oracle
    solves."""
    w = W.get("C4")
    inp = W.make_inputs(w)
    announce("shared factor C4 (check, n=5000, 600 columns on one factor)")
    g = _gpu(inp, "check", True)
    p = _gpu(inp, "check", False)
    agree = _modes_agree(g, p, "C4")
    rng = np.random.default_rng(19)
    cells = sorted({(0, int(rng.integers(3)), int(rng.integers(w.V)), int(rng.integers(w.L)))
                    for _ in range(8)})
    o = oracle_cells(inp, "check", cells, g["alpha"].shape)
    worst = compare_cells(g, o, inp, "check", cells=cells)
    print("C4 shared vs per-fold", agree, "sampled worst", worst, "shared timings",
          {k: v for k, v in g["timings"].items() if not isinstance(v, list)},
          "per-fold", {k: v for k, v in p["timings"].items() if not isinstance(v, list)})


@pytest.mark.parametrize("loss", ["hinge", "logistic"])
def test_leave_one_out(loss):
    """Exact leave-one-out CV (Algorithm 1 as printed: V = n, one point held
    out per fold, every fold on the one factor): n = 64, 4 lambdas, 256
    (fold, lambda) columns, every cell against the oracle's fold solves."""
    inp = W.small_problem(loss, 64, 3, seed=23, V=5, L=4, lam_lo=-3.0, lam_hi=0.0)
    n = inp["X"].shape[0]
    inp["fold_id"] = np.arange(n, dtype=np.int32)
    inp["V"] = n
    announce(f"leave-one-out n=64 loss={loss}")
    g = _gpu(inp, loss, True)
    o = _oracle(inp, loss)
    cv = np.array(o["cv_sum"])
    worst = compare_cells(g, o, inp, loss, cv_expected=cv)
    assert np.array_equal(g["selected"], expected_selection(o, cv, inp["lambdas"], n))
    print(loss, "leave-one-out worst", worst, "selected", g["selected"].ravel())


def test_shared_c3_full_size():
    """The n = 10000 smoothed-hinge workload (10 folds x 100 lambdas = 1000
    columns on one factor of order 10000): the seven stored oracle cells of
    fold 0 (the four smallest lambdas among them), every cell's held-out sum
    against the oracle's, and the selected lambda."""
    from tests.gpu_common import check_selection, fixture, fixture_cells
    w = W.get("C3")
    inp = W.make_inputs(w)
    fx = fixture("c3_cells.npz")
    announce("shared factor C3 (hinge, n=10000, 1000 columns on one factor)")
    g = _gpu(inp, "hinge", True)
    print("C3 shared timings", {k: v for k, v in g["timings"].items() if not isinstance(v, list)},
          flush=True)
    T = np.flatnonzero(inp["fold_id"] != 0)
    o, cells = fixture_cells(fx, g["alpha"].shape, T)
    worst = compare_cells(g, o, inp, "hinge", cells=cells)
    sel = fixture("c3_selection.npz")
    cvw = check_selection(g, sel, w.n, "C3 shared")
    print("C3 shared fixture cells worst", worst, "all-cell held-out sums", cvw)
