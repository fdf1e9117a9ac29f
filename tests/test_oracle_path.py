"""The oracle's whole-path driver: layout, per-cell agreement, selection rule."""
import numpy as np
import pytest

import workloads as W
from oracle import cell, gram, losses as Ls, path


@pytest.mark.parametrize("loss", ["hinge", "logistic", "check"])
def test_fit_path_cells_and_layout(loss):
    inp = W.small_problem(loss, 47, 3, seed=31, V=3, L=4, sigma_mults=(0.7, 1.4), taus=(0.3, 0.8))
    X, y, fold, V = inp["X"], inp["y"], inp["fold_id"], inp["V"]
    lam = inp["lambdas"]
    r = path.fit_path(X, y, loss, inp["sigmas"], lam, fold, V, taus=inp["taus"])
    S, Q = len(inp["sigmas"]), (len(inp["taus"]) if loss == "check" else 1)
    assert r["alpha"].shape == (S, Q, V, len(lam), len(y))
    delta = None if loss == "logistic" else 2.0 ** -6
    for s in range(S):
        for q in range(Q):
            tau = inp["taus"][q] if loss == "check" else None
            for v in range(V):
                Kv, Kc, T, H = gram.fold_blocks(X, fold, v, inp["sigmas"][s])
                for l in range(len(lam)):
                    a = r["alpha"][s, q, v, l]
                    assert np.all(a[H] == 0.0)
                    assert cell.kkt_residual(Kv, y[T], a[T], r["beta"][s, q, v, l], lam[l], loss, delta, tau) <= 1e-11
                    F = cell.objective(Kv, y[T], a[T], r["beta"][s, q, v, l], lam[l], loss, delta, tau)
                    assert F == r["objective"][s, q, v, l]
                    fH = Kc @ a[T] + r["beta"][s, q, v, l]
                    assert r["cv_sum"][s, q, v, l] == pytest.approx(Ls.eval_loss(loss, y[H], fH, tau).sum(), rel=1e-14)
                    if loss != "check":
                        assert r["cv_err"][s, q, v, l] == np.count_nonzero(y[H] * fH <= 0)
            score = r["cv_sum"][s, q].sum(axis=0) / len(y)
            assert r["selected"][s, q] == int(np.argmin(score))


def test_selection_tie_breaks():
    lam = np.array([1e-3, 1e-2, 1e-1, 1.0])
    cv = np.array([[1.0, 0.5, 0.5, 2.0], [1.0, 0.5, 0.5, 2.0]])
    assert path.select(cv, lam, 10)[0] == 2                     # tie -> larger lambda
    assert path.select(cv, lam[::-1], 10)[0] == 1               # grid in decreasing order
    cvs = np.stack([cv, cv])                                    # two sigmas, identical scores
    assert path.select_joint(cvs, lam, np.array([1.0, 2.0]), 10) == (1, 2)
    cvs2 = cvs.copy()
    cvs2[0, :, 1] = 0.1
    assert path.select_joint(cvs2, lam, np.array([1.0, 2.0]), 10) == (0, 1)


def test_fit_path_process_pool_matches_serial():
    inp = W.small_problem("hinge", 40, 3, seed=17, V=4, L=3)
    args = (inp["X"], inp["y"], "hinge", inp["sigmas"], inp["lambdas"], inp["fold_id"], inp["V"])
    r1 = path.fit_path(*args)
    r2 = path.fit_path(*args, workers=2)
    for k in ("alpha", "beta", "objective", "cv_sum", "selected"):
        assert np.array_equal(r1[k], r2[k])
