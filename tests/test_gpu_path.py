"""The whole CV path (kmp_fit_path) against the oracle, cell by cell.

Bars: objectives within 1e-8 relative, coefficients within 1e-6 of
max |alpha|, intercepts within 1e-6 (or inside the oracle's optimal
interval when the intercept is not unique), held-out loss sums within 1e-6,
selected lambda index identical.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from oracle import gram as OG
from tests.gpu_common import announce, compare_cells, device, expected_selection, kkt_of

pytestmark = pytest.mark.gpu


def _gpu(inp, loss, **spec):
    from paper_2606_06742_amd import kmpath as km
    device()
    taus = inp["taus"] if loss == "check" else None
    r = km.fit_path(inp["X"], inp["y"], loss, inp["sigmas"], inp["lambdas"], inp["fold_id"],
                    inp["V"], taus=taus, **{"max_iter": 20000, **spec})
    assert r["code"] == 0, r["code"]
    assert np.all(r["status"] == 0)
    return r


def _oracle(inp, loss):
    return oracle.fit_path(inp["X"], inp["y"], loss, inp["sigmas"], inp["lambdas"], inp["fold_id"],
                           inp["V"], taus=inp["taus"] if loss == "check" else None,
                           workers=oracle.path.default_workers())


def test_path_c1_full_parity():
    inp = W.make_inputs(W.get("C1"))
    announce("fit_path C1 (hinge, n=200, 5 folds, 10 lambdas)")
    g = _gpu(inp, "hinge")
    o = _oracle(inp, "hinge")
    cv = np.array(o["cv_sum"])
    worst = compare_cells(g, o, inp, "hinge", cv_expected=cv)
    assert np.array_equal(g["selected"], expected_selection(o, cv, inp["lambdas"], inp["X"].shape[0]))
    print("C1 worst relative errors", worst, "iterations", g["timings"]["cell_iterations"])


@pytest.mark.parametrize("loss", ["hinge", "logistic", "check"])
def test_path_small_ragged(loss):
    inp = W.small_problem(loss, 203, 5, seed=41, V=5, L=6, lam_lo=-4.0, lam_hi=0.5,
                          sigma_mults=(0.6, 1.5), taus=(0.25, 0.75))
    announce(f"fit_path ragged n=203 loss={loss}")
    g = _gpu(inp, loss)
    o = _oracle(inp, loss)
    cv = np.array(o["cv_sum"])
    worst = compare_cells(g, o, inp, loss, cv_expected=cv)
    assert np.array_equal(g["selected"], expected_selection(o, cv, inp["lambdas"], inp["X"].shape[0]))
    print(loss, "worst", worst)


@pytest.mark.parametrize("loss", ["hinge", "check"])
def test_path_global_solve(loss):
    """The banded solve with its working vector in device memory (taken
    above 8192 rows per fold, forced here at a small order) meets the same
    bars against the oracle as the LDS one. Its reductions run in another
    order, so the two agree to rounding, not bit for bit."""
    from paper_2606_06742_amd import kmpath as km
    inp = W.small_problem(loss, 203, 5, seed=43, V=5, L=6, lam_lo=-4.0, lam_hi=0.5,
                          sigma_mults=(0.8,), taus=(0.3, 0.6))
    announce(f"fit_path device-memory solve, ragged n=203 loss={loss}")
    b = _gpu(inp, loss, flags=km.KMP_FLAG_RESTART | km.KMP_FLAG_GLOBAL_SOLVE)
    o = _oracle(inp, loss)
    cv = np.array(o["cv_sum"])
    worst = compare_cells(b, o, inp, loss, cv_expected=cv)
    assert np.array_equal(b["selected"], expected_selection(o, cv, inp["lambdas"], inp["X"].shape[0]))
    print(loss, "device-memory solve worst", worst)


def test_path_deterministic():
    inp = W.small_problem("logistic", 150, 4, seed=5, V=3, L=5)
    announce("fit_path determinism, logistic n=150")
    a = _gpu(inp, "logistic")
    b = _gpu(inp, "logistic")
    for k in ("alpha", "beta", "objective", "cv_sum", "iters"):
        assert np.array_equal(a[k], b[k]), k


def test_path_c2_full_size_sampled():
    w = W.get("C2")
    inp = W.make_inputs(w)
    announce("fit_path C2 full size (logistic, n=2000, 3 sigmas, 50 lambdas)")
    g = _gpu(inp, "logistic")
    # every cell: stationarity of the returned solution under the oracle's K
    y, fold = inp["y"], inp["fold_id"]
    for s in range(3):
        for v in range(w.V):
            Kv, _, T, _ = OG.fold_blocks(inp["X"], fold, v, inp["sigmas"][s])
            for l in range(w.L):
                a = g["alpha"][s, 0, v, l][T]
                k = kkt_of(Kv, y[T], a, g["beta"][s, 0, v, l], inp["lambdas"][l], "logistic", None, None)
                assert k <= 1e-8, (s, v, l, k)
    # sampled cells against independent oracle solves
    cells = [(1, 0, 0, 0), (1, 0, 0, 17), (1, 0, 3, 49), (0, 0, 2, 0), (2, 0, 4, 30), (0, 0, 1, 8)]
    o = {k: np.zeros_like(g[k]) for k in ("alpha", "beta", "objective", "cv_sum", "cv_err")}
    o["beta_lo"] = np.zeros_like(g["beta"])
    o["beta_hi"] = np.zeros_like(g["beta"])
    for (s, q, v, l) in cells:
        Kv, Kc, T, H = OG.fold_blocks(inp["X"], fold, v, inp["sigmas"][s])
        lam = inp["lambdas"][l]
        a, b, info = oracle.solve_cell(Kv, y[T], lam, "logistic")
        o["alpha"][s, q, v, l][T] = a
        o["beta"][s, q, v, l] = o["beta_lo"][s, q, v, l] = o["beta_hi"][s, q, v, l] = b
        o["objective"][s, q, v, l] = oracle.objective(Kv, y[T], a, b, lam, "logistic")
        fH = Kc @ a + b
        o["cv_sum"][s, q, v, l] = oracle.losses.eval_loss("logistic", y[H], fH).sum()
        o["cv_err"][s, q, v, l] = np.count_nonzero(y[H] * fH <= 0)
    worst = compare_cells(g, o, inp, "logistic", cells=cells)
    print("C2 sampled worst", worst, g["timings"])


def test_path_rejects_bad_inputs():
    """Non-finite X or y and non +-1 labels are refused before any solve;
    a valid call afterwards still succeeds."""
    from paper_2606_06742_amd import kmpath as km
    device()
    inp = W.small_problem("hinge", 64, 3, seed=9, V=3, L=3)
    announce("fit_path input checks, hinge n=64")
    cases = []
    X = inp["X"].copy(); X[5, 1] = np.nan
    cases.append((X, inp["y"], km.KMP_ENONFINITE, "X"))
    y = inp["y"].copy(); y[7] = np.inf
    cases.append((inp["X"], y, km.KMP_ENONFINITE, "y"))
    y = inp["y"].copy(); y[2] = 0.5
    cases.append((inp["X"], y, km.KMP_EINVAL, "labels"))
    for Xc, yc, code, what in cases:
        with pytest.raises(km.KmpError) as e:
            km.fit_path(Xc, yc, "hinge", inp["sigmas"], inp["lambdas"], inp["fold_id"], inp["V"])
        assert e.value.code == code, (what, str(e.value))
    r = _gpu(inp, "hinge")
    assert np.all(np.isfinite(r["objective"]))


def test_path_c4_full_parity():
    """Kernel quantile regression at full size (n = 5000, 5 folds, 3 tau
    levels sharing each fold's factor, 40 lambdas): every one of the 600
    cells against the oracle."""
    w = W.get("C4")
    inp = W.make_inputs(w)
    announce("fit_path C4 full size (check, n=5000, 3 taus, 40 lambdas)")
    g = _gpu(inp, "check")
    o = _oracle(inp, "check")
    cv = np.array(o["cv_sum"])
    worst = compare_cells(g, o, inp, "check", cv_expected=cv)
    assert np.array_equal(g["selected"], expected_selection(o, cv, inp["lambdas"], inp["X"].shape[0]))
    print("C4 worst", worst, "iterations", g["timings"]["iterations"],
          g["timings"]["cell_iterations"])


def test_path_c3_full_size_sampled():
    """Smoothed-hinge SVM at full size (n = 10000, d = 100, 10 folds, 100
    lambdas in [1e-6, 1e1]; 9000 training points per fold).

    Every cell must converge. On fold 0, sampled cells are solved by the
    oracle and compared at the usual bars, and every cell's stationarity
    residual is measured under the oracle's kernel matrix. The GPU iterates
    to its tolerance on its own factorisation Q B Q' of its own Gram matrix,
    whose entries differ from the oracle's by a few N eps; through the loss
    curvature 1/(2 delta) that moves the residual by up to
    (1/(2 delta)) max_i sum_j |dK_ij| |alpha_j| <= (1/(2 delta)) 4 N eps
    ||alpha||_1, which is the allowance added to the tolerance."""
    w = W.get("C3")
    inp = W.make_inputs(w)
    announce("fit_path C3 full size (hinge, n=10000, d=100, 10 folds, 100 lambdas)")
    g = _gpu(inp, "hinge")
    print("C3 timings", {k: v for k, v in g["timings"].items() if not isinstance(v, list)}, flush=True)
    y, fold = inp["y"], inp["fold_id"]
    delta = 2.0 ** -6
    Kv, Kc, T, H = OG.fold_blocks(inp["X"], fold, 0, inp["sigmas"][0])
    n, N = T.size, int(np.ceil(T.size / 64) * 64)
    eps = np.finfo(float).eps
    worst = 0.0
    for l in range(w.L):
        a = g["alpha"][0, 0, 0, l][T]
        k = kkt_of(Kv, y[T], a, g["beta"][0, 0, 0, l], inp["lambdas"][l], "hinge", delta, None)
        bar = 2e-9 + (1.0 / (2.0 * delta)) * 4.0 * N * eps * np.abs(a).sum()
        assert k <= bar, (l, k, bar)
        worst = max(worst, k / bar)
    cells = [(0, 0, 0, l) for l in (10, 20, 45, 70, 99)]
    o = {k: np.zeros_like(g[k]) for k in ("alpha", "beta", "objective", "cv_sum", "cv_err")}
    o["beta_lo"] = np.zeros_like(g["beta"])
    o["beta_hi"] = np.zeros_like(g["beta"])
    for (s, q, v, l) in cells:
        lam = inp["lambdas"][l]
        a, b, info = oracle.solve_cell(Kv, y[T], lam, "hinge", delta)
        o["alpha"][s, q, v, l][T] = a
        o["beta"][s, q, v, l] = b
        o["beta_lo"][s, q, v, l], o["beta_hi"][s, q, v, l] = oracle.beta_interval(Kv, y[T], a, b, "hinge", delta, None)
        o["objective"][s, q, v, l] = oracle.objective(Kv, y[T], a, b, lam, "hinge", delta)
        fH = Kc @ a + b
        o["cv_sum"][s, q, v, l] = oracle.losses.eval_loss("hinge", y[H], fH).sum()
        o["cv_err"][s, q, v, l] = np.count_nonzero(y[H] * fH <= 0)
    worst_cells = compare_cells(g, o, inp, "hinge", cells=cells)
    print("C3 sampled worst", worst_cells, "stationarity / allowance", worst)


def test_path_h1_mixture_sampled():
    """The appendix's mixture-of-Gaussians simulation at n = 1000 (p = 10,
    5 folds, 50 lambdas, smoothed hinge): ten sampled cells against
    independent oracle solves."""
    from oracle.cell import beta_interval
    w = W.get("H1")
    inp = W.make_inputs(w)
    announce("fit_path H1 mixture (hinge, n=1000, 5 folds, 50 lambdas)")
    g = _gpu(inp, "hinge")
    y, fold, delta = inp["y"], inp["fold_id"], 2.0 ** -6
    rng = np.random.default_rng(5)
    cells = sorted({(0, 0, int(rng.integers(w.V)), int(rng.integers(w.L))) for _ in range(10)})
    o = {k: np.zeros_like(g[k]) for k in ("alpha", "beta", "objective", "cv_sum", "cv_err")}
    o["beta_lo"] = np.zeros_like(g["beta"])
    o["beta_hi"] = np.zeros_like(g["beta"])
    for (s, q, v, l) in cells:
        Kv, Kc, T, H = OG.fold_blocks(inp["X"], fold, v, inp["sigmas"][s])
        lam = inp["lambdas"][l]
        a, b, info = oracle.solve_cell(Kv, y[T], lam, "hinge", delta)
        o["alpha"][s, q, v, l][T] = a
        o["beta"][s, q, v, l] = b
        o["beta_lo"][s, q, v, l], o["beta_hi"][s, q, v, l] = beta_interval(Kv, y[T], a, b, "hinge", delta)
        o["objective"][s, q, v, l] = oracle.objective(Kv, y[T], a, b, lam, "hinge", delta)
        fH = Kc @ a + b
        o["cv_sum"][s, q, v, l] = oracle.losses.eval_loss("hinge", y[H], fH).sum()
        o["cv_err"][s, q, v, l] = np.count_nonzero(y[H] * fH <= 0)
    worst = compare_cells(g, o, inp, "hinge", cells=cells)
    print("H1 sampled worst", worst, g["timings"])
