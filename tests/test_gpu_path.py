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
from tests.gpu_common import (announce, check_selection, compare_cells, device, expected_selection,
                              fixture, fixture_cells, kkt_of, oracle_cells)

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


@pytest.mark.parametrize("name", ["C1", "H1"])
def test_path_graph_replay_matches_eager(name):
    """Orders up to 2048 replay the iterations between polls from a recorded
    HIP graph (replayed many times per call, with the convergence polls and
    host waits between replays). Two graph runs must agree bit for bit, and
    with launches issued one by one (KMP_FLAG_EAGER) to the parity bars (the
    graph's split-K factor covers all columns, so the rounding differs)."""
    inp = W.make_inputs(W.get(name))
    announce(f"fit_path {name}: graph replay against eager launches")
    _gpu(inp, "hinge")                                   # warm-up (code objects, allocations)
    e = _gpu(inp, "hinge", eager=True)
    a = _gpu(inp, "hinge")
    b = _gpu(inp, "hinge")
    for k in ("alpha", "beta", "objective", "cv_sum", "cv_err", "iters", "status", "selected"):
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(a["selected"], e["selected"])
    assert np.abs(a["objective"] - e["objective"]).max() <= 1e-10 * np.abs(e["objective"]).max()
    amax = np.abs(e["alpha"]).max(axis=-1, keepdims=True)
    assert np.all(np.abs(a["alpha"] - e["alpha"]) <= 1e-7 * amax + 1e-300)
    assert np.abs(a["cv_sum"] - e["cv_sum"]).max() <= 1e-8 * max(1.0, np.abs(e["cv_sum"]).max())
    te, ta = e["timings"], a["timings"]
    print(f"{name}: path {te['path_ms']:.2f} ms eager ({te['iterations']} iterations, "
          f"{1e3 * te['path_ms'] / max(1, te['iterations']):.1f} us each), "
          f"{ta['path_ms']:.2f} ms graph ({ta['iterations']} iterations, "
          f"{1e3 * ta['path_ms'] / max(1, ta['iterations']):.1f} us each)")


def test_path_c2_full_size_sampled():
    """Kernel logistic regression at full size (n = 2000, 3 bandwidths,
    5 folds, 50 lambdas): every cell's stationarity under the oracle's K,
    six cells against independent oracle solves, every cell's held-out loss
    sum against the oracle's, the selected lambda per bandwidth and the joint
    (sigma, lambda) choice."""
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
    cells = [(1, 0, 0, 0), (1, 0, 0, 17), (1, 0, 3, 49), (0, 0, 2, 0), (2, 0, 4, 30), (0, 0, 1, 8)]
    o = oracle_cells(inp, "logistic", cells, g["alpha"].shape)
    worst = compare_cells(g, o, inp, "logistic", cells=cells)
    sel = fixture("c2_selection.npz")
    assert np.allclose(sel["sigmas"], inp["sigmas"], rtol=1e-14, atol=0)
    cvw = check_selection(g, sel, w.n, "C2")
    print("C2 sampled worst", worst, "all-cell held-out sums", cvw, "selected", g["selected"].ravel(),
          "joint", g["selected_joint"].ravel(), g["timings"])


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


def test_path_c3_full_size():
    """Smoothed-hinge SVM at full size (n = 10000, d = 100, 10 folds, 100
    lambdas in [1e-6, 1e1]; 9000 training points per fold, the device-memory
    solve).

    Every cell must converge. Seven cells of fold 0 (the four smallest
    lambdas, 1e-6 to 2.3e-6, where the fp64 sensitivity is largest, and
    three across the grid) are compared with stored oracle solves at the
    usual bars; every one of the 1000 cells' held-out loss sums is compared
    with the oracle's and the selected lambda must be the oracle's. The
    stored solves and sums come from tests/golden/make_oracle_fixtures.py
    (the smallest-lambda oracle solve takes minutes)."""
    from oracle.cell import residual_ext
    w = W.get("C3")
    inp = W.make_inputs(w)
    fx = fixture("c3_cells.npz")
    assert abs(fx["sigma"] - inp["sigmas"][0]) <= 1e-14 * inp["sigmas"][0]
    announce("fit_path C3 full size (hinge, n=10000, d=100, 10 folds, 100 lambdas)")
    g = _gpu(inp, "hinge")
    print("C3 timings", {k: v for k, v in g["timings"].items() if not isinstance(v, list)}, flush=True)
    T = np.flatnonzero(inp["fold_id"] != 0)
    o, cells = fixture_cells(fx, g["alpha"].shape, T)
    worst = compare_cells(g, o, inp, "hinge", cells=cells)
    print("C3 fixture cells", [c[3] for c in cells], "worst", worst,
          "oracle noise floor at lambda=1e-6", fx["noise_floor"][0], flush=True)
    sel = fixture("c3_selection.npz")
    cvw = check_selection(g, sel, w.n, "C3")
    # stationarity of every fold-0 cell under the oracle's K, evaluated in
    # extended precision (no fp64 evaluation floor)
    Kv, _, T, _ = OG.fold_blocks(inp["X"], inp["fold_id"], 0, inp["sigmas"][0])
    y = inp["y"]
    ks = [residual_ext(Kv, y[T], g["alpha"][0, 0, 0, l][T], g["beta"][0, 0, 0, l],
                       inp["lambdas"][l], "hinge", 2.0 ** -6)[3] for l in range(w.L)]
    print("C3 all-cell held-out sums worst", cvw, "fold-0 stationarity under the oracle's K:",
          "max", max(ks), "at l =", int(np.argmax(ks)))


def test_path_c5_unit():
    """Smoothed-hinge SVM at the largest size (n = 40000, d = 28, 5 folds of
    32000 training points, 20 lambdas in [1e-6, 1]), one bandwidth
    (sigma = median distance): the unit of work one GPU holds at its real
    shape. Fold-0 cells at lambda index 0, 5, 10 and 19 against stored oracle
    solves (hours of CPU time at the smallest lambda)."""
    w = W.get("C5")
    fx = fixture("c5_cells.npz")
    X, y = W.make_data(w)
    fold = W.make_folds(w.n, w.V, w.fold_seed)
    lam = W.lambda_grid(w.lam_lo, w.lam_hi, w.L)
    inp = {"X": X, "y": y, "fold_id": fold, "V": w.V, "lambdas": lam, "sigmas": np.array([float(fx["sigma"])]),
           "taus": np.zeros(0)}
    announce("fit_path C5 unit (hinge, n=40000, d=28, sigma=median, 5 folds, 20 lambdas)")
    g = _gpu(inp, "hinge")
    print("C5 unit timings", {k: v for k, v in g["timings"].items() if not isinstance(v, list)}, flush=True)
    T = np.flatnonzero(fold != 0)
    o, cells = fixture_cells(fx, g["alpha"].shape, T)
    worst = compare_cells(g, o, inp, "hinge", cells=cells)
    print("C5 fixture cells", [c[3] for c in cells], "worst", worst, "noise floor",
          fx["noise_floor"].tolist())


def test_path_h1_mixture_sampled():
    """The appendix's mixture-of-Gaussians simulation at n = 1000 (p = 10,
    5 folds, 50 lambdas, smoothed hinge): ten sampled cells against
    independent oracle solves."""
    w = W.get("H1")
    inp = W.make_inputs(w)
    announce("fit_path H1 mixture (hinge, n=1000, 5 folds, 50 lambdas)")
    g = _gpu(inp, "hinge")
    y, fold, delta = inp["y"], inp["fold_id"], 2.0 ** -6
    rng = np.random.default_rng(5)
    cells = sorted({(0, 0, int(rng.integers(w.V)), int(rng.integers(w.L))) for _ in range(10)})
    o = oracle_cells(inp, "hinge", cells, g["alpha"].shape, delta)
    worst = compare_cells(g, o, inp, "hinge", cells=cells)
    print("H1 sampled worst", worst, g["timings"])


def test_path_return_code_without_status_array():
    """The return code reports cells that stopped at max_iter, or whose
    iteration went non-finite, also when the caller passes no per-cell
    status array. The non-finite case is forced from the host with a valid
    but extreme penalty (lambda = 1e308: 2 lambda overflows, so the residual
    w = zhat + 2 lambda abar is NaN already at the zero start, where its other
    term 1'z is finite; the column is flagged and every kernel exits
    normally)."""
    import torch
    from paper_2606_06742_amd import kmpath as km
    device()
    inp = W.small_problem("hinge", 120, 4, seed=13, V=3, L=3)
    announce("fit_path return codes with status=NULL, hinge n=120")

    def call(lambdas, **spec):
        r = km.PathRunner(inp["X"], inp["y"], "hinge", inp["sigmas"], lambdas, inp["fold_id"],
                          inp["V"], device="cuda", **spec)
        code = km.kmp_fit_path(km._stream_ptr(None), r.spec, r.X, r.y, r.sigmas, r.taus, r.lambdas,
                               r.fold, r.V, r.workspace.data_ptr(), r.ws_bytes, r.alpha, r.beta,
                               r.objective, r.cv_sum, r.cv_err, None, None, None, None)
        torch.cuda.synchronize()
        return code

    assert call(inp["lambdas"]) == km.KMP_OK
    assert call(inp["lambdas"], max_iter=1) == km.KMP_WMAXITER
    lam = np.array([inp["lambdas"][0], 1e308, inp["lambdas"][-1]])
    assert call(lam) == km.KMP_ENONFINITE
