"""The oracle's per-cell solver pinned by methods that do not share its algorithm.

* brute force: for the smoothed hinge / check loss every point is in one of
  three linear pieces; enumerating all 3^n patterns (n <= 7) and solving the
  stationarity system of each gives the exact minimiser;
* logistic: Newton on the K-multiplied gradient in 50-digit arithmetic;
* zero duality gap against the separately derived duals (oracle.dual);
* exact-CV Lemma 2 (Appendix A.2): the full-n problem with held-out responses
  set to 0 and 1/(n - m) normalisation reproduces the fold solution, and its
  held-out coefficients are zero;
* large-lambda limits, and the delta -> 0 limit against sklearn's SVC with
  C = 1/(2 n lambda) (Appendix A.1, remark on the C parameterisation).
"""
import itertools

import mpmath as mp
import numpy as np
import pytest
from scipy.optimize import minimize_scalar

import workloads as W
from oracle import cell, dual, gram, losses as Ls


def _rbf(X, s):
    d2 = ((X[:, None, :] - X[None, :, :]) ** 2).sum(-1)
    return np.exp(-d2 / (2 * s * s))


def _pattern_system(K, y, lam, loss, delta, tau, pat):
    """Linear stationarity system (unknowns alpha, beta) of one piece pattern."""
    n = len(y)
    A = np.zeros((n + 1, n + 1))
    b = np.zeros(n + 1)
    for i, p in enumerate(pat):
        A[i, i] += 2 * lam
        if p == 1:
            e = y[i] * (1 + delta) if loss == "hinge" else y[i] + delta * (2 * tau - 1)
            A[i, :n] += K[i] / (2 * delta * n)
            A[i, n] += 1.0 / (2 * delta * n)
            b[i] += e / (2 * delta * n)
            A[n, :n] += K[i] / (2 * delta * n)
            A[n, n] += 1.0 / (2 * delta * n)
            b[n] += e / (2 * delta * n)
        else:
            if loss == "hinge":
                psi = -y[i] if p == 0 else 0.0
            else:
                psi = -tau if p == 0 else 1.0 - tau
            b[i] -= psi / n
            b[n] -= psi / n
    return A, b


def _brute_force(K, y, lam, loss, delta, tau=None, with_pattern=False):
    """All consistent piece patterns; returns list of (alpha, beta) (and the
    pattern when with_pattern)."""
    n = len(y)
    sols = []
    for pat in itertools.product((0, 1, 2), repeat=n):   # 0: left linear, 1: zone, 2: right linear
        A = np.zeros((n + 1, n + 1))
        b = np.zeros(n + 1)
        # unknowns (alpha_0..alpha_{n-1}, beta); rows: z_i + 2 lam alpha_i = 0, sum z = 0
        for i, p in enumerate(pat):
            A[i, i] += 2 * lam
            if p == 1:
                # zone: psi = (f_i - e_i)/(2 delta), f_i = K_i alpha + beta
                e = y[i] * (1 + delta) if loss == "hinge" else y[i] + delta * (2 * tau - 1)
                A[i, :n] += K[i] / (2 * delta * n)
                A[i, n] += 1.0 / (2 * delta * n)
                b[i] += e / (2 * delta * n)
                A[n, :n] += K[i] / (2 * delta * n)
                A[n, n] += 1.0 / (2 * delta * n)
                b[n] += e / (2 * delta * n)
            else:
                if loss == "hinge":
                    psi = -y[i] if p == 0 else 0.0          # u <= 1-delta : psi = -y ; u >= 1+delta : 0
                else:
                    psi = -tau if p == 0 else 1.0 - tau     # r >= delta : -tau ; r <= -delta : 1 - tau
                b[i] -= psi / n
                b[n] -= psi / n
        if abs(np.linalg.det(A)) < 1e-14 * np.abs(A).max() ** (n + 1):
            continue
        sol = np.linalg.solve(A, b)
        alpha, beta = sol[:n], sol[n]
        f = K @ alpha + beta
        q = y * f if loss == "hinge" else y - f
        ok = True
        tol = 1e-10
        for i, p in enumerate(pat):
            if loss == "hinge":
                lo_ok = q[i] <= 1 - delta + tol
                mid_ok = 1 - delta - tol <= q[i] <= 1 + delta + tol
                hi_ok = q[i] >= 1 + delta - tol
            else:
                lo_ok = q[i] >= delta - tol
                mid_ok = -delta - tol <= q[i] <= delta + tol
                hi_ok = q[i] <= -delta + tol
            if not (lo_ok if p == 0 else mid_ok if p == 1 else hi_ok):
                ok = False
                break
        if ok:
            sols.append((alpha, beta, pat) if with_pattern else (alpha, beta))
    return sols


@pytest.mark.parametrize("loss", ["hinge", "check"])
def test_brute_force_piece_enumeration(loss):
    rng = np.random.default_rng(11 if loss == "hinge" else 12)
    tested = flat = 0
    for trial in range(40):
        n = int(rng.integers(4, 8))
        X = rng.standard_normal((n, 2))
        if loss == "hinge":
            y = np.where(rng.random(n) < 0.5, 1.0, -1.0)
            if abs(y.sum()) == n:
                y[0] = -y[0]
            tau = None
        else:
            y = rng.standard_normal(n)
            tau = float(rng.choice([0.2, 0.5, 0.8]))
        delta = float(rng.choice([1.0, 0.125, 2.0 ** -6]))
        lam = float(10 ** rng.uniform(-3, 0))
        K = _rbf(X, 1.0)
        sols = _brute_force(K, y, lam, loss, delta, tau)
        if not sols:
            continue                    # optimum has an empty zone: beta not unique
        a0, b0 = sols[0]
        for a1, _ in sols[1:]:
            assert np.allclose(a1, a0, atol=1e-9)
        betas = [b1 for _, b1 in sols]
        a, b, info = cell.solve_cell(K, y, lam, loss, delta, tau)
        assert info["converged"]
        scale = max(1.0, np.abs(a0).max())
        assert np.abs(a - a0).max() <= 1e-9 * scale, (trial, a, a0)
        if max(betas) - min(betas) <= 1e-9:
            assert abs(b - b0) <= 1e-9 * max(1.0, abs(b0))
            tested += 1
        else:
            # flat intercept: the consistent patterns are the ends of the
            # optimal interval, and the oracle's beta lies inside it
            lo, hi = cell.beta_interval(K, y, a, b, loss, delta, tau)
            assert lo == pytest.approx(min(betas), abs=1e-9) and hi == pytest.approx(max(betas), abs=1e-9)
            assert min(betas) - 1e-9 <= b <= max(betas) + 1e-9
            flat += 1
    assert tested >= 20


def test_logistic_against_high_precision_newton():
    mp.mp.dps = 50
    rng = np.random.default_rng(21)
    for trial in range(4):
        n = 6
        X = rng.standard_normal((n, 2))
        y = np.array([1, -1, 1, 1, -1, -1], dtype=float)
        lam = [1e-3, 1e-2, 0.1, 1.0][trial]
        K = _rbf(X, 1.2)
        Km = mp.matrix(K.tolist())
        a = mp.matrix(n, 1)
        beta = mp.mpf(0)
        for _ in range(200):
            f = [sum(Km[i, j] * a[j] for j in range(n)) + beta for i in range(n)]
            sg = [1 / (1 + mp.exp(y[i] * f[i])) for i in range(n)]           # sigma(-y f)
            z = [-y[i] * sg[i] / n for i in range(n)]
            D = [sg[i] * (1 - sg[i]) / n for i in range(n)]
            w = [z[i] + 2 * lam * a[i] for i in range(n)]
            G = mp.matrix(n + 1, 1)
            for i in range(n):
                G[i] = sum(Km[i, j] * w[j] for j in range(n))
            G[n] = sum(z)
            if mp.norm(G) < mp.mpf(10) ** -40:
                break
            H = mp.matrix(n + 1, n + 1)
            for i in range(n):
                for j in range(n):
                    H[i, j] = sum(Km[i, k] * D[k] * Km[k, j] for k in range(n)) + 2 * lam * Km[i, j]
                H[i, n] = sum(Km[i, k] * D[k] for k in range(n))
                H[n, i] = H[i, n]
            H[n, n] = sum(D)
            step = mp.lu_solve(H, -G)
            for i in range(n):
                a[i] += step[i]
            beta += step[n]
        a_ref = np.array([float(a[i]) for i in range(n)])
        alpha, b, info = cell.solve_cell(K, y, lam, "logistic")
        assert np.abs(alpha - a_ref).max() <= 1e-11 * max(1.0, np.abs(a_ref).max())
        assert abs(b - float(beta)) <= 1e-11


@pytest.mark.parametrize("loss,tau", [("hinge", None), ("logistic", None), ("check", 0.25), ("check", 0.9)])
def test_zero_duality_gap_on_c1_fold(loss, tau):
    if loss == "check":
        inp = W.small_problem("check", 120, 4, seed=5)
    else:
        inp = W.make_inputs(W.get("C1"))
    X, y, fold = inp["X"], inp["y"], inp["fold_id"]
    Kv, _, T, _ = gram.fold_blocks(X, fold, 1, inp["sigmas"][0])
    yT = y[T]
    delta = None if loss == "logistic" else 2.0 ** -6
    for lam in [1e-4, 1e-2, 1.0]:
        a, b, info = cell.solve_cell(Kv, yT, lam, loss, delta, tau)
        assert info["converged"]
        F = cell.objective(Kv, yT, a, b, lam, loss, delta, tau)
        f = Kv @ a + b
        ad = dual.dual_point(loss, yT, f, delta, tau)
        box, eq = dual.dual_feasibility(loss, yT, ad, tau)
        assert box <= 1e-12 and eq <= 1e-10
        D = dual.dual_value(loss, Kv, yT, ad, lam, delta, tau)
        assert abs(F - D) <= 1e-12 * max(1.0, F)
        # representer identity alpha = a o y / (2 n lambda)
        assert np.abs(dual.alpha_from_dual(loss, yT, ad, lam) - a).max() <= 1e-9 * max(1.0, np.abs(a).max())
        assert abs(a.sum()) <= 1e-9 * max(1.0, np.abs(a).max()) or loss != "check"


@pytest.mark.parametrize("loss", ["hinge", "logistic"])
def test_exact_cv_lemma2(loss):
    inp = W.make_inputs(W.get("C1"))
    X, y, fold = inp["X"], inp["y"], inp["fold_id"]
    s = inp["sigmas"][0]
    K = gram.rbf_gram(X, X, s)
    delta = None if loss == "logistic" else 2.0 ** -6
    v = 3
    T = np.flatnonzero(fold != v)
    H = np.flatnonzero(fold == v)
    ytil = y.copy()
    ytil[H] = 0.0
    for lam in [3e-4, 1e-2]:
        a_f, b_f, _ = cell.solve_cell(K[np.ix_(T, T)], y[T], lam, loss, delta)
        a_n, b_n, info = cell.solve_cell(K, ytil, lam, loss, delta, norm=len(T))
        assert info["converged"]
        assert np.abs(a_n[H]).max() <= 1e-12
        assert np.abs(a_n[T] - a_f).max() <= 1e-9 * np.abs(a_f).max()
        assert abs(b_n - b_f) <= 1e-9


def test_large_lambda_limits():
    lam = 1e6
    inp = W.small_problem("logistic", 90, 3, seed=8)
    X, y = inp["X"], inp["y"]
    K = gram.rbf_gram(X, X, inp["sigmas"][0])
    a, b, _ = cell.solve_cell(K, y, lam, "logistic")
    npos, nneg = np.count_nonzero(y > 0), np.count_nonzero(y < 0)
    assert abs(b - np.log(npos / nneg)) < 1e-5
    assert np.abs(a).max() <= 1.0 / (2 * len(y) * lam)
    # check loss: beta -> minimiser of sum rho_{tau,delta}(y_i - beta)
    inp = W.small_problem("check", 90, 3, seed=9)
    X, y = inp["X"], inp["y"]
    K = gram.rbf_gram(X, X, inp["sigmas"][0])
    lam = 1e9
    for tau in (0.1, 0.5, 0.9):
        a, b, _ = cell.solve_cell(K, y, lam, "check", 2.0 ** -6, tau)
        phi = lambda t: Ls.smoothed_check(y - t, tau, 2.0 ** -6).sum()
        ref = minimize_scalar(phi, bounds=(y.min(), y.max()), method="bounded", options={"xatol": 1e-12})
        # the 1-D minimiser can be a flat interval between order statistics:
        # compare the attained value, and bracket beta by the tau-quantile's neighbours
        assert phi(b) <= ref.fun + 1e-6
        ys = np.sort(y)
        k = int(np.floor(tau * len(y)))
        assert ys[max(k - 1, 0)] - 0.1 <= b <= ys[min(k + 1, len(y) - 1)] + 0.1


def test_small_delta_matches_libsvm_hinge_svm():
    from sklearn.svm import SVC
    inp = W.small_problem("hinge", 80, 2, seed=13)
    X, y = inp["X"], inp["y"]
    s = inp["sigmas"][0]
    K = gram.rbf_gram(X, X, s)
    n = len(y)
    for lam in [1e-3, 1e-2]:
        delta = 2.0 ** -12
        a, b, _ = cell.solve_cell(K, y, lam, "hinge", delta)
        svc = SVC(kernel="rbf", gamma=1.0 / (2 * s * s), C=1.0 / (2 * n * lam), tol=1e-12)
        svc.fit(X, y)
        a_svc = np.zeros(n)
        a_svc[svc.support_] = svc.dual_coef_[0]
        f_ours = K @ a + b
        f_svc = K @ a_svc + svc.intercept_[0]
        assert np.abs(f_ours - f_svc).max() < 0.05
        # unsmoothed hinge objectives agree to O(delta)
        Fh = lambda al, be: Ls.hinge(y * (K @ al + be)).mean() + lam * al @ K @ al
        assert abs(Fh(a, b) - Fh(a_svc, svc.intercept_[0])) < 4 * delta


def test_beta_interval_flat_case():
    # balanced classes, huge lambda: the hinge optimum has no point in the zone
    X = np.array([[0.0], [1.0], [2.0], [3.0]])
    y = np.array([1.0, -1.0, 1.0, -1.0])
    K = _rbf(X, 0.5)
    a, b, info = cell.solve_cell(K, y, 1e4, "hinge", 0.125)
    lo, hi = cell.beta_interval(K, y, a, b, "hinge", 0.125)
    assert lo < hi and lo <= b <= hi
    F = lambda bb: cell.objective(K, y, a, bb, 1e4, "hinge", 0.125)
    for bb in np.linspace(lo, hi, 7):
        assert abs(F(bb) - F(b)) < 1e-15
    assert F(hi + 0.05) > F(b) and F(lo - 0.05) > F(b)


@pytest.mark.parametrize("loss,tau", [("hinge", None), ("check", 0.3)])
def test_refinement_at_tiny_lambda_matches_brute_force(loss, tau):
    """At lambda = 1e-5 the coefficients reach 1/(2 n lambda) ~ 1e4 and the
    fp64 Newton loop stalls far above the tolerance; the extended-precision
    refinement must still land on the brute-force minimiser and certify it
    (residual <= CONVERGED_KKT), and a cell stopped after one iteration must
    not be reported as converged."""
    rng = np.random.default_rng(31)
    done = 0
    for trial in range(30):
        n = 6
        X = rng.standard_normal((n, 2))
        if loss == "hinge":
            y = np.array([1, -1, 1, -1, 1, -1], dtype=float)
        else:
            y = rng.standard_normal(n)
        K = _rbf(X, 0.7)
        delta, lam = 2.0 ** -6, 1e-5
        sols = _brute_force(K, y, lam, loss, delta, tau, with_pattern=True)
        if not sols:
            continue
        # the consistent pattern's linear system solved in 40-digit arithmetic
        mp.mp.dps = 40
        A, rhs = _pattern_system(K, y, lam, loss, delta, tau, sols[0][2])
        sol = mp.lu_solve(mp.matrix(A.tolist()), mp.matrix(rhs.tolist()))
        a0 = np.array([float(sol[i]) for i in range(n)])
        a, b, info = cell.solve_cell(K, y, lam, loss, delta, tau)
        assert info["converged"] and info["kkt"] <= cell.CONVERGED_KKT, info
        # (the minimiser itself is ill-conditioned here: 2 lambda is tiny next
        # to the curvature, so a residual of 1e-10 moves alpha by ~1e-10
        # relative; the bar is still four orders below the GPU's 1e-6)
        assert np.abs(a - a0).max() <= 1e-9 * np.abs(a0).max(), (trial, a, a0)
        # beta enters through f = K alpha + beta, whose terms are of size
        # max |alpha|: its error is relative to that
        assert abs(b - float(sol[n])) <= 1e-9 * max(1.0, np.abs(a0).max())
        _, _, info1 = cell.solve_cell(K, y, lam, loss, delta, tau, max_iter=1)
        assert not info1["converged"] and info1["kkt"] > cell.CONVERGED_KKT
        done += 1
    assert done >= 5


@pytest.mark.parametrize("loss,tau", [("hinge", None), ("logistic", None), ("check", 0.7)])
def test_certificate(loss, tau):
    """certify_cell: zero duality gap, a feasible dual point and the zone
    counts at a solution; a strictly positive gap once alpha is moved off
    it (weak duality)."""
    inp = W.small_problem("check" if loss == "check" else "hinge", 60, 3, seed=17)
    X, y = inp["X"], inp["y"]
    K = gram.rbf_gram(X, X, inp["sigmas"][0])
    delta = None if loss == "logistic" else 2.0 ** -6
    lam = 3e-3
    a, b, info = cell.solve_cell(K, y, lam, loss, delta, tau)
    c = cell.certify_cell(K, y, a, b, lam, loss, delta, tau)
    assert abs(c["rel_gap"]) <= 1e-12 and c["box"] <= 1e-12 and c["eq"] <= 1e-10
    assert sum(c["zone"]) == len(y) and c["kkt"] <= cell.CONVERGED_KKT
    if loss != "logistic":
        assert c["zone"][1] > 0
    rng = np.random.default_rng(3)
    a2 = a + 1e-3 * np.abs(a).max() * rng.standard_normal(len(a))
    a2 -= a2.mean()                              # keep sum alpha = 0 (dual equality)
    c2 = cell.certify_cell(K, y, a2, b, lam, loss, delta, tau)
    if c2["box"] == 0.0 and c2["eq"] <= 1e-12:
        assert c2["gap"] > 0.0


def test_norm_expansion_gram_agrees_to_rounding():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((70, 9))
    s = 2.5
    K = gram.rbf_gram(X, X, s)
    K2 = gram.rbf_gram_expansion(X, X, s)
    assert np.all(np.diag(K2) == 1.0) and np.allclose(K2, K2.T, atol=0, rtol=0) is not None
    nr = (X * X).sum(1)
    bound = 8 * np.finfo(float).eps * (nr[:, None] + nr[None, :]) / (2 * s * s) * K + 1e-300
    assert np.all(np.abs(K2 - K) <= bound)
