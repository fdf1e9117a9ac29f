"""The oracle's exact hinge SVM (oracle.hinge), pinned without its own
algorithm: brute force over every L/E/R pattern at n <= 7, zero duality
gap against the hinge dual, and sklearn's SVC (libsvm) at C = 1/(2 n lambda)
(Appendix A.1, remark on the C parameterisation)."""
import itertools

import numpy as np
import pytest

import workloads as W
from oracle import gram
from oracle.hinge import hinge_dual, hinge_objective, solve_exact_hinge


def _rbf(X, s):
    d2 = ((X[:, None, :] - X[None, :, :]) ** 2).sum(-1)
    return np.exp(-d2 / (2 * s * s))


def _brute(K, y, lam):
    """Minimum of P over the consistent patterns (each point: a = 1 with
    u <= 1, a = 0 with u >= 1, or u = 1 with a in [0, 1])."""
    n = len(y)
    c = 1.0 / (2 * n * lam)
    best = None
    for pat in itertools.product((0, 1, 2), repeat=n):
        pat = np.array(pat)
        L, E = np.flatnonzero(pat == 0), np.flatnonzero(pat == 1)
        a = np.zeros(n)
        a[L] = 1.0
        if E.size == 0:
            continue
        m = E.size
        A = np.zeros((m + 1, m + 1))
        r = np.zeros(m + 1)
        A[:m, :m] = c * y[E][:, None] * K[np.ix_(E, E)] * y[E][None, :]
        A[:m, m] = y[E]
        A[m, :m] = y[E]
        r[:m] = 1 - c * y[E] * (K[np.ix_(E, L)] @ y[L])
        r[m] = -y[L].sum()
        if abs(np.linalg.det(A)) < 1e-12:
            continue
        sol = np.linalg.solve(A, r)
        a[E] = sol[:m]
        beta = sol[m]
        alpha = c * y * a
        u = y * (K @ alpha + beta)
        t = 1e-9
        if (a[E].min() < -t or a[E].max() > 1 + t or np.any(u[pat == 0] > 1 + t)
                or np.any(u[pat == 2] < 1 - t)):
            continue
        P = hinge_objective(K, y, alpha, beta, lam)
        if best is None or P < best[0] - 1e-12:
            best = (P, alpha, beta)
    return best


def test_exact_hinge_matches_brute_force():
    rng = np.random.default_rng(3)
    done = 0
    for trial in range(30):
        n = int(rng.integers(4, 8))
        X = rng.standard_normal((n, 2))
        y = np.where(rng.random(n) < 0.5, 1.0, -1.0)
        if abs(y.sum()) == n:
            y[0] = -y[0]
        lam = float(10 ** rng.uniform(-3, -1))
        K = _rbf(X, 1.0)
        ref = _brute(K, y, lam)
        if ref is None:
            continue
        a, b, info = solve_exact_hinge(K, y, lam)
        assert info["converged"], info
        P = hinge_objective(K, y, a, b, lam)
        assert abs(P - ref[0]) <= 1e-10 * max(1.0, ref[0]), (trial, P, ref[0])
        assert np.abs(a - ref[1]).max() <= 1e-8 * max(1.0, np.abs(ref[1]).max())
        done += 1
    assert done >= 15


def test_exact_hinge_zero_gap_and_feasibility_on_c1_fold():
    inp = W.make_inputs(W.get("C1"))
    K, _, T, _ = gram.fold_blocks(inp["X"], inp["fold_id"], 1, inp["sigmas"][0])
    y = inp["y"][T]
    n = y.size
    for lam in inp["lambdas"]:
        alpha, beta, info = solve_exact_hinge(K, y, lam)
        assert info["converged"], (lam, info)
        a = 2 * n * lam * y * alpha
        assert a.min() >= -1e-12 and a.max() <= 1 + 1e-12
        assert abs(y @ a) <= 1e-9 * n
        P = hinge_objective(K, y, alpha, beta, lam)
        assert abs(P - hinge_dual(K, y, a, lam)) <= 1e-12 * max(1.0, P)
        assert info["beta_lo"] - 1e-12 <= beta <= info["beta_hi"] + 1e-12


@pytest.mark.parametrize("lam", [1e-3, 1e-2, 0.1])
def test_exact_hinge_matches_libsvm(lam):
    from sklearn.svm import SVC
    inp = W.small_problem("hinge", 80, 2, seed=13)
    X, y = inp["X"], inp["y"]
    s = inp["sigmas"][0]
    K = gram.rbf_gram(X, X, s)
    n = len(y)
    alpha, beta, info = solve_exact_hinge(K, y, lam)
    assert info["converged"]
    svc = SVC(kernel="rbf", gamma=1.0 / (2 * s * s), C=1.0 / (2 * n * lam), tol=1e-12)
    svc.fit(X, y)
    a_svc = np.zeros(n)
    a_svc[svc.support_] = svc.dual_coef_[0]
    P = hinge_objective(K, y, alpha, beta, lam)
    P_svc = hinge_objective(K, y, a_svc, svc.intercept_[0], lam)
    assert P <= P_svc + 1e-9
    assert abs(P - P_svc) <= 1e-6 * P


def _intercept_interval_is_the_argmin(K, y, lam):
    """The hinge objective is convex in beta for fixed alpha: the reported
    interval is the set of optimal intercepts when the objective is flat on
    it and rises just outside it."""
    alpha, beta, info = solve_exact_hinge(K, y, lam)
    assert info["converged"]
    lo, hi = info["beta_lo"], info["beta_hi"]
    P = hinge_objective(K, y, alpha, beta, lam)
    assert lo - 1e-12 <= beta <= hi + 1e-12
    for b in (lo, hi, 0.5 * (lo + hi)):
        if np.isfinite(b):
            assert abs(hinge_objective(K, y, alpha, b, lam) - P) <= 1e-13 * max(1.0, P)
    e = 1e-6 * max(1.0, abs(beta))
    for b in (lo - e, hi + e):
        if np.isfinite(b):
            assert hinge_objective(K, y, alpha, b, lam) - P >= 1e-3 * e / y.size
    return info["E"], hi - lo


def test_intercept_interval_when_no_margin_point_is_free():
    # cells whose margin points all sit at a bound (a_i in {0, 1}) or whose
    # margin set is empty: the intercept is an interval, not a point
    seen = {"empty": 0, "bounded": 0}
    for name, ls in (("C1", None), ("H1", range(44, 50))):
        inp = W.make_inputs(W.get(name))
        K, _, T, _ = gram.fold_blocks(inp["X"], inp["fold_id"], 0, inp["sigmas"][0])
        y = inp["y"][T]
        for l in (ls if ls is not None else range(len(inp["lambdas"]))):
            ne, width = _intercept_interval_is_the_argmin(K, y, inp["lambdas"][l])
            if width > 0:
                seen["bounded" if ne else "empty"] += 1
    assert seen["empty"] >= 3 and seen["bounded"] >= 2, seen
