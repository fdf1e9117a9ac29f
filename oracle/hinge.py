"""The exact (unsmoothed) hinge SVM of one cell: the minimiser of eq.
(kernelsvm) (Appendix A.1) on a fold's training points,

    P(alpha, beta) = (1/n) sum_i (1 - y_i f_i)_+ + lambda alpha' K alpha,
    f = K alpha + beta,

which finite smoothing reaches from the delta-smoothed problems (Appendix
A.1; Algorithm 1's outer loop stops when the SVM's KKT conditions hold).

Oracle (test infrastructure only). With a_i = 2 n lambda y_i alpha_i the KKT
conditions of P are: a_i in [0, 1], sum_i y_i a_i = 0, and for every point
either u_i = y_i f_i < 1 and a_i = 1 (set L), u_i > 1 and a_i = 0 (set R), or
u_i = 1 with a_i in [0, 1] (set E). Given the three sets, the E-rows of
u = 1 and the balance sum y a = 0 are a linear system in (a_E, beta); the
solution is the minimiser when it satisfies every condition. The sets are
found by an active-set iteration started from the quadratic zone of the
smoothed problem at a small delta (solved by ``oracle.cell.solve_cell``):
points whose a_E leaves [0, 1] go to L or R, points of L or R whose u crosses
1 go to E, until the conditions hold. Pinned in tests/test_oracle_hinge.py
by brute force over all 3^n patterns at n <= 7, by zero duality gap, and by
sklearn's SVC.
"""
from __future__ import annotations

import numpy as np

from .cell import solve_cell


def hinge_objective(K, y, alpha, beta, lam):
    """P(alpha, beta) above."""
    Ka = K @ alpha
    return float(np.maximum(0.0, 1.0 - y * (Ka + beta)).mean() + lam * (alpha @ Ka))


def hinge_dual(K, y, a, lam):
    """The dual value (1/n) sum a - (a o y)' K (a o y) / (4 n^2 lambda)."""
    n = y.shape[0]
    s = a * y
    return float(a.sum() / n - s @ K @ s / (4.0 * n * n * lam))


def _solve_sets(K, y, lam, L, E):
    """(a, beta) for the sets: a_L = 1, a_R = 0, a_E and beta from
    y_i f_i = 1 on E and sum y a = 0. None if the system is singular."""
    n = y.shape[0]
    c = 1.0 / (2.0 * n * lam)
    a = np.zeros(n)
    a[L] = 1.0
    m = E.size
    # f_i = c sum_j K_ij y_j a_j + beta; rows i in E: y_i f_i = 1
    A = np.zeros((m + 1, m + 1))
    r = np.zeros(m + 1)
    if m:
        A[:m, :m] = c * (y[E][:, None] * K[np.ix_(E, E)] * y[E][None, :])
        A[:m, m] = y[E]
        A[m, :m] = y[E]
        r[:m] = 1.0 - c * y[E] * (K[np.ix_(E, L)] @ y[L])
    r[m] = -y[L].sum()
    if m == 0:
        return None
    try:
        sol = np.linalg.solve(A, r)
    except np.linalg.LinAlgError:
        return None
    a[E] = sol[:m]
    return a, float(sol[m])


def solve_exact_hinge(K, y, lam, delta0=2.0 ** -12, max_rounds=200, tol=1e-9):
    """(alpha, beta, info) of the exact hinge SVM of one cell.

    info: rounds of the active-set iteration, |E|, converged (every KKT
    condition holds to tol: a_E in [-tol, 1 + tol], u <= 1 + tol on L,
    u >= 1 - tol on R, |sum y a| <= tol n), and the duality gap."""
    K = np.asarray(K, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    n = y.shape[0]
    a0, b0, _ = solve_cell(K, y, lam, "hinge", delta0)
    u = y * (K @ a0 + b0)
    state = np.where(u <= 1.0 - delta0, 0, np.where(u >= 1.0 + delta0, 2, 1))   # 0 L, 1 E, 2 R
    seen = set()
    rounds = 0
    ok = False
    a = 2.0 * n * lam * y * a0
    beta = b0
    beta_lo = beta_hi = beta
    for rounds in range(1, max_rounds + 1):
        L = np.flatnonzero(state == 0)
        E = np.flatnonzero(state == 1)
        if E.size == 0:
            # no point on the margin: a is fixed by the sets, the balance
            # must hold by itself and beta is any value keeping every point
            # on its side; otherwise the point nearest the margin joins E
            a = np.zeros(n)
            a[L] = 1.0
            alpha = y * a / (2.0 * n * lam)
            g = K @ alpha
            if abs(y[L].sum()) > tol * n:
                state = state.copy()
                state[int(np.argmin(np.abs(y * (g + beta) - 1.0)))] = 1
                continue
            # y_i (g_i + beta) <= 1 on L and >= 1 on R; with y_i = +-1 each is
            # an upper or a lower bound on beta
            R = np.flatnonzero(state == 2)
            t = 1.0 - y * g                      # y_i beta <= t_i on L, >= t_i on R
            up = np.concatenate([t[L][y[L] > 0], -t[R][y[R] < 0]])
            dn = np.concatenate([-t[L][y[L] < 0], t[R][y[R] > 0]])
            hi = float(up.min()) if up.size else np.inf
            lo = float(dn.max()) if dn.size else -np.inf
            if lo > hi + tol:
                state = state.copy()
                state[int(np.argmin(np.abs(y * (g + beta) - 1.0)))] = 1
                continue
            beta_lo, beta_hi = lo, hi
            beta = float(min(max(beta, lo), hi))
            ok = True
            break
        res = _solve_sets(K, y, lam, L, E)
        if res is None:
            break
        a, beta = res
        beta_lo = beta_hi = beta
        alpha = y * a / (2.0 * n * lam)
        u = y * (K @ alpha + beta)
        bad_lo = (state == 1) & (a < -tol)
        bad_hi = (state == 1) & (a > 1.0 + tol)
        bad_L = (state == 0) & (u > 1.0 + tol)
        bad_R = (state == 2) & (u < 1.0 - tol)
        if not (bad_lo.any() or bad_hi.any() or bad_L.any() or bad_R.any()):
            ok = True
            break
        key = state.tobytes()
        if key in seen:
            break
        seen.add(key)
        state = state.copy()
        state[bad_lo] = 2
        state[bad_hi] = 0
        state[bad_L | bad_R] = 1
    a = np.clip(a, 0.0, 1.0) if ok else a
    alpha = y * a / (2.0 * n * lam)
    if ok and beta_lo == beta_hi:
        # points on the margin with a strictly inside (0, 1) pin beta; when
        # every one sits at a bound the intercept is an interval, the points
        # at a = 1 keeping u <= 1 and those at a = 0 keeping u >= 1
        E = np.flatnonzero(state == 1)
        free = (a[E] > tol) & (a[E] < 1.0 - tol)
        if not free.any():
            g = K @ alpha
            t = 1.0 - y * g
            Lb = np.flatnonzero((state == 0) | ((state == 1) & (a >= 1.0 - tol)))
            Rb = np.flatnonzero((state == 2) | ((state == 1) & (a <= tol)))
            up = np.concatenate([t[Lb][y[Lb] > 0], -t[Rb][y[Rb] < 0]])
            dn = np.concatenate([-t[Lb][y[Lb] < 0], t[Rb][y[Rb] > 0]])
            beta_hi = float(up.min()) if up.size else np.inf
            beta_lo = float(dn.max()) if dn.size else -np.inf
    P = hinge_objective(K, y, alpha, beta, lam)
    D = hinge_dual(K, y, a, lam)
    info = {"rounds": rounds, "E": int(np.count_nonzero(state == 1)), "converged": ok,
            "gap": P - D, "objective": P, "beta_lo": beta_lo, "beta_hi": beta_hi}
    return alpha, beta, info
