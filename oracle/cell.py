"""One cross-validation cell solved on its own, to machine precision.

Oracle (test infrastructure only). A cell is one (kernel, fold, lambda)
problem: the fold-restricted kernel machine of Appendix A.2 (training points
T_v only, 1/n_v normalisation),

    F(alpha, beta) = (1/n_v) sum_i loss(y_i, f_i) + lambda alpha' K alpha,
    f = K alpha + beta 1,

which is eq. (kernelsvm) of Appendix A.1 with the smoothed loss in place of
the hinge. Its minimiser is unique in alpha (strictly concave dual, see
``oracle.dual``); beta can be non-unique for the smoothed hinge / check loss
when no training point lies in the quadratic zone (``beta_interval``).

The solver is NOT the paper's spectral majorise-minimise iteration: it is a
damped semismooth Newton method on the representer-form stationarity system

    R(alpha, beta) = ( z + 2 lambda alpha ,  1'z ) = 0,   z_i = psi(y_i, f_i)/n_v,

(grad F = diag(K, 1) R, so R = 0 is stationarity), with generalised Jacobian
J = [[2 lambda I + D K, D 1], [1' D K, 1' D 1]], D = diag(curv)/n_v.
Each Newton step is globalised by an exact line search on F (F is convex
along any line); when J is singular or its direction is not a descent
direction, the direction of a dense majorise-minimise step
(``oracle.mm.mm_step``) is searched instead; when no point has curvature
(empty quadratic zone) alpha and beta are minimised in turn exactly (after 16
such alternating steps in a row, the majorise-minimise direction). For piecewise-
quadratic losses only rows with nonzero curvature couple, so the linear
system is reduced to those rows exactly (Mangasarian 2002, "A finite Newton
method for classification"; Keerthi and DeCoste 2005).

Certified convergence. At small lambda the coefficients reach 1/(2 n lambda)
and an fp64 evaluation of f = K alpha + beta carries rounding that the loss
curvature 1/(2 delta) amplifies: the fp64 residual stops falling well above
the tolerance. The last steps are therefore Newton corrections by iterative
refinement: the Newton matrix is formed and solved in fp64 exactly as above,
but the residual it is applied to and the iterate it corrects are carried in
numpy's extended type (x87 long double, 64-bit significand), with
f = K alpha + beta accumulated in it. The residual reported for a cell is that
of the refined extended-precision point, of which the returned fp64 values
are the rounding (within half an ulp each), and a cell counts as converged
only when it is at most ``CONVERGED_KKT``.
"""
from __future__ import annotations

import numpy as np

from . import dual as Dl
from . import losses as Ls
from .mm import mm_step

# A cell counts as solved when n_v * max(||z + 2 lambda alpha||_inf, |1'z|),
# evaluated in extended precision at the refined point, is at most this.
CONVERGED_KKT = 1e-10


def _ext_matvec(K, a, rows=512):
    """K @ a with the products and sums in numpy's extended type."""
    out = np.empty(K.shape[0], dtype=np.longdouble)
    for i0 in range(0, K.shape[0], rows):
        out[i0:i0 + rows] = K[i0:i0 + rows].astype(np.longdouble) @ a
    return out


def residual_ext(K, y, alpha, beta, lam, loss, delta=None, tau=None, norm=None):
    """(R_alpha, R_beta, f, kkt) with f = K alpha + beta, z and R in extended
    precision; kkt = norm * max(||R_alpha||_inf, |R_beta|) as a float."""
    ld = np.longdouble
    n = y.shape[0]
    N = ld(n if norm is None else norm)
    a = np.asarray(alpha).astype(ld)
    f = _ext_matvec(K, a) + ld(beta)
    z = Ls.point_psi(loss, np.asarray(y).astype(ld), f, delta, tau) / N
    Ra = z + 2 * ld(lam) * a
    Rb = z.sum()
    kkt = float(N * max(np.max(np.abs(Ra)) if Ra.size else ld(0), abs(Rb)))
    return Ra, Rb, f, kkt


def objective(K, y, alpha, beta, lam, loss, delta=None, tau=None, norm=None):
    """F(alpha, beta) of the cell (training loss at the given delta).

    ``norm`` is the loss normaliser (default: the number of points); the
    exact-CV form of Appendix A.2 uses n - m with held-out responses zeroed.
    """
    Ka = K @ alpha
    f = Ka + beta
    n = y.shape[0] if norm is None else norm
    return float(Ls.point_loss(loss, y, f, delta, tau).sum() / n + lam * (alpha @ Ka))


def stationarity(K, y, alpha, beta, lam, loss, delta=None, tau=None, norm=None):
    """(R_alpha, R_beta, f, z): R_alpha = z + 2 lambda alpha, R_beta = 1'z."""
    n = y.shape[0] if norm is None else norm
    f = K @ alpha + beta
    z = Ls.point_psi(loss, y, f, delta, tau) / n
    return z + 2.0 * lam * alpha, float(z.sum()), f, z


def kkt_residual(K, y, alpha, beta, lam, loss, delta=None, tau=None, norm=None):
    """n_v * max(||z + 2 lambda alpha||_inf, |1'z|)."""
    Ra, Rb, _, _ = stationarity(K, y, alpha, beta, lam, loss, delta, tau, norm)
    n = y.shape[0] if norm is None else norm
    return float(n * max(np.max(np.abs(Ra)) if Ra.size else 0.0, abs(Rb)))


def _newton_direction(K, y, alpha, beta, lam, loss, delta, tau, Ra, Rb, f, norm):
    n = y.shape[0]
    D = Ls.point_curv(loss, y, f, delta, tau) / norm
    A = np.flatnonzero(D > 0.0)
    I = np.flatnonzero(D <= 0.0)
    if A.size == 0:
        return None
    da = np.empty(n)
    da[I] = -Ra[I] / (2.0 * lam)
    DA = D[A]
    KAA = K[np.ix_(A, A)]
    KAI = K[np.ix_(A, I)]
    carry = KAI @ da[I]                       # K[A, I] dalpha_I
    m = A.size
    J = np.empty((m + 1, m + 1))
    J[:m, :m] = DA[:, None] * KAA
    J[:m, :m][np.diag_indices(m)] += 2.0 * lam
    J[:m, m] = DA
    J[m, :m] = DA @ KAA
    J[m, m] = DA.sum()
    rhs = np.empty(m + 1)
    rhs[:m] = -Ra[A] - DA * carry
    rhs[m] = -Rb - DA @ carry
    try:
        sol = np.linalg.solve(J, rhs)
    except np.linalg.LinAlgError:
        return None
    if not np.all(np.isfinite(sol)):
        return None
    da[A] = sol[:m]
    return da, float(sol[m])


def _line_minimum(K, y, alpha, beta, da, db, lam, loss, delta, tau, Ka, slope0, norm):
    """Exact minimiser t > 0 of phi(t) = F(alpha + t da, beta + t db).

    phi is convex (piecewise quadratic for hinge/check), so its derivative
    phi'(t) = df' z(t) + 2 lambda (Kda' alpha + t Kda' da), with
    f(t) = f0 + t df, is nondecreasing; the root is bracketed by doubling and
    found by bisection. A near-zero phi'(1) keeps the full step.
    """
    n = norm
    Kd = K @ da
    f0 = Ka + beta
    df = Kd + db
    c1 = 2.0 * lam * float(Kd @ alpha)
    c2 = 2.0 * lam * float(Kd @ da)

    def dphi(t):
        z = Ls.point_psi(loss, y, f0 + t * df, delta, tau) / n
        return float(df @ z) + c1 + t * c2

    d1 = dphi(1.0)
    if abs(d1) <= 1e-3 * abs(slope0):
        return 1.0
    if d1 < 0.0:
        lo, hi = 1.0, 2.0
        while dphi(hi) < 0.0 and hi < 2.0 ** 60:
            lo, hi = hi, 2.0 * hi
    else:
        lo, hi = 0.0, 1.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if mid <= lo or mid >= hi:
            break
        if dphi(mid) < 0.0:
            lo = mid
        else:
            hi = mid
    return hi if lo == 0.0 else 0.5 * (lo + hi)


def solve_cell(K, y, lam, loss, delta=None, tau=None, tol=1e-13, max_iter=500,
               alpha0=None, beta0=0.0, norm=None):
    """Minimise F for one cell. Returns (alpha, beta, info).

    The fp64 Newton loop stops when norm * max(||z + 2 lambda alpha||_inf,
    |1'z|) <= tol, or when that residual has stopped falling at its rounding
    floor (<= 1e-7); extended-precision refinement follows. info["kkt"] is
    the refined point's extended-precision residual (the returned values are
    that point rounded to fp64) and info["converged"]
    holds only when it is at most CONVERGED_KKT (a stall alone never counts).
    """
    K = np.asarray(K, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    n = y.shape[0]
    norm = float(n if norm is None else norm)
    alpha = np.zeros(n) if alpha0 is None else np.array(alpha0, dtype=np.float64)
    beta = float(beta0)
    best = np.inf
    stall = 0
    it = 0
    newton_steps = mm_steps = split_steps = split_run = 0
    res = np.inf
    for it in range(1, max_iter + 1):
        Ra, Rb, f, z = stationarity(K, y, alpha, beta, lam, loss, delta, tau, norm)
        res = norm * max(np.max(np.abs(Ra)), abs(Rb))
        if res <= tol:
            break
        if res < 0.5 * best:
            best = res
            stall = 0
        else:
            stall += 1
            if stall >= 8 and res <= 1e-7:
                break                       # stagnated at the rounding floor
        gK = K @ Ra                          # grad_alpha F = K (z + 2 lambda alpha)
        step = _newton_direction(K, y, alpha, beta, lam, loss, delta, tau, Ra, Rb, f, norm)
        if step is None and split_run >= 16:
            # alternating exact steps can cycle at tiny lambda (each alpha step
            # overshoots the zone): take the majorise-minimise direction instead
            split_run = 0
        elif step is None:
            split_run += 1
            # No point has curvature: on this piece F is linear in f plus
            # lambda alpha'K alpha, whose minimiser in alpha is -z/(2 lambda).
            # Take that step, then minimise exactly over beta alone.
            da = -Ra / (2.0 * lam)
            sl = float(gK @ da)
            if sl < 0.0:
                t = _line_minimum(K, y, alpha, beta, da, 0.0, lam, loss, delta, tau, f - beta, sl, norm)
                alpha = alpha + t * da
            Ra, Rb, f, z = stationarity(K, y, alpha, beta, lam, loss, delta, tau, norm)
            if Rb != 0.0:
                zero = np.zeros(n)
                t = _line_minimum(K, y, alpha, beta, zero, -Rb, lam, loss, delta, tau, f - beta, -Rb * Rb, norm)
                beta = beta - t * Rb
            split_steps += 1
            continue
        if step is not None:
            split_run = 0
        slope = 0.0
        if step is not None:
            da, db = step
            slope = float(gK @ da + Rb * db)
            if slope < 0.0:
                newton_steps += 1
        if not slope < 0.0:
            kap = Ls.kappa(loss, delta)
            a1, b1 = mm_step(K, y, alpha, beta, lam, loss, delta, tau, kap=kap, norm=norm)
            da, db = a1 - alpha, b1 - beta
            slope = float(gK @ da + Rb * db)
            mm_steps += 1
            if not slope < 0.0:
                break                       # no descent left at rounding level
        t = _line_minimum(K, y, alpha, beta, da, db, lam, loss, delta, tau, f - beta, slope, norm)
        alpha = alpha + t * da
        beta = beta + t * db
    alpha, beta, kkt, refine_steps = _refine(K, y, alpha, beta, lam, loss, delta, tau, norm)
    info = {"iters": it, "kkt": kkt, "kkt_fp64": float(res), "newton_steps": newton_steps,
            "mm_steps": mm_steps, "split_steps": split_steps, "refine_steps": refine_steps,
            "converged": bool(kkt <= CONVERGED_KKT)}
    return alpha, beta, info


def _refine(K, y, alpha, beta, lam, loss, delta, tau, norm, max_steps=12):
    """Newton corrections with extended-precision residuals (see the module
    note). Above the convergence bar a step that does not lower the residual
    is halved until it does (at most 12 times); the refinement stops when no
    step lowers it, or at the bar after a full step that does not. Returns the
    refined point rounded to fp64 (half an ulp per entry), the residual of the
    refined point itself and the number of corrections taken."""
    ld = np.longdouble
    a = np.asarray(alpha).astype(ld)
    b = ld(beta)
    Ra, Rb, f, res = residual_ext(K, y, a, b, lam, loss, delta, tau, norm)
    steps = 0
    for _ in range(max_steps):
        if res == 0.0:
            break
        step = _newton_direction(K, y, a.astype(np.float64), float(b), lam, loss, delta, tau,
                                 Ra.astype(np.float64), float(Rb), f.astype(np.float64), norm)
        if step is None:
            break
        da, db = step
        a2 = a + da.astype(ld)
        b2 = b + ld(db)
        Ra2, Rb2, f2, res2 = residual_ext(K, y, a2, b2, lam, loss, delta, tau, norm)
        if not res2 < res:
            if res <= CONVERGED_KKT:
                break
            # the stationarity conditions are only piecewise smooth (a point
            # entering or leaving its quadratic zone), so a full step can
            # overshoot: halve it until the residual falls, up to 12 times
            t = 1.0
            for _ in range(12):
                t *= 0.5
                a2 = a + (t * da).astype(ld)
                b2 = b + ld(t * db)
                Ra2, Rb2, f2, res2 = residual_ext(K, y, a2, b2, lam, loss, delta, tau, norm)
                if res2 < res:
                    break
            if not res2 < res:
                break
        a, b, Ra, Rb, f, res = a2, b2, Ra2, Rb2, f2, res2
        steps += 1
    return a.astype(np.float64), float(b), res, steps


def beta_interval(K, y, alpha, beta, loss, delta=None, tau=None):
    """Set of optimal intercepts at the optimal alpha, as (lo, hi).

    With alpha fixed, F is a convex function of beta alone. If some point is
    strictly inside its quadratic zone, the minimiser is unique (lo == hi ==
    beta). Otherwise F is locally linear with zero slope and stays flat until
    the nearest point enters its zone on either side.
    """
    if loss == "logistic":
        return beta, beta
    g = K @ alpha
    if loss == "hinge":
        # zone of point i in beta: y_i (g_i + beta) in (1 - delta, 1 + delta)
        c = y * 1.0 - g                 # beta at which y(g+beta) = 1
        lo_b = c - delta
        hi_b = c + delta
    else:
        c = y - g                       # beta at which r = y - g - beta = 0
        lo_b = c - delta
        hi_b = c + delta
    inside = (beta > lo_b) & (beta < hi_b)
    if np.any(inside):
        return beta, beta
    above = lo_b[lo_b >= beta]
    below = hi_b[hi_b <= beta]
    hi = float(above.min()) if above.size else np.inf
    lo = float(below.max()) if below.size else -np.inf
    return lo, hi


def certify_cell(K, y, alpha, beta, lam, loss, delta=None, tau=None):
    """Certificate of a solved cell (fold-restricted problem, 1/n_v scaling).

    The dual point is read off the loss derivative at f = K alpha + beta
    (``oracle.dual``); the certificate holds its box and equality
    violations, the dual value, the duality gap F - D (zero at the optimum,
    where the dual point is feasible and alpha = its image), the gap relative
    to max(1, F), the KKT residual in extended precision, and how many points
    lie below, inside and above the quadratic zone of the smoothed loss
    (hinge: u = y f against 1 -+ delta; check: r = y - f against -+ delta;
    logistic: all points have curvature and count as inside).
    """
    f = K @ alpha + beta
    F = objective(K, y, alpha, beta, lam, loss, delta, tau)
    a = Dl.dual_point(loss, y, f, delta, tau)
    box, eq = Dl.dual_feasibility(loss, y, a, tau)
    D = Dl.dual_value(loss, K, y, a, lam, delta, tau)
    if loss == "hinge":
        u = y * f
        zone = (int(np.count_nonzero(u <= 1.0 - delta)),
                int(np.count_nonzero((u > 1.0 - delta) & (u < 1.0 + delta))),
                int(np.count_nonzero(u >= 1.0 + delta)))
    elif loss == "check":
        r = y - f
        zone = (int(np.count_nonzero(r <= -delta)),
                int(np.count_nonzero((r > -delta) & (r < delta))),
                int(np.count_nonzero(r >= delta)))
    else:
        zone = (0, int(y.shape[0]), 0)
    _, _, _, kkt = residual_ext(K, y, alpha, beta, lam, loss, delta, tau)
    return {"objective": F, "dual": D, "gap": F - D, "rel_gap": (F - D) / max(1.0, abs(F)),
            "box": box, "eq": eq, "kkt": kkt, "zone": zone}
