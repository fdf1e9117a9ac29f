"""Losses of the three kernel machines, their f-derivatives and curvatures.

Oracle (test infrastructure only). Plain numpy, fp64 (inputs given in
numpy's extended type are evaluated in it).

* Smoothed hinge L_delta (Appendix A.1, definition of the delta-smoothed
  hinge): 1-u for u <= 1-delta, (u-1-delta)^2/(4 delta) for |u-1| < delta,
  0 for u >= 1+delta. Used with u = y f. Curvature bound 1/(2 delta), so the
  majorisation constant is kappa = 2 delta (Algorithm 1, first step).
* Logistic loss log(1 + exp(-y f)) (kernel logistic regression, Section 2).
  Its second derivative is at most 1/4, so kappa = 4 and no smoothing stage.
* Smoothed check loss for kernel quantile regression (Section 2 names the
  method; the paper gives no formula). Reading used here: the Moreau-type
  smoothing rho_{tau,delta}(r) = max_{a in [tau-1, tau]} [a r + delta (a-tau+1)
  (tau-a)], with r = y - f. It equals tau r for r >= delta, (tau-1) r for
  r <= -delta, and (r^2 + 2 r delta (2 tau - 1) + delta^2)/(4 delta) between;
  curvature 1/(2 delta), kappa = 2 delta, and rho_{1,delta}(1-u) = L_delta(u).

``psi`` is d loss / d f at fixed y; ``curv`` is d psi / d f (the generalised
second derivative; the zone value on the zone boundaries' open side).
"""
from __future__ import annotations

import numpy as np

LOSSES = ("hinge", "logistic", "check")


def _arr(u):
    """u as an fp64 array, or kept in numpy's extended type (longdouble) when
    given in it (the solver's refinement evaluates residuals that way)."""
    u = np.asarray(u)
    return u if u.dtype == np.longdouble else u.astype(np.float64)


def smoothed_hinge(u, delta):
    u = _arr(u)
    return np.where(u <= 1.0 - delta, 1.0 - u,
                    np.where(u >= 1.0 + delta, 0.0, (u - 1.0 - delta) ** 2 / (4.0 * delta)))


def smoothed_hinge_d1(u, delta):
    u = _arr(u)
    return np.where(u <= 1.0 - delta, -1.0,
                    np.where(u >= 1.0 + delta, 0.0, (u - 1.0 - delta) / (2.0 * delta)))


def smoothed_hinge_d2(u, delta):
    u = _arr(u)
    return np.where((u > 1.0 - delta) & (u < 1.0 + delta), 1.0 / (2.0 * delta), 0.0)


def hinge(u):
    return np.maximum(1.0 - _arr(u), 0.0)


def smoothed_check(r, tau, delta):
    r = _arr(r)
    mid = (r * r + 2.0 * r * delta * (2.0 * tau - 1.0) + delta * delta) / (4.0 * delta)
    return np.where(r >= delta, tau * r, np.where(r <= -delta, (tau - 1.0) * r, mid))


def smoothed_check_d1(r, tau, delta):
    r = _arr(r)
    return np.where(r >= delta, tau,
                    np.where(r <= -delta, tau - 1.0, (r + delta * (2.0 * tau - 1.0)) / (2.0 * delta)))


def smoothed_check_d2(r, tau, delta):
    r = _arr(r)
    return np.where((r > -delta) & (r < delta), 1.0 / (2.0 * delta), 0.0)


def check(r, tau):
    r = _arr(r)
    return r * (tau - (r < 0.0))


def logistic(u):
    """log(1 + exp(-u)), evaluated without overflow."""
    return np.logaddexp(0.0, -_arr(u))


def sigmoid(t):
    t = _arr(t)
    e = np.exp(-np.abs(t))
    return np.where(t >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def kappa(loss, delta):
    """Majorisation constant: loss curvature in f is bounded by 1/kappa."""
    if loss == "logistic":
        return 4.0
    if loss in ("hinge", "check"):
        return 2.0 * delta
    raise ValueError(loss)


def point_loss(loss, y, f, delta=None, tau=None):
    """Training (smoothed) loss of each point."""
    if loss == "hinge":
        return smoothed_hinge(y * f, delta)
    if loss == "logistic":
        return logistic(y * f)
    if loss == "check":
        return smoothed_check(y - f, tau, delta)
    raise ValueError(loss)


def point_psi(loss, y, f, delta=None, tau=None):
    """d/df of the training loss of each point."""
    if loss == "hinge":
        return y * smoothed_hinge_d1(y * f, delta)
    if loss == "logistic":
        return -y * sigmoid(-y * f)
    if loss == "check":
        return -smoothed_check_d1(y - f, tau, delta)
    raise ValueError(loss)


def point_curv(loss, y, f, delta=None, tau=None):
    """d^2/df^2 of the training loss of each point (generalised)."""
    if loss == "hinge":
        return smoothed_hinge_d2(y * f, delta) * (y * y)
    if loss == "logistic":
        s = sigmoid(y * f)
        return s * (1.0 - s) * (y * y)
    if loss == "check":
        return smoothed_check_d2(y - f, tau, delta)
    raise ValueError(loss)


def eval_loss(loss, y, f, tau=None):
    """Unsmoothed loss used for the held-out CV score."""
    if loss == "hinge":
        return hinge(y * f)
    if loss == "logistic":
        return logistic(y * f)
    if loss == "check":
        return check(y - f, tau)
    raise ValueError(loss)
