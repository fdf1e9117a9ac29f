"""Dual problems of the three fold-restricted kernel machines.

Oracle (test infrastructure only). Each training loss is a maximum over a
box of functions linear in f, so exchanging min and max in
F(alpha, beta) = (1/n) sum loss(y_i, f_i) + lambda alpha'K alpha gives a
concave dual whose optimal value equals min F (zero gap):

* smoothed hinge, L_delta(u) = max_{a in [0,1]} a(1 - u + delta) - delta a^2:
  D(a) = (1/n) sum [(1 + delta) a_i - delta a_i^2] - s'K s/(4 n^2 lambda),
  s = a o y, constraint y'a = 0, and alpha = s/(2 n lambda).
* logistic, log(1 + e^-u) = max_{a in [0,1]} -a u + H_b(a) (binary entropy):
  D(a) = (1/n) sum H_b(a_i) - s'K s/(4 n^2 lambda), same constraint and map.
* smoothed check, rho(r) = max_{a in [tau-1, tau]} a r + delta (a-tau+1)(tau-a):
  D(a) = (1/n) sum [a_i y_i + delta (a_i-tau+1)(tau-a_i)] - a'K a/(4 n^2 lambda),
  constraint 1'a = 0 and alpha = a/(2 n lambda).

From a primal point the dual variable is read off the loss derivative:
a = -n (y o z) for margin losses, a = -n z for the check loss, where
z = psi(y, f)/n.
"""
from __future__ import annotations

import numpy as np

from . import losses as Ls


def dual_point(loss, y, f, delta=None, tau=None):
    n = y.shape[0]
    z = Ls.point_psi(loss, y, f, delta, tau) / n
    if loss in ("hinge", "logistic"):
        return -n * y * z
    return -n * z


def _entropy(a):
    a = np.asarray(a, dtype=np.float64)
    out = np.zeros_like(a)
    m = (a > 0.0) & (a < 1.0)
    out[m] = -a[m] * np.log(a[m]) - (1.0 - a[m]) * np.log1p(-a[m])
    return out


def dual_value(loss, K, y, a, lam, delta=None, tau=None):
    n = y.shape[0]
    if loss == "hinge":
        s = a * y
        return float(((1.0 + delta) * a - delta * a * a).sum() / n - s @ K @ s / (4.0 * n * n * lam))
    if loss == "logistic":
        s = a * y
        return float(_entropy(a).sum() / n - s @ K @ s / (4.0 * n * n * lam))
    if loss == "check":
        return float((a * y + delta * (a - tau + 1.0) * (tau - a)).sum() / n
                     - a @ K @ a / (4.0 * n * n * lam))
    raise ValueError(loss)


def dual_feasibility(loss, y, a, tau=None):
    """(box violation, equality violation) of a dual point."""
    if loss in ("hinge", "logistic"):
        box = max(0.0, float(-a.min()), float(a.max() - 1.0))
        eq = abs(float(y @ a))
    else:
        box = max(0.0, float((tau - 1.0) - a.min()), float(a.max() - tau))
        eq = abs(float(a.sum()))
    return box, eq


def alpha_from_dual(loss, y, a, lam):
    n = y.shape[0]
    if loss in ("hinge", "logistic"):
        return a * y / (2.0 * n * lam)
    return a / (2.0 * n * lam)
