"""The paper's majorise-minimise (proximal-gradient) update, dense.

Oracle (test infrastructure only). Appendix A.1 gives the update

    (beta, alpha)_{k+1} - (beta, alpha)_k = - H^{-1} (1'z ; K z + 2 lambda K alpha),

with loss-curvature bound 1/kappa (kappa = 2 delta for the smoothed hinge).
Reading of H (the paper writes only its alpha-block 2 lambda K + K K/(n kappa)):
it is the (n+1)-square Hessian of the quadratic majoriser of F in (beta, alpha),

    H = [[ 1/kappa        , 1'K/(n kappa)              ],
         [ K 1/(n kappa)  , 2 lambda K + K K/(n kappa) ]],

whose block inverse is the rank-one-plus-spectral form of Appendix A.3 with
v = (2 lambda I + K/(n kappa))^{-1} 1/(n kappa) and g = 1/s,
s = 1/kappa - 1'K v/(n kappa) (the Schur complement of the alpha-block).

``mm_step`` applies H^{-1} through the well-conditioned SPD matrix
M = 2 lambda I + K/(n kappa), using A^{-1} K = M^{-1} (K and M commute); this
equals ``mm_step_literal`` (an explicit solve with H) whenever K is
nonsingular, and stays defined when the RBF kernel is numerically singular.
"""
from __future__ import annotations

import numpy as np

from . import losses as Ls


def _spd_solve(M, B):
    L = np.linalg.cholesky(M)
    return np.linalg.solve(L.T, np.linalg.solve(L, B))


def mm_step(K, y, alpha, beta, lam, loss, delta=None, tau=None, kap=None, norm=None):
    """(alpha_new, beta_new) after one majorise-minimise step from (alpha, beta).

    ``norm`` replaces n as the loss normaliser (n in the paper's formulas);
    with norm = n the intercept block of H is 1/kappa.
    """
    n = y.shape[0]
    N = float(n if norm is None else norm)
    if kap is None:
        kap = Ls.kappa(loss, delta)
    f = K @ alpha + beta
    z = Ls.point_psi(loss, y, f, delta, tau) / N
    w = z + 2.0 * lam * alpha                  # K w = K z + 2 lambda K alpha
    d0 = z.sum()                               # 1'z
    M = 2.0 * lam * np.eye(n) + K / (N * kap)
    X = _spd_solve(M, np.stack([w, np.ones(n)], axis=1))
    x = X[:, 0]                                # A^{-1} K w
    v = X[:, 1] / (N * kap)                    # A^{-1} K 1/(N kappa)
    s = n / (N * kap) - (K @ v).sum() / (N * kap)
    g = 1.0 / s
    t = v @ (K @ w)                            # v' K w
    dbeta = g * (d0 - t)
    dalpha = g * (t - d0) * v + x
    return alpha - dalpha, beta - dbeta


def majoriser_hessian(K, lam, kap):
    """The (n+1)-square H above, intercept first."""
    n = K.shape[0]
    H = np.empty((n + 1, n + 1))
    H[0, 0] = 1.0 / kap
    H[0, 1:] = K.sum(axis=0) / (n * kap)
    H[1:, 0] = K.sum(axis=1) / (n * kap)
    H[1:, 1:] = 2.0 * lam * K + (K @ K) / (n * kap)
    return H


def mm_step_literal(K, y, alpha, beta, lam, loss, delta=None, tau=None, kap=None):
    """Same step by an explicit solve with H (needs a well-conditioned K)."""
    n = y.shape[0]
    if kap is None:
        kap = Ls.kappa(loss, delta)
    f = K @ alpha + beta
    z = Ls.point_psi(loss, y, f, delta, tau) / n
    d = np.concatenate([[z.sum()], K @ z + 2.0 * lam * (K @ alpha)])
    step = np.linalg.solve(majoriser_hessian(K, lam, kap), d)
    return alpha - step[1:], beta - step[0]


def accelerated_iteration(K, y, alpha, beta, alpha_prev, beta_prev, r, lam, loss,
                          delta=None, tau=None):
    """One pass of the accelerated inner loop of Algorithm 1 (no restart).

    r' = (1 + sqrt(1 + 4 r^2))/2; extrapolate (alpha_bar, beta_bar) =
    current + ((r - 1)/r') (current - previous); take the majorise-minimise
    step from the extrapolated point. Returns (alpha_new, beta_new,
    alpha_prev_new, beta_prev_new, r_new, alpha_bar, beta_bar).
    """
    r1 = 0.5 * (1.0 + np.sqrt(1.0 + 4.0 * r * r))
    c = (r - 1.0) / r1
    ab = alpha + c * (alpha - alpha_prev)
    bb = beta + c * (beta - beta_prev)
    an, bn = mm_step(K, y, ab, bb, lam, loss, delta, tau)
    return an, bn, alpha, beta, r1, ab, bb
