"""RBF kernel matrix by direct differences.

Oracle (test infrastructure only). The paper uses an RBF kernel
(``kernel="rbf"``, Section 2) without stating its parameterisation; the
reading used throughout is K(x, x') = exp(-||x - x'||^2 / (2 sigma^2)).
Distances are formed as sums of squared coordinate differences, never by
the norm expansion, so the diagonal is exactly 1.
"""
from __future__ import annotations

import numpy as np


def rbf_gram(XA, XB, sigma):
    """K[i, j] = exp(-||XA[i] - XB[j]||^2 / (2 sigma^2))."""
    XA = np.asarray(XA, dtype=np.float64)
    XB = np.asarray(XB, dtype=np.float64)
    out = np.empty((XA.shape[0], XB.shape[0]))
    for i in range(XA.shape[0]):
        diff = XB - XA[i]
        out[i] = np.exp(-np.einsum("ij,ij->i", diff, diff) / (2.0 * sigma * sigma))
    return out


def fold_blocks(X, fold_id, v, sigma):
    """(K_v, K_cross, train_idx, held_idx) for fold v.

    K_v = K[T_v, T_v] over the training points of fold v (all points whose
    fold id is not v, in increasing index order); K_cross = K[H_v, T_v] over
    the held-out points H_v (fold id == v). This is the fold-restricted kernel
    of the exact-CV problem in Appendix A.2.
    """
    fold_id = np.asarray(fold_id)
    T = np.flatnonzero(fold_id != v)
    H = np.flatnonzero(fold_id == v)
    Kv = rbf_gram(X[T], X[T], sigma)
    Kc = rbf_gram(X[H], X[T], sigma)
    return Kv, Kc, T, H


def rbf_gram_expansion(XA, XB, sigma):
    """The same kernel with squared distances by the norm expansion
    ||a||^2 + ||b||^2 - 2 a'b (clamped at 0; exactly 1 where the rows are the
    same point). It differs from ``rbf_gram`` by rounding only; re-solving a
    cell with it measures how far fp64 rounding of K alone moves the
    solution (the cell's noise floor)."""
    XA = np.asarray(XA, dtype=np.float64)
    XB = np.asarray(XB, dtype=np.float64)
    na = np.einsum("ij,ij->i", XA, XA)
    nb = np.einsum("ij,ij->i", XB, XB)
    d2 = np.maximum(na[:, None] + nb[None, :] - 2.0 * (XA @ XB.T), 0.0)
    K = np.exp(-d2 / (2.0 * sigma * sigma))
    if XA is XB or (XA.shape == XB.shape and np.array_equal(XA, XB)):
        np.fill_diagonal(K, 1.0)
    return K
