"""Oracle RBF Gram against a library routine and the properties of a kernel matrix."""
import numpy as np
import pytest
from sklearn.metrics.pairwise import rbf_kernel

import workloads as W
from oracle import gram


def test_rbf_matches_sklearn():
    rng = np.random.default_rng(5)
    XA, XB = rng.standard_normal((37, 6)), rng.standard_normal((29, 6))
    for sigma in [0.7, 2.0, 5.0]:
        ref = rbf_kernel(XA, XB, gamma=1.0 / (2.0 * sigma * sigma))
        assert np.allclose(gram.rbf_gram(XA, XB, sigma), ref, rtol=1e-12, atol=1e-300)


def test_gram_symmetric_unit_diagonal_psd():
    inp = W.make_inputs(W.get("C1"))
    K = gram.rbf_gram(inp["X"], inp["X"], inp["sigmas"][0])
    assert np.array_equal(K, K.T)
    assert np.all(np.diag(K) == 1.0)
    assert np.all(K > 0) and np.all(K <= 1.0)
    ev = np.linalg.eigvalsh(K)
    assert ev.min() >= -K.shape[0] * np.finfo(float).eps * ev.max()


def test_fold_blocks_are_submatrices():
    inp = W.small_problem("hinge", 23, 3, seed=4, V=4)
    X, fold, s = inp["X"], inp["fold_id"], inp["sigmas"][0]
    K = gram.rbf_gram(X, X, s)
    seen = np.zeros(23, dtype=int)
    for v in range(4):
        Kv, Kc, T, H = gram.fold_blocks(X, fold, v, s)
        assert np.array_equal(np.sort(np.concatenate([T, H])), np.arange(23))
        assert np.all(fold[H] == v) and np.all(fold[T] != v)
        assert np.array_equal(Kv, K[np.ix_(T, T)]) and np.array_equal(Kc, K[np.ix_(H, T)])
        seen[H] += 1
    assert np.all(seen == 1)
