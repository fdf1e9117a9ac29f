"""a2 (per-fold factorisation K = Q T Q') through the C ABI.

Pinned by the definition (backward error of Q T Q' and orthogonality of Q,
both within a small multiple of N * eps) and by the spectrum: the
eigenvalues of T must equal numpy's eigenvalues of the input.
"""
import numpy as np
import pytest
from scipy.linalg import eigvalsh_tridiagonal

import workloads as W
from oracle import gram as OG
from tests.gpu_common import announce, device

pytestmark = pytest.mark.gpu
EPS = np.finfo(float).eps


def _factor(A):
    import torch
    from paper_2606_06742_amd import kmpath as km
    dev = device()
    G, N, _ = A.shape
    At = torch.tensor(A, device=dev)
    Q = torch.empty_like(At)
    d = torch.empty((G, N), dtype=torch.float64, device=dev)
    e = torch.empty((G, N), dtype=torch.float64, device=dev)
    km.kmp_tridiag(At, Q, d, e)
    torch.cuda.synchronize()
    return Q.cpu().numpy(), d.cpu().numpy(), e.cpu().numpy()


def _check(A, Q, d, e, c=30.0):
    G, N, _ = A.shape
    for g in range(G):
        T = np.diag(d[g]) + np.diag(e[g, :-1], -1) + np.diag(e[g, :-1], 1)
        assert e[g, -1] == 0.0
        nA = np.linalg.norm(A[g])
        R = Q[g] @ T @ Q[g].T - A[g]
        assert np.linalg.norm(R) <= c * N * EPS * nA, (g, np.linalg.norm(R) / nA)
        assert np.abs(Q[g].T @ Q[g] - np.eye(N)).max() <= c * N * EPS
        ev_t = eigvalsh_tridiagonal(d[g], e[g, :-1])
        ev_a = np.linalg.eigvalsh(A[g])
        assert np.abs(ev_t - ev_a).max() <= c * N * EPS * np.abs(ev_a).max()


@pytest.mark.parametrize("N,G", [(32, 1), (96, 3), (256, 2)])
def test_tridiag_random_symmetric(N, G):
    rng = np.random.default_rng(N + G)
    B = rng.standard_normal((G, N, N))
    A = B + B.transpose(0, 2, 1)
    announce(f"tridiag random symmetric N={N} G={G}")
    Q, d, e = _factor(A.copy())
    _check(A, Q, d, e)


def test_tridiag_rbf_folds_with_padding():
    inp = W.make_inputs(W.get("C1"))
    X, fold = inp["X"], inp["fold_id"]
    N = 192
    A = np.zeros((5, N, N))
    nv = []
    for v in range(5):
        Kv, _, T, _ = OG.fold_blocks(X, fold, v, inp["sigmas"][0])
        A[v, :T.size, :T.size] = Kv
        nv.append(T.size)
    announce("tridiag C1 folds N=192 (zero padding)")
    Q, d, e = _factor(A.copy())
    _check(A, Q, d, e)
    for v in range(5):
        m = nv[v]
        assert np.array_equal(Q[v, m:, m:], np.eye(N - m))
        assert np.all(Q[v, :m, m:] == 0.0) and np.all(Q[v, m:, :m] == 0.0)
        assert np.all(d[v, m:] == 0.0) and np.all(e[v, m - 1:] == 0.0)


def test_tridiag_c2_sized_fold():
    inp = W.make_inputs(W.get("C2"))
    Kv, _, T, _ = OG.fold_blocks(inp["X"], inp["fold_id"], 0, inp["sigmas"][1])
    announce("tridiag C2 fold 0, N=1600")
    Q, d, e = _factor(Kv[None].copy())
    _check(Kv[None], Q, d, e)
