"""a2 in band form (per-fold factorisation K = Q B Q', B banded) through the C ABI.

Pinned by the definition (backward error of Q B Q' and orthogonality of Q,
both within a small multiple of N * eps), by the spectrum (the eigenvalues
of B equal numpy's eigenvalues of the input) and, with zero padding rows, by
the exact structure of the padded block.
"""
import numpy as np
import pytest

import workloads as W
from oracle import gram as OG
from tests.gpu_common import announce, device

pytestmark = pytest.mark.gpu
EPS = np.finfo(float).eps


def _reduce(A):
    import torch
    from paper_2606_06742_amd import kmpath as km
    dev = device()
    G, N, _ = A.shape
    At = torch.tensor(A, device=dev)
    Q = torch.empty_like(At)
    band = torch.empty((G, km.KMP_BAND + 1, N), dtype=torch.float64, device=dev)
    km.kmp_band_reduce(At, Q, band)
    torch.cuda.synchronize()
    return Q.cpu().numpy(), band.cpu().numpy()


def _dense(band):
    b1, N = band.shape
    B = np.zeros((N, N))
    for r in range(b1):
        idx = np.arange(N - r)
        B[idx + r, idx] = band[r, :N - r]
        B[idx, idx + r] = band[r, :N - r]
    return B


def _check(A, Q, band, c=40.0):
    G, N, _ = A.shape
    for g in range(G):
        for r in range(band.shape[1]):
            assert np.all(band[g, r, N - r:] == 0.0)
        B = _dense(band[g])
        nA = np.linalg.norm(A[g])
        R = Q[g] @ B @ Q[g].T - A[g]
        assert np.linalg.norm(R) <= c * N * EPS * nA, (g, np.linalg.norm(R) / nA)
        assert np.abs(Q[g].T @ Q[g] - np.eye(N)).max() <= c * N * EPS
        ev_b = np.linalg.eigvalsh(B)
        ev_a = np.linalg.eigvalsh(A[g])
        assert np.abs(ev_b - ev_a).max() <= c * N * EPS * np.abs(ev_a).max()


# orders 64 .. 320 take every arrangement of the accumulation of Q: the
# partial last block alone (64, 128), then pairs of 64-blocks with (256) or
# without (192, 320) a single block left at the bottom
@pytest.mark.parametrize("N,G", [(64, 1), (128, 3), (192, 2), (256, 2), (320, 1)])
def test_band_random_symmetric(N, G):
    rng = np.random.default_rng(N + G)
    B = rng.standard_normal((G, N, N))
    A = B + B.transpose(0, 2, 1)
    announce(f"band reduction random symmetric N={N} G={G}")
    Q, band = _reduce(A.copy())
    _check(A, Q, band)


def test_band_rbf_folds_with_padding():
    inp = W.make_inputs(W.get("C1"))
    X, fold = inp["X"], inp["fold_id"]
    N = 192
    A = np.zeros((5, N, N))
    nv = []
    for v in range(5):
        Kv, _, T, _ = OG.fold_blocks(X, fold, v, inp["sigmas"][0])
        A[v, :T.size, :T.size] = Kv
        nv.append(T.size)
    announce("band reduction C1 folds N=192 (zero padding)")
    Q, band = _reduce(A.copy())
    _check(A, Q, band)
    for v in range(5):
        m = nv[v]
        assert np.array_equal(Q[v, m:, m:], np.eye(N - m))
        assert np.all(Q[v, :m, m:] == 0.0) and np.all(Q[v, m:, :m] == 0.0)
        B = _dense(band[v])
        assert np.all(B[m:, :] == 0.0)


def test_band_c2_sized_fold():
    inp = W.make_inputs(W.get("C2"))
    Kv, _, T, _ = OG.fold_blocks(inp["X"], inp["fold_id"], 0, inp["sigmas"][1])
    announce("band reduction C2 fold 0, N=1600")
    Q, band = _reduce(Kv[None].copy())
    _check(Kv[None], Q, band)


def test_band_long_panels():
    """Orders above 2048 + 16 rows take the streaming panel factorisation
    (the panel no longer fits in registers) for the first panels."""
    N = 2176
    rng = np.random.default_rng(11)
    B = rng.standard_normal((N, N))
    A = (B + B.T)[None]
    announce(f"band reduction random symmetric N={N} (streaming panels)")
    Q, band = _reduce(A.copy())
    _check(A, Q, band)


def test_band_groups_beyond_32bit_grid():
    """Five folds of order 29376 (more than 2^32 entries over the batch, as
    with five folds of 32000 points): every group is reduced, identical
    inputs give identical factors, and sampled rows of Q B Q' reproduce the
    input."""
    import torch
    from paper_2606_06742_amd import kmpath as km
    dev = device()
    N, G = 29376, 5
    announce(f"band reduction G={G} N={N} ({G * N * N} entries)")
    torch.manual_seed(0)
    X = torch.randn(N, 8, dtype=torch.float64, device=dev)
    d2 = (X * X).sum(1)
    A0 = torch.exp(-(d2[:, None] + d2[None, :] - 2 * X @ X.T).clamp_min(0) / 16.0)
    A0.fill_diagonal_(1.0)
    A = torch.empty((G, N, N), dtype=torch.float64, device=dev)
    for g in range(G):
        A[g] = A0
    Q = torch.empty_like(A)
    band = torch.empty((G, km.KMP_BAND + 1, N), dtype=torch.float64, device=dev)
    km.kmp_band_reduce(A, Q, band)
    torch.cuda.synchronize()
    del A
    for g in range(1, G):
        assert torch.equal(Q[g], Q[0]) and torch.equal(band[g], band[0]), g
    Q0 = Q[0]
    assert (Q0[:, :64].T @ Q0[:, :64] - torch.eye(64, dtype=torch.float64, device=dev)).abs().max().item() <= 40 * N * EPS
    b = band[0]
    for i in (0, 1, N // 2, N - 1):
        q = Q0[i]
        r = b[0] * q                                     # r = B q (B symmetric, banded)
        for k in range(1, km.KMP_BAND + 1):
            r[k:] += b[k, :N - k] * q[:N - k]
            r[:N - k] += b[k, :N - k] * q[k:]
        row = Q0 @ r
        assert (row - A0[i]).abs().max().item() <= 40 * N * EPS, i
