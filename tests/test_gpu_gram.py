"""a1 (Gram + fold gather) through the C ABI against the oracle Gram."""
import numpy as np
import pytest

import workloads as W
from oracle import gram as OG
from tests.gpu_common import announce, device

pytestmark = pytest.mark.gpu


def _run(X, rows, cols, sigmas, ld=None):
    import torch
    from paper_2606_06742_amd import kmpath as km
    dev = device()
    m, p = len(rows), len(cols)
    ld = ld or p
    out = torch.full((len(sigmas), m, ld), np.nan, dtype=torch.float64, device=dev)
    km.kmp_rbf_gram(torch.tensor(X, device=dev), torch.tensor(rows, dtype=torch.int32, device=dev),
                    torch.tensor(cols, dtype=torch.int32, device=dev), sigmas, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _check(X, rows, cols, sigmas, got):
    for s, sig in enumerate(sigmas):
        for i, r in enumerate(rows):
            for_cols = np.asarray(cols)
            valid = (for_cols >= 0) & (r >= 0)
            row = got[s, i, :len(cols)]
            assert np.all(row[~valid] == 0.0)
            if r < 0:
                continue
            c = for_cols[valid]
            ref = OG.rbf_gram(X[[r]], X[c], sig)[0]
            # norm-expansion rounding: |dK| <~ K * eps * (|x_r|^2 + |x_c|^2) / sigma^2
            bound = 64 * np.finfo(float).eps * ref * ((X[r] ** 2).sum() + (X[c] ** 2).sum(1)) / (2 * sig * sig)
            assert np.all(np.abs(row[valid] - ref) <= bound + 1e-300), (s, i)
            same = c == r
            assert np.all(row[valid][same] == 1.0)


def test_gram_c1_fold_block_with_padding():
    inp = W.make_inputs(W.get("C1"))
    X, fold = inp["X"], inp["fold_id"]
    T = np.flatnonzero(fold != 2)
    idx = np.full(192, -1, dtype=np.int32)
    idx[:T.size] = T
    sig = [inp["sigmas"][0], 0.5 * inp["sigmas"][0]]
    announce(f"gram C1 fold 2, N=192, sigmas={sig}")
    got = _run(X, idx, idx, sig)
    _check(X, idx, idx, sig, got)
    Kref = OG.rbf_gram(X[T], X[T], sig[0])
    assert np.abs(got[0, :T.size, :T.size] - Kref).max() < 1e-14
    assert np.array_equal(got[0, :T.size, :T.size], got[0, :T.size, :T.size].T)


def test_gram_ragged_rectangular():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((300, 37)) * 0.7
    rows = rng.choice(300, 70, replace=False).astype(np.int32)
    cols = rng.choice(300, 45, replace=False).astype(np.int32)
    cols[[3, 17]] = -1
    rows[5] = -1
    cols[20] = rows[9]                         # one coincident pair -> exactly 1
    sig = [1.3, 4.0, 9.0]
    announce("gram ragged 70x45, d=37, 3 sigmas, ld=53")
    got = _run(X, rows, cols, sig, ld=53)
    _check(X, rows, cols, sig, got)
    assert np.all(np.isnan(got[:, :, 45:]))    # nothing written past p
