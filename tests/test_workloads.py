"""Seeded input generators: SplitMix64, fold assignment, bandwidth, data shapes."""
import os
from itertools import permutations

import numpy as np
import pytest
from scipy.spatial.distance import pdist

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64_seed1234567.txt")


def _golden():
    with open(GOLDEN) as fh:
        return [int(line) for line in fh if line.strip() and not line.startswith("#")]


def test_splitmix64_reference_outputs():
    assert W.splitmix64_stream(1234567, 5) == _golden()


def test_folds_balanced_and_deterministic():
    for n, V, seed in [(200, 5, 2001), (2000, 5, 2002), (203, 5, 9), (17, 4, 1), (7, 7, 3)]:
        f = W.make_folds(n, V, seed)
        assert f.dtype == np.int32 and f.shape == (n,)
        counts = np.bincount(f, minlength=V)
        assert counts.max() - counts.min() <= 1 and counts.sum() == n
        assert np.array_equal(f, W.make_folds(n, V, seed))
    assert not np.array_equal(W.make_folds(200, 5, 1), W.make_folds(200, 5, 2))


def test_folds_shuffle_is_uniform():
    # With V = n the fold vector is the inverse of the shuffled permutation:
    # Fisher-Yates with uniform draws makes all n! permutations equally likely.
    n, trials = 4, 24000
    seen = {}
    for s in range(trials):
        key = tuple(W.make_folds(n, n, s).tolist())
        seen[key] = seen.get(key, 0) + 1
    assert set(seen) == set(permutations(range(n)))
    expected = trials / 24.0
    chi2 = sum((c - expected) ** 2 / expected for c in seen.values())
    assert chi2 < 60.0          # 23 dof; p ~ 4e-5


def test_median_distance_matches_library():
    rng = np.random.default_rng(0)
    for n, d in [(2, 3), (3, 2), (10, 4), (57, 5), (120, 10)]:
        X = rng.standard_normal((n, d))
        assert W.median_pairwise_distance(X) == pytest.approx(float(np.median(pdist(X))), rel=1e-14)


def test_median_even_count_half_split():
    rng = np.random.default_rng(1)
    X = rng.standard_normal((40, 3))          # 780 pairs, even
    m = W.median_pairwise_distance(X)
    dists = pdist(X)
    assert np.count_nonzero(dists < m) == dists.size // 2


@pytest.mark.parametrize("name", ["C1", "C2", "C4", "H1"])
def test_workload_shapes(name):
    w = W.get(name)
    X, y = W.make_data(w)
    assert X.shape == (w.n, w.d) and X.dtype == np.float64 and X.flags.c_contiguous
    assert y.shape == (w.n,)
    if w.loss == "check":
        assert np.all(np.isfinite(y))
    else:
        assert set(np.unique(y).tolist()) == {-1.0, 1.0}
    lam = W.lambda_grid(w.lam_lo, w.lam_hi, w.L)
    assert lam.size == w.L and lam[0] == pytest.approx(10 ** w.lam_lo) and lam[-1] == pytest.approx(10 ** w.lam_hi)
    X2, y2 = W.make_data(w)
    assert np.array_equal(X, X2) and np.array_equal(y, y2)


def test_c1_class_means():
    X, y = W.make_data(W.get("C1"))
    assert np.all(y[:100] == 1) and np.all(y[100:] == -1)
    assert abs(X[:100].mean() - 0.5) < 0.1 and abs(X[100:].mean() + 0.5) < 0.1


def test_cell_counts():
    assert [W.get(k).cells for k in ["C1", "C2", "C3", "C4", "C5"]] == [50, 750, 1000, 600, 500]


def test_mixture_workload_structure():
    """The appendix mixture (H2, n = 10000): balanced classes; each class
    mean sits near its centres' mean (mu = 2 on its own half of the
    coordinates, 0 on the other, up to the spread of ten unit-variance
    centres); the within-class variance per coordinate is the centres'
    spread plus sigma = 3."""
    w = W.get("H2")
    X, y = W.make_data(w)
    assert np.count_nonzero(y == 1.0) == w.n // 2
    Xp, Xn = X[y == 1.0], X[y == -1.0]
    h = w.d // 2
    # the mean of ten N(mu, 1) centres has standard deviation 1/sqrt(10)
    assert np.all(np.abs(Xp[:, :h].mean(0) - 2.0) < 1.3) and np.all(np.abs(Xp[:, h:].mean(0)) < 1.3)
    assert np.all(np.abs(Xn[:, h:].mean(0) - 2.0) < 1.3) and np.all(np.abs(Xn[:, :h].mean(0)) < 1.3)
    # variance: 3 from the noise plus about 0.9 from the centres
    v = np.concatenate([Xp.var(0), Xn.var(0)])
    assert np.all(v > 3.0) and np.all(v < 6.0)
