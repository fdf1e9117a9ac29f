"""The C-ABI library on the host: symbols, fold generator, validation errors.

No GPU is needed: every call here returns before the library touches the
device (argument errors are detected on the host first).
"""
import ctypes as C
import os
import re

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kmpath.h")


@pytest.fixture(scope="module")
def km():
    from paper_2606_06742_amd import kmpath
    if not os.path.exists(kmpath.LIB_PATH):
        from paper_2606_06742_amd import build
        build.build()
    kmpath.lib()
    return kmpath


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kmp_[a-z_]+)\s*\(", src)))


def test_header_symbols_exported(km):
    names = _declared()
    assert {"kmp_fit_path", "kmp_workspace_bytes", "kmp_make_folds", "kmp_rbf_gram",
            "kmp_tridiag", "kmp_strerror", "kmp_version", "kmp_default_spec"} <= set(names)
    L = km.lib()
    for name in names:
        assert hasattr(L, name), name
    assert set(km.EXPORTED) == set(names)


def test_make_folds_bit_exact(km):
    for n, V, seed in [(200, 5, 2001), (2000, 5, 2002), (10000, 10, 2003), (203, 5, 9), (5, 5, 0),
                       (17, 3, 2 ** 63 + 12345)]:
        assert np.array_equal(km.kmp_make_folds(n, V, seed), W.make_folds(n, V, seed))


def test_default_spec(km):
    s = km.kmp_default_spec("logistic")
    assert s.loss == km.KMP_LOGISTIC and s.delta0 == 1.0 and s.eta == 0.125
    assert s.n_stages == 3 and s.tol == 1e-9 and s.flags & km.KMP_FLAG_RESTART


def test_workspace_bytes(km):
    w = W.get("C2")
    fold = W.make_folds(w.n, w.V, w.fold_seed)
    spec = km.kmp_default_spec("logistic")
    b3 = km.kmp_workspace_bytes(spec, w.n, w.d, w.L, fold, w.V, 3, 1, 3)
    b1 = km.kmp_workspace_bytes(spec, w.n, w.d, w.L, fold, w.V, 3, 1, 1)
    N = 1600
    assert b3 > 3 * 5 * 2 * N * N * 8 and b1 < b3 and b1 > 5 * 2 * N * N * 8
    assert km.kmp_workspace_bytes(spec, w.n, w.d, w.L, fold, w.V, 3, 1, 4) == 0
    bad = fold.copy()
    bad[0] = 7
    assert km.kmp_workspace_bytes(spec, w.n, w.d, w.L, bad, w.V, 3, 1, 1) == 0


class _Fake:
    """Stands in for a device tensor in calls that fail validation first."""

    def __init__(self, shape, ptr=0x1000):
        self.shape = shape
        self._ptr = ptr

    def data_ptr(self):
        return self._ptr

    def stride(self, i):
        return self.shape[1] if i == 0 else 1


def _call(km, loss="hinge", n=20, d=3, sigmas=(1.0,), lambdas=(0.1, 1.0), fold=None, V=4,
          taus=(0.5,), ws=1 << 20, spec=None):
    fold = np.arange(n) % V if fold is None else fold
    spec = spec or km.kmp_default_spec(loss)
    X, y = _Fake((n, d)), _Fake((n,))
    out = _Fake((1,))
    return km.kmp_fit_path(None, spec, X, y, np.array(sigmas), np.array(taus), np.array(lambdas),
                           fold, V, 0x2000, ws, out, out, out, out, None, None, None, None, None)


def test_refit_flag_shapes(km):
    """A full-data refit (KMP_FLAG_REFIT) is one fold with no held-out rows:
    it takes V = 1, needs no fold ids, and its workspace holds one group of
    all n rows per bandwidth; without the flag V = 1 is refused."""
    w = W.get("C2")
    spec = km.kmp_default_spec("logistic")
    spec.flags |= km.KMP_FLAG_REFIT
    zeros = np.zeros(w.n, dtype=np.int32)
    b_refit = km.kmp_workspace_bytes(spec, w.n, w.d, w.L, zeros, 1, 3, 1, 3)
    assert b_refit > 0
    assert km.kmp_workspace_bytes(spec, w.n, w.d, w.L, zeros, 2, 3, 1, 3) == 0
    plain = km.kmp_default_spec("logistic")
    assert km.kmp_workspace_bytes(plain, w.n, w.d, w.L, zeros, 1, 3, 1, 3) == 0
    fold = km.kmp_make_folds(w.n, w.V, 1)
    b_cv = km.kmp_workspace_bytes(plain, w.n, w.d, w.L, fold, w.V, 3, 1, 3)
    # V groups of n(V-1)/V rows against one group of n rows per bandwidth
    assert b_refit < b_cv


def test_fit_path_argument_errors(km):
    assert _call(km, sigmas=(0.0,)) == km.KMP_EINVAL
    assert _call(km, sigmas=(np.inf,)) == km.KMP_EINVAL
    assert _call(km, lambdas=(0.1, -1.0)) == km.KMP_EINVAL
    assert _call(km, loss="check", taus=(1.0,)) == km.KMP_EINVAL
    assert _call(km, loss="check", taus=(0.0,)) == km.KMP_EINVAL
    fold = np.arange(20) % 4
    fold[3] = 9
    assert _call(km, fold=fold) == km.KMP_EFOLD
    assert _call(km, fold=np.arange(20) % 3, V=4) == km.KMP_EFOLD       # fold 3 empty
    assert _call(km, V=1, fold=np.zeros(20, dtype=np.int32)) == km.KMP_EINVAL
    spec = km.kmp_default_spec("hinge", eta=1.5)
    assert _call(km, spec=spec) == km.KMP_EINVAL
    spec = km.kmp_default_spec("hinge", tol=0.0)
    assert _call(km, spec=spec) == km.KMP_EINVAL
    assert "fold" in km.kmp_strerror(km.KMP_EFOLD) or km.kmp_strerror(km.KMP_EFOLD)
    assert km.kmp_version().startswith("kmpath")


def test_binding_refuses_missing_library(monkeypatch):
    from paper_2606_06742_amd import kmpath
    monkeypatch.setattr(kmpath, "_lib", None)
    monkeypatch.setattr(kmpath, "LIB_PATH", "/nonexistent/libkmpath.so")
    with pytest.raises(RuntimeError):
        kmpath.lib()


def test_shared_factor_workspace(km):
    """KMP_FLAG_SHARED_FACTOR: one group of all n rows per bandwidth with
    V x L columns; refused together with a refit, with V > n, and above the
    largest shared order."""
    w = W.get("C3")
    fold = W.make_folds(w.n, w.V, w.fold_seed)
    spec = km.kmp_default_spec("hinge")
    spec.flags |= km.KMP_FLAG_SHARED_FACTOR
    b = km.kmp_workspace_bytes(spec, w.n, w.d, w.L, fold, w.V, 1, 1, 1)
    N = 10048                              # 10000 rounded up to 64
    assert b > 2 * N * N * 8
    plain = km.kmp_default_spec("hinge")
    b_fold = km.kmp_workspace_bytes(plain, w.n, w.d, w.L, fold, w.V, 1, 1, 1)
    assert b < b_fold                      # one n x n pair against ten of 9024 x 9024
    # leave-one-out: V = n, fold i = point i
    loo = np.arange(200, dtype=np.int32)
    assert km.kmp_workspace_bytes(spec, 200, 3, 10, loo, 200, 1, 1, 1) > 0
    assert km.kmp_workspace_bytes(spec, 200, 3, 10, loo, 201, 1, 1, 1) == 0
    both = km.kmp_default_spec("hinge")
    both.flags |= km.KMP_FLAG_SHARED_FACTOR | km.KMP_FLAG_REFIT
    assert km.kmp_workspace_bytes(both, 200, 3, 10, np.zeros(200, np.int32), 1, 1, 1, 1) == 0
    big = np.arange(41000, dtype=np.int32) % 5
    assert km.kmp_workspace_bytes(spec, 41000, 3, 2, big, 5, 1, 1, 1) == 0


def test_single_step_entry_points_validate_on_host(km):
    """kmp_path_step and kmp_dgemm_grouped refuse bad arguments before any
    device work; an empty product is a no-op."""
    L = km.lib()
    lam = np.array([0.1, -1.0])
    tau = np.array([0.5, 0.5])
    dp = lambda a: a.ctypes.data_as(C.POINTER(C.c_double))
    ok_lam = np.array([0.1, 1.0])
    # negative lambda, bad tau, bad loss, n < 2
    assert L.kmp_path_step(None, 0, 0.1, 0x1000, 50, 0x1000, dp(lam), None, 2, 0x1000, 0x1000,
                           0x1000, 0x1000, None) == km.KMP_EINVAL
    assert L.kmp_path_step(None, 2, 0.1, 0x1000, 50, 0x1000, dp(ok_lam), dp(np.array([0.5, 1.0])),
                           2, 0x1000, 0x1000, 0x1000, 0x1000, None) == km.KMP_EINVAL
    assert L.kmp_path_step(None, 7, 0.1, 0x1000, 50, 0x1000, dp(ok_lam), None, 2, 0x1000, 0x1000,
                           0x1000, 0x1000, None) == km.KMP_EINVAL
    assert L.kmp_path_step(None, 0, 0.1, 0x1000, 1, 0x1000, dp(ok_lam), None, 2, 0x1000, 0x1000,
                           0x1000, 0x1000, None) == km.KMP_EINVAL
    assert L.kmp_path_step(None, 0, 0.0, 0x1000, 50, 0x1000, dp(ok_lam), dp(tau), 2, 0x1000,
                           0x1000, 0x1000, 0x1000, None) == km.KMP_EINVAL
    assert L.kmp_dgemm_grouped(None, -1, 4, 4, 4, 0x1000, 0x1000, 0x1000) == km.KMP_EINVAL
    assert L.kmp_dgemm_grouped(None, 2, 4, 4, 4, None, 0x1000, 0x1000) == km.KMP_EINVAL
    assert L.kmp_dgemm_grouped(None, 0, 4, 4, 4, None, None, None) == km.KMP_OK


def test_exact_hinge_flag_validation(km):
    """KMP_FLAG_EXACT_HINGE needs the hinge loss and per-fold factors."""
    fold = np.arange(20, dtype=np.int32) % 4
    for loss, extra in (("logistic", 0), ("check", 0), ("hinge", km.KMP_FLAG_SHARED_FACTOR)):
        spec = km.kmp_default_spec(loss)
        spec.flags |= km.KMP_FLAG_EXACT_HINGE | extra
        assert km.kmp_workspace_bytes(spec, 20, 3, 2, fold, 4, 1, 1, 1) == 0
    spec = km.kmp_default_spec("hinge")
    spec.flags |= km.KMP_FLAG_EXACT_HINGE
    assert km.kmp_workspace_bytes(spec, 20, 3, 2, fold, 4, 1, 1, 1) > 0
