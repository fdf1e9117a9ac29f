"""The allocation-free Gram entry point (kmp_rbf_gram_noalloc, for callers
that cannot allocate device memory) against kmp_rbf_gram: the same kernels
on the same inputs, two calls in a row (the second smaller, reusing the
static scratch), and its size limit refused on the host."""
import numpy as np
import pytest

from tests.gpu_common import announce, device

pytestmark = pytest.mark.gpu


def _call(fn, X, rows, cols, sigmas, out):
    import ctypes as C
    from paper_2606_06742_amd import kmpath as km
    sig = np.ascontiguousarray(sigmas, dtype=np.float64)
    return fn(km._stream_ptr(None), X.data_ptr(), X.shape[0], X.shape[1], X.stride(0),
              rows.data_ptr(), rows.numel(), cols.data_ptr(), cols.numel(),
              sig.ctypes.data_as(C.POINTER(C.c_double)), sig.size, out.data_ptr(), out.stride(-2))


def test_rbf_gram_noalloc_matches_allocating_entry_point():
    import torch
    from paper_2606_06742_amd import kmpath as km
    dev = device()
    L = km.lib()
    rng = np.random.default_rng(29)
    for (n, d, m, p, S) in [(300, 7, 100, 90, 2), (120, 3, 50, 40, 1)]:
        announce(f"kmp_rbf_gram_noalloc n={n} d={d} m={m} p={p} S={S}")
        X = torch.as_tensor(rng.standard_normal((n, d)), device=dev)
        r = rng.integers(0, n, m).astype(np.int32)
        c = rng.integers(0, n, p).astype(np.int32)
        r[-3:] = -1                                   # padding rows
        c[:2] = r[:2]                                 # some diagonal entries
        rows = torch.as_tensor(r, device=dev)
        cols = torch.as_tensor(c, device=dev)
        sig = rng.uniform(0.5, 3.0, S)
        ref = torch.full((S, m, p), np.nan, dtype=torch.float64, device=dev)
        got = torch.full((S, m, p), np.nan, dtype=torch.float64, device=dev)
        assert _call(L.kmp_rbf_gram, X, rows, cols, sig, ref) == km.KMP_OK
        assert _call(L.kmp_rbf_gram_noalloc, X, rows, cols, sig, got) == km.KMP_OK
        torch.cuda.synchronize()
        a, b = ref.cpu().numpy(), got.cpu().numpy()
        assert np.all(np.isfinite(b))
        assert np.array_equal(a, b)
    # above the static scratch: refused before any launch (X is large enough
    # that no access could leave it in any case)
    n = 70000
    X = torch.zeros((n, 1), dtype=torch.float64, device=dev)
    rows = torch.zeros(4, dtype=torch.int32, device=dev)
    out = torch.zeros((1, 4, 4), dtype=torch.float64, device=dev)
    assert _call(L.kmp_rbf_gram_noalloc, X, rows, rows, [1.0], out) == km.KMP_EINVAL
    assert "static scratch" in km.kmp_strerror(km.KMP_EINVAL)
