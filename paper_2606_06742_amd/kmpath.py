"""ctypes binding of libkmpath.so: the same entry points as include/kmpath.h.

Argument marshalling only. Device arrays are torch tensors on the HIP device
(``torch.device("cuda")`` on ROCm); every computation runs in the library.
Loading fails loudly when the built library is missing: there is no
fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np

# KMPATH_LIB points the binding at another build of the library (the
# host-sanitized build of the CPU tests); default: the in-tree libkmpath.so
LIB_PATH = os.environ.get("KMPATH_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libkmpath.so")

KMP_OK, KMP_WMAXITER = 0, 1
KMP_EINVAL, KMP_EFOLD, KMP_EWORKSPACE, KMP_EHIP, KMP_ENONFINITE = -1, -2, -3, -4, -5
KMP_HINGE, KMP_LOGISTIC, KMP_CHECK = 0, 1, 2
KMP_FLAG_RESTART = 1
KMP_FLAG_GLOBAL_SOLVE = 2
KMP_FLAG_REFIT = 4
KMP_FLAG_SHARED_FACTOR = 8
KMP_FLAG_EXACT_HINGE = 16
KMP_FLAG_EAGER = 32
KMP_WNOTEXACT = 2
KMP_NKC = 10
KERNEL_CLASSES = ("gram", "panel", "panel_wy", "trail_update", "q_form", "precompute", "gemm_f",
                  "gemm_zhat", "update", "finalize")
LOSS_CODES = {"hinge": KMP_HINGE, "logistic": KMP_LOGISTIC, "check": KMP_CHECK}


class kmp_path_spec(C.Structure):
    _fields_ = [("loss", C.c_int32), ("delta0", C.c_double), ("eta", C.c_double),
                ("n_stages", C.c_int32), ("tol", C.c_double), ("max_iter", C.c_int32),
                ("poll_every", C.c_int32), ("flags", C.c_int32), ("timing_mask", C.c_int32),
                ("timing_every", C.c_int32)]


class kmp_timings(C.Structure):
    _fields_ = [("gram_ms", C.c_double), ("factor_ms", C.c_double),
                ("precompute_ms", C.c_double), ("path_ms", C.c_double),
                ("finalize_ms", C.c_double), ("total_ms", C.c_double),
                ("iterations", C.c_int64), ("cell_iterations", C.c_int64),
                ("kernel_ms", C.c_double * KMP_NKC), ("kernel_launches", C.c_int64 * KMP_NKC),
                ("kernel_seen", C.c_int64 * KMP_NKC),
                ("kernel_bytes", C.c_double * KMP_NKC), ("kernel_flops", C.c_double * KMP_NKC),
                ("kernel_ms_mb", C.c_double * KMP_NKC), ("kernel_launches_mb", C.c_int64 * KMP_NKC),
                ("kernel_bytes_mb", C.c_double * KMP_NKC), ("kernel_flops_mb", C.c_double * KMP_NKC)]

    def as_dict(self):
        return {k: (list(getattr(self, k)) if k.startswith("kernel_") else getattr(self, k))
                for k, _ in self._fields_}

    def kernels(self):
        """{class: (ms, bracketed launches, all launches, bytes, flops, and
        ms, launches, bytes, flops of the bracketed launches above the ridge
        point)} of the timed classes; ms, bytes and flops cover the bracketed
        launches."""
        return {KERNEL_CLASSES[i]: (self.kernel_ms[i], int(self.kernel_launches[i]),
                                    int(self.kernel_seen[i]), self.kernel_bytes[i],
                                    self.kernel_flops[i], self.kernel_ms_mb[i],
                                    int(self.kernel_launches_mb[i]), self.kernel_bytes_mb[i],
                                    self.kernel_flops_mb[i])
                for i in range(KMP_NKC) if self.kernel_launches[i] > 0}


class KmpError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"kmpath error {code}: {msg}")
        self.code = code


_lib = None
_VP, _DP, _IP = C.c_void_p, C.POINTER(C.c_double), C.POINTER(C.c_int32)


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_06742_amd.build`")
        L = C.CDLL(LIB_PATH)
        L.kmp_default_spec.argtypes = [C.POINTER(kmp_path_spec)]
        L.kmp_default_spec.restype = None
        L.kmp_workspace_bytes.argtypes = [C.POINTER(kmp_path_spec), C.c_int64, C.c_int64, C.c_int32,
                                          _IP, C.c_int32, C.c_int32, C.c_int32, C.c_int32]
        L.kmp_workspace_bytes.restype = C.c_size_t
        L.kmp_fit_path.argtypes = [_VP, C.POINTER(kmp_path_spec), _VP, C.c_int64, C.c_int64,
                                   C.c_int64, _VP, _DP, C.c_int32, _DP, C.c_int32, _DP, C.c_int32,
                                   _IP, C.c_int32, _VP, C.c_size_t, _VP, _VP, _VP, _VP, _VP, _VP,
                                   _VP, _IP, _IP, C.POINTER(kmp_timings)]
        L.kmp_fit_path.restype = C.c_int
        L.kmp_make_folds.argtypes = [C.c_int64, C.c_int32, C.c_uint64, _IP]
        L.kmp_make_folds.restype = C.c_int
        L.kmp_rbf_gram.argtypes = [_VP, _VP, C.c_int64, C.c_int64, C.c_int64, _VP, C.c_int64, _VP,
                                   C.c_int64, _DP, C.c_int32, _VP, C.c_int64]
        L.kmp_rbf_gram.restype = C.c_int
        L.kmp_rbf_gram_noalloc.argtypes = L.kmp_rbf_gram.argtypes
        L.kmp_rbf_gram_noalloc.restype = C.c_int
        L.kmp_tridiag.argtypes = [_VP, _VP, C.c_int32, C.c_int32, _VP, _VP, _VP]
        L.kmp_tridiag.restype = C.c_int
        L.kmp_band_reduce.argtypes = [_VP, _VP, C.c_int32, C.c_int32, _VP, _VP]
        L.kmp_band_reduce.restype = C.c_int
        L.kmp_path_step.argtypes = [_VP, C.c_int32, C.c_double, _VP, C.c_int64, _VP, _DP, _DP,
                                    C.c_int32, _VP, _VP, _VP, _VP, _VP]
        L.kmp_path_step.restype = C.c_int
        L.kmp_dgemm_grouped.argtypes = [_VP, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _VP, _VP,
                                        _VP]
        L.kmp_dgemm_grouped.restype = C.c_int
        L.kmp_strerror.argtypes = [C.c_int]
        L.kmp_strerror.restype = C.c_char_p
        L.kmp_version.argtypes = []
        L.kmp_version.restype = C.c_char_p
        L.kmp_kernel_class_name.argtypes = [C.c_int]
        L.kmp_kernel_class_name.restype = C.c_char_p
        _lib = L
    return _lib


EXPORTED = ("kmp_default_spec", "kmp_workspace_bytes", "kmp_fit_path", "kmp_make_folds",
            "kmp_rbf_gram", "kmp_rbf_gram_noalloc", "kmp_tridiag", "kmp_band_reduce",
            "kmp_path_step",
            "kmp_dgemm_grouped", "kmp_strerror", "kmp_version", "kmp_kernel_class_name")
KMP_BAND = 16


def kmp_kernel_class_name(cls: int) -> str:
    return lib().kmp_kernel_class_name(int(cls)).decode()


def kmp_strerror(code: int) -> str:
    return lib().kmp_strerror(int(code)).decode()


def kmp_version() -> str:
    return lib().kmp_version().decode()


def _check(code: int, allow_maxiter: bool = True) -> int:
    if code == KMP_OK or (allow_maxiter and code in (KMP_WMAXITER, KMP_WNOTEXACT)):
        return code
    raise KmpError(code, kmp_strerror(code))


def kmp_default_spec(loss: str = "hinge", **overrides) -> kmp_path_spec:
    s = kmp_path_spec()
    lib().kmp_default_spec(C.byref(s))
    s.loss = LOSS_CODES[loss] if isinstance(loss, str) else int(loss)
    for k, v in overrides.items():
        setattr(s, k, v)
    return s


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def kmp_make_folds(n: int, V: int, seed: int) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    _check(lib().kmp_make_folds(int(n), int(V), C.c_uint64(seed & (2 ** 64 - 1)),
                                out.ctypes.data_as(_IP)))
    return out


def kmp_workspace_bytes(spec, n, d, L, fold_id, V, S, Q, sigma_batch) -> int:
    f = _i32(fold_id)
    return int(lib().kmp_workspace_bytes(C.byref(spec), int(n), int(d), int(L),
                                         f.ctypes.data_as(_IP), int(V), int(S), int(Q),
                                         int(sigma_batch)))


def _stream_ptr(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def kmp_rbf_gram(X, rows, cols, sigmas, out, stream=None) -> None:
    """a1 on its own (see kmpath.h). X, rows, cols, out are device tensors."""
    sig = _f64(sigmas)
    _check(lib().kmp_rbf_gram(_stream_ptr(stream), X.data_ptr(), X.shape[0], X.shape[1],
                              X.stride(0), rows.data_ptr(), rows.numel(), cols.data_ptr(),
                              cols.numel(), sig.ctypes.data_as(_DP), sig.size, out.data_ptr(),
                              out.stride(-2)))


def kmp_tridiag(A, Q, diag, off, stream=None) -> None:
    """a2 on its own: A (G, N, N) device tensor, destroyed; Q/diag/off outputs."""
    G, N = A.shape[0], A.shape[1]
    _check(lib().kmp_tridiag(_stream_ptr(stream), A.data_ptr(), G, N, Q.data_ptr(),
                             diag.data_ptr(), off.data_ptr()))


def kmp_band_reduce(A, Q, band, stream=None) -> None:
    """a2 on its own, band form: A (G, N, N) device tensor, destroyed; Q
    (G, N, N) and band (G, KMP_BAND+1, N) outputs, band[g, r, j] = B[j+r, j]."""
    G, N = A.shape[0], A.shape[1]
    _check(lib().kmp_band_reduce(_stream_ptr(stream), A.data_ptr(), G, N, Q.data_ptr(),
                                 band.data_ptr()))


def kmp_path_step(loss, delta, K, y, lambdas, alpha_in, beta_in, alpha_out, beta_out,
                  kkt_out=None, taus=None, stream=None) -> None:
    """a4-a7 on their own (see kmpath.h): K (n, n), y (n), alpha (C, n), beta
    (C) device tensors; lambdas (and taus) host arrays of C entries."""
    lam = _f64(lambdas)
    tau = _f64(taus) if taus is not None else None
    code = lib().kmp_path_step(
        _stream_ptr(stream), LOSS_CODES[loss] if isinstance(loss, str) else int(loss),
        float(delta if delta is not None else 1.0), K.data_ptr(), K.shape[0], y.data_ptr(),
        lam.ctypes.data_as(_DP), tau.ctypes.data_as(_DP) if tau is not None else None, lam.size,
        alpha_in.data_ptr(), beta_in.data_ptr(), alpha_out.data_ptr(), beta_out.data_ptr(),
        kkt_out.data_ptr() if kkt_out is not None else None)
    _check(code, allow_maxiter=False)


def kmp_dgemm_grouped(A, B, C, stream=None) -> None:
    """C[g] = A[g] @ B[g] for (G, M, K), (G, K, N), (G, M, N) device tensors."""
    G, M, K = A.shape
    N = B.shape[2]
    _check(lib().kmp_dgemm_grouped(_stream_ptr(stream), G, M, N, K, A.data_ptr(), B.data_ptr(),
                                   C.data_ptr()), allow_maxiter=False)


def kmp_fit_path(stream, spec, X, y, sigmas, taus, lambdas, fold_id, V, workspace, ws_bytes,
                 alpha, beta, objective, cv_sum, cv_err, iters, status, selected, timings,
                 selected_joint=None) -> int:
    """Direct call of the C entry point (device pointers as ints, host arrays as numpy)."""
    sig, tau, lam, fold = _f64(sigmas), _f64(taus), _f64(lambdas), _i32(fold_id)
    return lib().kmp_fit_path(
        stream, C.byref(spec), X.data_ptr(), X.shape[0], X.shape[1], X.stride(0), y.data_ptr(),
        sig.ctypes.data_as(_DP), sig.size, tau.ctypes.data_as(_DP), max(1, tau.size),
        lam.ctypes.data_as(_DP), lam.size, fold.ctypes.data_as(_IP), int(V), workspace,
        int(ws_bytes), alpha.data_ptr(), beta.data_ptr(), objective.data_ptr(), cv_sum.data_ptr(),
        cv_err.data_ptr() if cv_err is not None else None,
        iters.data_ptr() if iters is not None else None,
        status.data_ptr() if status is not None else None,
        selected.ctypes.data_as(_IP) if selected is not None else None,
        selected_joint.ctypes.data_as(_IP) if selected_joint is not None else None,
        C.byref(timings) if timings is not None else None)


class PathRunner:
    """Holds the workspace and output tensors for repeated fits of one problem shape."""

    def __init__(self, X, y, loss, sigmas, lambdas, fold_id, V, taus=None, device="cuda",
                 sigma_batch: Optional[int] = None, kernel_timing=(), refit: bool = False,
                 shared: bool = False, exact_hinge: bool = False, eager: bool = False,
                 **spec_overrides):
        """refit=True: every (sigma, tau, lambda) on all n points (fold_id and V
        are ignored; outputs have V = 1, no CV sums, no selection).
        shared=True: exact CV on one factor of the full K per bandwidth
        (KMP_FLAG_SHARED_FACTOR); V = n with fold_id = 0..n-1 is leave-one-out.
        eager=True: every iteration launched directly, never from a recorded
        HIP graph (KMP_FLAG_EAGER)."""
        import torch
        self.torch = torch
        self.loss = loss
        self.spec = kmp_default_spec(loss, **spec_overrides)
        if refit:
            self.spec.flags |= KMP_FLAG_REFIT
            fold_id, V = np.zeros(np.shape(X)[0], dtype=np.int32), 1
        if shared:
            self.spec.flags |= KMP_FLAG_SHARED_FACTOR
        if exact_hinge:
            self.spec.flags |= KMP_FLAG_EXACT_HINGE
        if eager:
            self.spec.flags |= KMP_FLAG_EAGER
        self.set_kernel_timing(kernel_timing)
        self.X = torch.as_tensor(np.ascontiguousarray(X), dtype=torch.float64, device=device) \
            if not isinstance(X, torch.Tensor) else X
        self.y = torch.as_tensor(np.ascontiguousarray(y), dtype=torch.float64, device=device) \
            if not isinstance(y, torch.Tensor) else y
        self.sigmas = _f64(np.atleast_1d(sigmas))
        self.lambdas = _f64(lambdas)
        self.taus = _f64(taus) if (loss == "check") else np.zeros(1)
        self.fold = _i32(fold_id)
        self.V = int(V)
        n, d = self.X.shape
        S, Q, L = self.sigmas.size, (self.taus.size if loss == "check" else 1), self.lambdas.size
        self.shape = (S, Q, self.V, L)
        sb = S if sigma_batch is None else int(sigma_batch)
        self.ws_bytes = kmp_workspace_bytes(self.spec, n, d, L, self.fold, self.V, S, Q, sb)
        if self.ws_bytes == 0:
            raise KmpError(KMP_EINVAL, "invalid problem for workspace sizing")
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        cells = S * Q * self.V * L
        self.alpha = torch.empty((S, Q, self.V, L, n), dtype=torch.float64, device=device)
        self.beta = torch.empty(self.shape, dtype=torch.float64, device=device)
        self.objective = torch.empty(self.shape, dtype=torch.float64, device=device)
        self.cv_sum = torch.empty(self.shape, dtype=torch.float64, device=device)
        self.cv_err = torch.empty(self.shape, dtype=torch.int32, device=device)
        self.iters = torch.empty(self.shape, dtype=torch.int32, device=device)
        self.status = torch.empty(self.shape, dtype=torch.int32, device=device)
        self.selected = np.zeros((S, Q), dtype=np.int32)
        self.selected_joint = np.zeros((Q, 2), dtype=np.int32)
        self.timings = kmp_timings()
        self.cells = cells

    def set_kernel_timing(self, classes, every: int = 1) -> None:
        """Time the named kernel classes with HIP events on the next runs,
        bracketing one launch in every `every` of each class."""
        mask = 0
        for c in classes:
            mask |= 1 << (KERNEL_CLASSES.index(c) if isinstance(c, str) else int(c))
        self.spec.timing_mask = mask
        self.spec.timing_every = int(every)

    def kernel_times(self) -> dict:
        return self.timings.kernels()

    def run(self, stream=None) -> int:
        code = kmp_fit_path(_stream_ptr(stream), self.spec, self.X, self.y, self.sigmas,
                            self.taus, self.lambdas, self.fold, self.V, self.workspace.data_ptr(),
                            self.ws_bytes, self.alpha, self.beta, self.objective, self.cv_sum,
                            self.cv_err, self.iters, self.status, self.selected, self.timings,
                            self.selected_joint)
        return _check(code)

    def results(self) -> dict:
        out = {k: getattr(self, k).cpu().numpy() for k in
               ("alpha", "beta", "objective", "cv_sum", "cv_err", "iters", "status")}
        out["selected"] = self.selected.copy()
        out["selected_joint"] = self.selected_joint.copy()
        out["timings"] = self.timings.as_dict()
        return out


def fit_path(X, y, loss, sigmas, lambdas, fold_id, V, taus=None, **spec_overrides) -> dict:
    """One call of kmp_fit_path with freshly allocated outputs; returns numpy results."""
    r = PathRunner(X, y, loss, sigmas, lambdas, fold_id, V, taus=taus, **spec_overrides)
    code = r.run()
    out = r.results()
    out["code"] = code
    return out
