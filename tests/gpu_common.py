"""Shared helpers for the GPU tests (parity bars and announcements)."""
import sys

import numpy as np

from oracle import gram as OG
from oracle import losses as OL
from oracle.cell import CONVERGED_KKT

OBJ_RTOL = 1e-8      # objectives, relative
ALPHA_RTOL = 1e-6    # coefficients, relative to max |alpha|
CV_RTOL = 1e-6       # held-out loss sums
# the oracle's own residual n_v max(||z + 2 lambda alpha||_inf, |1'z|) at
# every cell it serves as the reference for (extended precision; the GPU
# stops at 1e-9 in its own norm)
ORACLE_KKT = CONVERGED_KKT


def announce(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def device():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU test run without a visible HIP device")
    return torch.device("cuda")


def compare_cells(g, o, inp, loss, cells=None, delta=2.0 ** -6, cv_expected=None):
    """Element-wise parity of GPU results g against oracle results o.

    cells: iterable of (s, q, v, l) to check, default all. Returns the worst
    relative errors seen, for reporting. cv_expected, if given (shape of
    o["cv_sum"]), receives the held-out loss sum each checked cell is held
    to: the oracle's, or, where the optimal intercept is an interval, the
    oracle's held-out loss at the GPU's intercept.
    """
    S, Q, V, L = g["objective"].shape
    X, y, fold = inp["X"], inp["y"], inp["fold_id"]
    worst = {"obj": 0.0, "alpha": 0.0, "beta": 0.0, "cv": 0.0, "oracle_kkt": 0.0}
    if cells is None:
        cells = [(s, q, v, l) for s in range(S) for q in range(Q) for v in range(V) for l in range(L)]
    blocks = {}
    for (s, q, v, l) in cells:
        key = (s, v)
        if key not in blocks:
            # only the held-out block K[H_v, T_v] is needed here
            T = np.flatnonzero(fold != v)
            H = np.flatnonzero(fold == v)
            blocks[key] = (OG.rbf_gram(X[H], X[T], inp["sigmas"][s]), T, H)
        Kc, T, H = blocks[key]
        tau = inp["taus"][q] if loss == "check" else None
        # the reference itself must be solved: its own residual, not a stall
        ko = float(o["kkt"][s, q, v, l])
        assert ko <= ORACLE_KKT, ("oracle cell not converged", (s, q, v, l), ko)
        worst["oracle_kkt"] = max(worst["oracle_kkt"], ko)
        Fo, Fg = o["objective"][s, q, v, l], g["objective"][s, q, v, l]
        assert abs(Fg - Fo) <= OBJ_RTOL * abs(Fo), ((s, q, v, l), Fg, Fo)
        worst["obj"] = max(worst["obj"], abs(Fg - Fo) / abs(Fo))
        ao, ag = o["alpha"][s, q, v, l], g["alpha"][s, q, v, l]
        assert np.all(ag[H] == 0.0)
        scale = np.abs(ao).max()
        err = np.abs(ag - ao).max()
        assert err <= ALPHA_RTOL * scale + 1e-15, ((s, q, v, l), err, scale)
        worst["alpha"] = max(worst["alpha"], err / max(scale, 1e-300))
        bo, bg = o["beta"][s, q, v, l], g["beta"][s, q, v, l]
        lo, hi = o["beta_lo"][s, q, v, l], o["beta_hi"][s, q, v, l]
        btol = ALPHA_RTOL * max(1.0, abs(bo))
        assert lo - btol <= bg <= hi + btol, ((s, q, v, l), bg, bo, lo, hi)
        if lo == hi:
            worst["beta"] = max(worst["beta"], abs(bg - bo) / max(1.0, abs(bo)))
        co, cg = o["cv_sum"][s, q, v, l], g["cv_sum"][s, q, v, l]
        if lo < hi:
            # the intercept is not unique and the held-out loss depends on
            # it: the expected sum is the oracle's held-out loss at the
            # oracle's alpha and the GPU's (admissible) intercept
            co = float(OL.eval_loss(loss, y[H], Kc @ ao[T] + bg, tau).sum())
        if cv_expected is not None:
            cv_expected[s, q, v, l] = co
        assert abs(cg - co) <= CV_RTOL * max(1.0, abs(co)), ((s, q, v, l), cg, co)
        worst["cv"] = max(worst["cv"], abs(cg - co) / max(1.0, abs(co)))
        if loss != "check":
            # misclassified held-out points at the oracle's alpha and the
            # intercept the sum above was held to; points within 1e-6 of the
            # boundary may go either way
            fH = Kc @ ao[T] + (bg if lo < hi else bo)
            border = int(np.count_nonzero(np.abs(fH) < 1e-6))
            eo = int(np.count_nonzero(y[H] * fH <= 0.0)) if lo < hi else int(o["cv_err"][s, q, v, l])
            assert abs(int(g["cv_err"][s, q, v, l]) - eo) <= border, ((s, q, v, l), g["cv_err"][s, q, v, l], eo)
    return worst


def kkt_of(Kv, yT, a, b, lam, loss, delta, tau):
    n = yT.shape[0]
    f = Kv @ a + b
    z = OL.point_psi(loss, yT, f, delta, tau) / n
    return n * max(np.abs(z + 2 * lam * a).max(), abs(z.sum()))


def expected_selection(o, cv_expected, lambdas, n):
    """Selected lambda index per (sigma, tau) from the expected held-out sums
    (the oracle's selection rule: argmin of the pooled mean, ties to the
    larger lambda)."""
    from oracle.path import select
    S, Q = cv_expected.shape[:2]
    out = np.zeros((S, Q), dtype=np.int32)
    for s in range(S):
        for q in range(Q):
            out[s, q], _ = select(cv_expected[s, q], lambdas, n)
    return out


def oracle_cells(inp, loss, cells, shape, delta=2.0 ** -6):
    """Independent oracle solves of the given (s, q, v, l) cells, laid out
    like the GPU results of the given (S, Q, V, L, n) shape (other cells 0)."""
    import oracle
    S, Q, V, L, n = shape
    o = {k: np.zeros((S, Q, V, L)) for k in ("beta", "objective", "cv_sum", "cv_err", "kkt",
                                             "beta_lo", "beta_hi")}
    o["alpha"] = np.zeros(shape)
    X, y, fold = inp["X"], inp["y"], inp["fold_id"]
    blocks = {}
    d = None if loss == "logistic" else delta
    for (s, q, v, l) in cells:
        if (s, v) not in blocks:
            blocks[(s, v)] = OG.fold_blocks(X, fold, v, inp["sigmas"][s])
        Kv, Kc, T, H = blocks[(s, v)]
        tau = inp["taus"][q] if loss == "check" else None
        lam = inp["lambdas"][l]
        a, b, info = oracle.solve_cell(Kv, y[T], lam, loss, d, tau)
        o["alpha"][s, q, v, l][T] = a
        o["beta"][s, q, v, l] = b
        o["beta_lo"][s, q, v, l], o["beta_hi"][s, q, v, l] = oracle.beta_interval(
            Kv, y[T], a, b, loss, d, tau)
        o["objective"][s, q, v, l] = oracle.objective(Kv, y[T], a, b, lam, loss, d, tau)
        fH = Kc @ a + b
        o["cv_sum"][s, q, v, l] = OL.eval_loss(loss, y[H], fH, tau).sum()
        o["cv_err"][s, q, v, l] = np.count_nonzero(y[H] * fH <= 0) if loss != "check" else 0
        o["kkt"][s, q, v, l] = info["kkt"]
    return o


def fixture(name):
    """An oracle-written fixture of tests/golden (see make_oracle_fixtures.py)."""
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", name)
    return dict(np.load(path, allow_pickle=False))


def fixture_cells(fx, shape, T, s=0, q=0, v=0):
    """Oracle results of a fixture's cells (fold v), in the GPU layout."""
    S, Q, V, L, n = shape
    o = {k: np.zeros((S, Q, V, L)) for k in ("beta", "objective", "cv_sum", "cv_err", "kkt",
                                             "beta_lo", "beta_hi")}
    o["alpha"] = np.zeros(shape)
    cells = []
    for i, l in enumerate(fx["l"]):
        l = int(l)
        cells.append((s, q, v, l))
        o["alpha"][s, q, v, l][T] = fx["alpha_T"][i]
        for k in ("beta", "objective", "cv_sum", "cv_err", "kkt", "beta_lo", "beta_hi"):
            o[k][s, q, v, l] = fx[k][i]
    return o, cells


def check_selection(g, sel, n, what):
    """Every cell's held-out loss sum against the oracle's (sel["cv_sum"]
    [s, v, l], Q = 1), then the selected penalty per bandwidth and the joint
    (sigma, lambda) choice."""
    cg = g["cv_sum"][:, 0]
    co = sel["cv_sum"]
    assert cg.shape == co.shape, (cg.shape, co.shape)
    assert np.all(sel["kkt"] <= ORACLE_KKT), ("oracle cells not converged", what,
                                             float(sel["kkt"].max()))
    rel = np.abs(cg - co) / np.maximum(1.0, np.abs(co))
    bad = np.argwhere(rel > CV_RTOL)
    assert bad.size == 0, (what, "held-out sums", bad[:5], rel.max())
    assert np.array_equal(g["selected"][:, 0], sel["selected"]), (what, g["selected"], sel["selected"])
    assert np.array_equal(g["selected_joint"][0], sel["selected_joint"]), (
        what, g["selected_joint"], sel["selected_joint"])
    return float(rel.max())
