"""The dense majorise-minimise step: literal H solve, block inverse, monotonicity."""
import numpy as np
import pytest

import workloads as W
from oracle import cell, gram, mm, losses as Ls

CASES = [("hinge", 0.125, None), ("logistic", None, None), ("check", 2.0 ** -6, 0.3)]


def _wellcond_problem(loss, seed=0, n=30):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, 3)) * 2.0
    K = gram.rbf_gram(X, X, 0.8)                  # close to identity: well conditioned
    y = rng.standard_normal(n) if loss == "check" else np.where(rng.random(n) < 0.5, 1.0, -1.0)
    return K, y, rng


@pytest.mark.parametrize("loss,delta,tau", CASES)
def test_mm_step_equals_literal_h_solve(loss, delta, tau):
    K, y, rng = _wellcond_problem(loss)
    assert np.linalg.cond(K) < 1e3
    for lam in [1e-3, 0.1, 3.0]:
        a = rng.standard_normal(len(y)) * 0.3
        b = float(rng.normal())
        a1, b1 = mm.mm_step(K, y, a, b, lam, loss, delta, tau)
        a2, b2 = mm.mm_step_literal(K, y, a, b, lam, loss, delta, tau)
        assert np.abs(a1 - a2).max() <= 1e-9 * max(1.0, np.abs(a2).max())
        assert abs(b1 - b2) <= 1e-9 * max(1.0, abs(b2))


def test_block_inverse_constants_reading():
    # H^{-1} = g (1; -v)(1; -v)' + blockdiag(0, U Pi^{-1} U') with the Schur
    # complement constants v = U D c/(n kappa), g = 1/(2 lambda c'D c/(n kappa)),
    # D = Lambda Pi^{-1}, c = U'1. The constants as printed (v = U D c,
    # g = 1/(n c' Lambda Pi^{-1} Lambda c)) do not invert H.
    K, _, _ = _wellcond_problem("hinge", seed=3, n=25)
    n = K.shape[0]
    mu, U = np.linalg.eigh(K)
    c = U.T @ np.ones(n)
    for lam, kap in [(1e-2, 0.25), (0.5, 4.0)]:
        H = mm.majoriser_hessian(K, lam, kap)
        Pi = 2 * lam * mu + mu * mu / (n * kap)
        D = mu / Pi
        core = np.zeros((n + 1, n + 1))
        core[1:, 1:] = U @ np.diag(1.0 / Pi) @ U.T
        v = U @ (D * c) / (n * kap)
        g = 1.0 / (2 * lam * (c @ (D * c)) / (n * kap))
        e = np.concatenate([[1.0], -v])
        Hinv = g * np.outer(e, e) + core
        assert np.abs(H @ Hinv - np.eye(n + 1)).max() < 1e-9
        v_p = U @ (D * c)
        g_p = 1.0 / (n * (c @ (mu * D * c)))
        e_p = np.concatenate([[1.0], -v_p])
        Hinv_p = g_p * np.outer(e_p, e_p) + core
        assert np.abs(H @ Hinv_p - np.eye(n + 1)).max() > 0.1


@pytest.mark.parametrize("loss,delta,tau", CASES)
def test_mm_step_decreases_objective(loss, delta, tau):
    inp = W.make_inputs(W.get("C1")) if loss != "check" else W.small_problem("check", 150, 4, seed=2)
    X, y = inp["X"], inp["y"]
    K = gram.rbf_gram(X, X, inp["sigmas"][0])
    rng = np.random.default_rng(7)
    for lam in [1e-4, 1e-2, 1.0]:
        a = rng.standard_normal(len(y)) * 0.05
        b = 0.1
        F0 = cell.objective(K, y, a, b, lam, loss, delta, tau)
        for _ in range(5):
            a, b = mm.mm_step(K, y, a, b, lam, loss, delta, tau)
            F1 = cell.objective(K, y, a, b, lam, loss, delta, tau)
            assert F1 <= F0 + 1e-14 * abs(F0)
            F0 = F1


@pytest.mark.parametrize("loss,delta,tau", CASES)
def test_solution_is_fixed_point_of_mm_step(loss, delta, tau):
    inp = W.small_problem(loss, 70, 3, seed=6)
    X, y = inp["X"], inp["y"]
    K = gram.rbf_gram(X, X, inp["sigmas"][0])
    for lam in [1e-3, 0.1]:
        a, b, info = cell.solve_cell(K, y, lam, loss, delta, tau)
        a1, b1 = mm.mm_step(K, y, a, b, lam, loss, delta, tau)
        assert np.abs(a1 - a).max() <= 1e-9 * max(1.0, np.abs(a).max())
        assert abs(b1 - b) <= 1e-9


def test_accelerated_iteration_with_r_one_is_plain_step():
    K, y, rng = _wellcond_problem("logistic", seed=4)
    a, ap = rng.standard_normal(len(y)), rng.standard_normal(len(y))
    out = mm.accelerated_iteration(K, y, a, 0.2, ap, -0.1, 1.0, 0.01, "logistic")
    a1, b1 = mm.mm_step(K, y, a, 0.2, 0.01, "logistic")
    assert np.array_equal(out[0], a1) and out[1] == b1 and out[4] == pytest.approx(0.5 * (1 + np.sqrt(5.0)))
    # r = 2: extrapolation coefficient (r-1)/r' with r' = (1 + sqrt(17))/2
    out = mm.accelerated_iteration(K, y, a, 0.2, ap, -0.1, 2.0, 0.01, "logistic")
    c = 1.0 / (0.5 * (1 + np.sqrt(17.0)))
    assert np.allclose(out[5], a + c * (a - ap)) and out[6] == pytest.approx(0.2 + c * 0.3)
