"""Oracle losses against their closed forms, conjugate representations and limits."""
import numpy as np
import pytest

from oracle import losses as Ls

DELTAS = [1.0, 0.125, 2.0 ** -6]


@pytest.mark.parametrize("delta", DELTAS)
def test_smoothed_hinge_closed_form_points(delta):
    assert Ls.smoothed_hinge(1.0 - delta, delta) == pytest.approx(delta)
    assert Ls.smoothed_hinge(1.0, delta) == pytest.approx(delta / 4.0)
    assert Ls.smoothed_hinge(1.0 + delta, delta) == 0.0
    assert Ls.smoothed_hinge(-3.0, delta) == 4.0
    assert Ls.smoothed_hinge(5.0, delta) == 0.0


@pytest.mark.parametrize("delta", DELTAS)
def test_smoothed_hinge_bounds_and_continuity(delta):
    u = np.linspace(-3, 3, 20001)
    L = Ls.smoothed_hinge(u, delta)
    h = Ls.hinge(u)
    assert np.all(L - h >= -1e-15) and np.all(L - h <= delta / 4 + 1e-15)
    for b in (1 - delta, 1 + delta):
        eps = 1e-9
        assert Ls.smoothed_hinge(b - eps, delta) == pytest.approx(Ls.smoothed_hinge(b + eps, delta), abs=1e-8)
        assert Ls.smoothed_hinge_d1(b - eps, delta) == pytest.approx(Ls.smoothed_hinge_d1(b + eps, delta), abs=1e-6)


@pytest.mark.parametrize("delta", DELTAS)
def test_smoothed_hinge_is_box_conjugate(delta):
    # L_delta(u) = max_{a in [0,1]} a (1 - u + delta) - delta a^2 (dual representation)
    a = np.linspace(0, 1, 200001)
    for u in [-2.0, 0.0, 1 - delta, 1 - 0.3 * delta, 1.0, 1 + 0.5 * delta, 1 + delta, 3.0]:
        val = np.max(a * (1 - u + delta) - delta * a * a)
        assert Ls.smoothed_hinge(u, delta) == pytest.approx(val, abs=1e-9)


def _fd(fun, x, h=1e-6):
    return (fun(x + h) - fun(x - h)) / (2 * h)


@pytest.mark.parametrize("loss,tau", [("hinge", None), ("logistic", None), ("check", 0.2), ("check", 0.9)])
def test_psi_and_curv_are_derivatives(loss, tau):
    delta = 0.125
    rng = np.random.default_rng(3)
    for _ in range(200):
        y = rng.choice([-1.0, 1.0]) if loss != "check" else rng.normal()
        f = rng.normal() * 2
        lo = lambda t: float(Ls.point_loss(loss, y, t, delta, tau))
        ps = lambda t: float(Ls.point_psi(loss, y, t, delta, tau))
        assert ps(f) == pytest.approx(_fd(lo, f), abs=1e-6)
        assert float(Ls.point_curv(loss, y, f, delta, tau)) == pytest.approx(_fd(ps, f), abs=1e-4)


@pytest.mark.parametrize("delta", DELTAS)
def test_check_loss_reduces_to_smoothed_hinge(delta):
    # rho_{1,delta}(1 - u) == L_delta(u) for every u
    u = np.linspace(-3, 3, 4001)
    assert np.max(np.abs(Ls.smoothed_check(1.0 - u, 1.0, delta) - Ls.smoothed_hinge(u, delta))) <= 1e-14


@pytest.mark.parametrize("tau", [0.1, 0.5, 0.9])
@pytest.mark.parametrize("delta", DELTAS)
def test_check_loss_conjugate_and_bounds(tau, delta):
    a = np.linspace(tau - 1, tau, 200001)
    for r in [-2.0, -delta, -0.4 * delta, 0.0, 0.7 * delta, delta, 1.5]:
        val = np.max(a * r + delta * (a - tau + 1) * (tau - a))
        assert Ls.smoothed_check(r, tau, delta) == pytest.approx(val, abs=1e-9)
    r = np.linspace(-3, 3, 20001)
    gap = Ls.smoothed_check(r, tau, delta) - Ls.check(r, tau)
    assert np.all(gap >= -1e-15) and np.all(gap <= delta / 4 + 1e-15)


def test_logistic_conjugate_entropy():
    a = np.linspace(1e-12, 1 - 1e-12, 400001)
    H = -a * np.log(a) - (1 - a) * np.log1p(-a)
    for u in [-5.0, -1.0, 0.0, 0.3, 2.0, 6.0]:
        assert float(Ls.logistic(u)) == pytest.approx(np.max(-a * u + H), abs=1e-9)


def test_logistic_curvature_bound_and_stability():
    u = np.linspace(-800, 800, 10001)
    c = Ls.point_curv("logistic", 1.0, u)
    assert np.all(c <= 0.25) and c.max() == pytest.approx(0.25)
    assert np.all(np.isfinite(Ls.logistic(u)))
    assert float(Ls.logistic(0.0)) == pytest.approx(np.log(2.0))


def test_kappa():
    assert Ls.kappa("logistic", None) == 4.0
    assert Ls.kappa("hinge", 0.125) == 0.25
    assert Ls.kappa("check", 2.0 ** -6) == 2.0 ** -5


def test_eval_losses():
    assert float(Ls.eval_loss("hinge", 1.0, 0.25)) == 0.75
    assert float(Ls.eval_loss("hinge", -1.0, -2.0)) == 0.0
    assert float(Ls.eval_loss("check", 1.0, 0.0, 0.3)) == pytest.approx(0.3)
    assert float(Ls.eval_loss("check", 0.0, 1.0, 0.3)) == pytest.approx(0.7)
