"""The single-step entry points against the oracle.

kmp_path_step: one majorise-minimise step of the path (Appendix A.1 update,
H applied through the block form of its inverse, Appendix A.3) from random
states, for all three losses, against the oracle's dense step
(``oracle.mm.mm_step``: an explicit solve with M = 2 lambda I + K/(n kappa),
pinned against a solve with the (n+1)-square majoriser H itself). This pins
the stage precompute (v, g), both path GEMMs, the loss derivative and the
update kernel at one step, not only at the fixed point they converge to.

kmp_dgemm_grouped: grouped fp64 products against numpy.
"""
import numpy as np
import pytest

from oracle import gram as OG
from oracle import losses as OL
from oracle.mm import mm_step
from tests.gpu_common import announce, device

pytestmark = pytest.mark.gpu

STEP_RTOL = 1e-9     # relative to the larger of the state's and the result's max |alpha|


@pytest.mark.parametrize("loss,tau", [("hinge", None), ("logistic", None), ("check", 0.3)])
def test_path_step_matches_dense_mm_step(loss, tau):
    import torch
    from paper_2606_06742_amd import kmpath as km
    dev = device()
    rng = np.random.default_rng({"hinge": 1, "logistic": 2, "check": 3}[loss])
    n, d = 150, 4
    X = rng.standard_normal((n, d))
    sigma = 2.0
    K = OG.rbf_gram(X, X, sigma)
    if loss == "check":
        y = np.sin(X[:, 0]) + 0.3 * rng.standard_normal(n)
    else:
        y = np.where(X[:, 0] + 0.5 * rng.standard_normal(n) > 0, 1.0, -1.0)
    lambdas = np.array([1e-3, 1e-2, 0.1, 1.0, 3e-3])
    C = lambdas.size
    delta = None if loss == "logistic" else 2.0 ** -4
    taus = np.full(C, tau) if loss == "check" else None
    # states around the scale of the solutions, 1/(2 n lambda)
    A = rng.uniform(-1, 1, (C, n)) / (2 * n * lambdas[:, None])
    B = rng.uniform(-0.5, 0.5, C)
    announce(f"kmp_path_step loss={loss} n={n} C={C}")
    t = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.float64, device=dev)
    a_out = torch.empty((C, n), dtype=torch.float64, device=dev)
    b_out = torch.empty(C, dtype=torch.float64, device=dev)
    k_out = torch.empty(C, dtype=torch.float64, device=dev)
    km.kmp_path_step(loss, delta, t(K), t(y), lambdas, t(A), t(B), a_out, b_out, k_out, taus=taus)
    torch.cuda.synchronize()
    ag, bg, kg = a_out.cpu().numpy(), b_out.cpu().numpy(), k_out.cpu().numpy()
    kap = OL.kappa(loss, delta)
    worst = 0.0
    for c in range(C):
        ao, bo = mm_step(K, y, A[c], B[c], lambdas[c], loss, delta, tau, kap=kap)
        scale = max(np.abs(ao).max(), np.abs(A[c]).max())
        err = np.abs(ag[c] - ao).max() / scale
        assert err <= STEP_RTOL, (c, err)
        assert abs(bg[c] - bo) <= STEP_RTOL * max(1.0, abs(bo), np.abs(A[c]).max()), (c, bg[c], bo)
        # the KKT measure at the given state: n max(||z + 2 lambda alpha||_2, |1'z|)
        z = OL.point_psi(loss, y, K @ A[c] + B[c], delta, tau) / n
        ko = n * max(np.linalg.norm(z + 2 * lambdas[c] * A[c]), abs(z.sum()))
        assert abs(kg[c] - ko) <= 1e-9 * ko, (c, kg[c], ko)
        worst = max(worst, err)
    print(loss, "worst step error", worst)


def test_dgemm_grouped_matches_numpy():
    import torch
    from paper_2606_06742_amd import kmpath as km
    dev = device()
    rng = np.random.default_rng(4)
    announce("kmp_dgemm_grouped G=3 M=100 N=70 K=130 and K=0")
    for (G, M, N, Kd) in [(3, 100, 70, 130), (2, 64, 64, 64), (1, 5, 1, 3), (2, 7, 9, 0)]:
        A = rng.standard_normal((G, M, Kd))
        B = rng.standard_normal((G, Kd, N))
        Ct = torch.full((G, M, N), np.nan, dtype=torch.float64, device=dev)
        km.kmp_dgemm_grouped(torch.as_tensor(A, device=dev), torch.as_tensor(B, device=dev), Ct)
        torch.cuda.synchronize()
        ref = A @ B
        got = Ct.cpu().numpy()
        bound = 4 * max(Kd, 1) * np.finfo(float).eps * (np.abs(A) @ np.abs(B) + 1e-300)
        assert np.all(np.abs(got - ref) <= bound), (G, M, N, Kd)
