"""CPU oracle for the cross-validated kernel-machine path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute anything in this package; only the tests, the smoke check and the
CPU-baseline leg of the benchmark use it. It shares no code with the GPU
library (the only common dependency is the seeded input generator module
``workloads``, which holds none of the method's arithmetic).

It is deliberately plain: numpy/scipy in fp64, every cell of the path solved
on its own from a cold start to machine precision by semismooth Newton
(not by the paper's spectral iteration), with dual certificates.

Parity status per function (what pins it; see tests/test_oracle_*.py):
* losses.*          closed forms, continuity, finite differences, the tau=1
                    reduction of the smoothed check loss to L_delta
* gram.rbf_gram     sklearn.metrics.pairwise.rbf_kernel, symmetry, PSD
* cell.solve_cell   brute-force zone enumeration (hinge, check; n <= 8),
                    50-digit mpmath Newton (logistic), zero duality gap,
                    exact-CV Lemma 2, large-lambda closed forms; its
                    extended-precision refinement by the same pins at small
                    lambda, where the fp64 loop alone stalls
* cell.certify_cell zero gap and feasibility at brute-force solutions,
                    a positive gap at perturbed points
* gram.rbf_gram_expansion  agreement with rbf_gram to rounding
* mm.mm_step        explicit solve with the (n+1)-square majoriser, monotone
                    decrease of F, fixed point at the cell solution
* path.fit_path     composition of the above; selection rule by brute force
* dual.*            closed-form conjugates checked pointwise by grid search
* hinge.*           brute force over all L/E/R patterns (n <= 7), zero duality
                    gap against the hinge dual, sklearn's SVC
"""
from . import losses, gram, cell, mm, dual, path, hinge  # noqa: F401
from .path import fit_path, select, select_joint  # noqa: F401
from .cell import solve_cell, objective, kkt_residual, beta_interval, certify_cell  # noqa: F401
