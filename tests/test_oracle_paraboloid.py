"""End-to-end behaviour of the method on the stiff paraboloid (section 5.3, appendix A.2),
through the CPU oracle.

The paper reports that 1.5-SPSA matches 1SPSA on a well-conditioned paraboloid and converges
faster as the condition number grows (up to 7x on average). Dimension, probe count, eps,
step sizes and the tolerance are not stated, so this is a qualitative check ("parity
unpinned" quantitatively): d = 16, K = 16, eps = 1e-2, each solver's step size tuned on a
small grid (the grids hold the best values of a wider sweep), convergence when J falls below
1e-6 of its start. 1.5-SPSA uses alpha = 1 (the probe-space Newton weighting of section
4.1); 1SPSA is alpha = 0. With fp32 weights and eps = 1e-3 the rounding of theta +- eps z
puts noise of order 20% into the curvature estimate near x ~ 1, which alpha = 1 amplifies;
eps = 1e-2 keeps it below 1%.
"""

import numpy as np
import pytest

import oracle
import workloads
from paraboloid import best_steps

D, K, EPS, TOL, MAX_STEPS = 16, 16, 1e-2, 1e-6, 1500
# (kappa, alpha) -> step sizes tried
LRS = {(1, 0.0): (0.1, 0.3), (1, 1.0): (3.0, 10.0), (100, 0.0): (0.01, 0.02), (100, 1.0): (1.0, 3.0)}


class OracleBackend:
    def __init__(self, A, seed):
        self.A, self.seed = A, seed

    def loss(self, x):
        v = x.astype(np.float64)
        return float(v @ self.A @ v)

    def perturb(self, x, k, e, step):
        return oracle.perturb(x, "f32", 0, self.seed, step, k, e)

    def coeffs(self, lp, lm, l0, eps, alpha):
        return oracle.probe_coeffs(lp, lm, l0, eps, alpha, 1.0)["c"]

    def update(self, x, c, lr, step):
        return oracle.update(x, "f32", 0, self.seed, step, c, lr)


def _steps(kappa, alpha, seed):
    def make():
        A, x0 = workloads.stiff_paraboloid(D, kappa, seed)
        return OracleBackend(A, seed), x0
    return best_steps(make, LRS[(kappa, alpha)], K, EPS, alpha, MAX_STEPS, TOL)


@pytest.mark.parametrize("seed", [0])
def test_well_conditioned_matches(seed):
    s0, s1 = _steps(1, 0.0, seed), _steps(1, 1.0, seed)
    assert s0 is not None and s1 is not None and s0 < 100 and s1 < 100
    assert 0.5 <= s0 / s1 <= 2.0


@pytest.mark.parametrize("seed", [0])
def test_ill_conditioned_is_faster(seed):
    s0, s1 = _steps(100, 0.0, seed), _steps(100, 1.0, seed)
    assert s0 is not None and s1 is not None
    assert s0 / s1 >= 2.0, (s0, s1)
