"""End-to-end behaviour of the method on the stiff paraboloid (section 5.3, appendix A.2),
through the CPU oracle.

The paper reports that 1.5-SPSA matches 1SPSA on a well-conditioned paraboloid and converges
faster as the condition number grows (up to 7x on average). Dimension, probe count, eps,
step sizes and the tolerance are not stated, so this is a qualitative check ("parity
unpinned" quantitatively): d = 16, K = 16, eps = 1e-2, each solver's step size tuned on a
grid around its best value (the grids hold the best values of a wider sweep on seed 0),
convergence when J falls below 1e-6 of its start, three seeds. 1.5-SPSA is run with alpha = 1
(the probe-space Newton weighting of section 4.1) and with the paper's default alpha = 0.1;
1SPSA is alpha = 0. With fp32 weights and eps = 1e-3 the rounding of theta +- eps z puts noise
of order 20% into the curvature estimate near x ~ 1, which alpha = 1 amplifies; eps = 1e-2
keeps it below 1%.

Running this file as a script prints the table of mean step counts and ratios.
"""

import os
import sys

import numpy as np
import pytest

if __name__ == "__main__":  # run as a script: the repository root holds oracle/ and workloads/
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle
import workloads
from paraboloid import best_steps, trend

D, K, EPS, TOL, MAX_STEPS = 16, 16, 1e-2, 1e-6, 6000
KAPPAS = (1, 10, 100, 1000)
ALPHAS = (0.0, 0.1, 1.0)
SEEDS = (0, 1, 2)
# (kappa, alpha) -> step sizes tried
LRS = {
    (1, 0.0): (0.2, 0.3, 0.42), (10, 0.0): (0.07, 0.1, 0.14), (100, 0.0): (0.007, 0.01, 0.014),
    (1000, 0.0): (0.001, 0.0014),
    (1, 0.1): (0.2, 0.3, 0.42), (10, 0.1): (0.07, 0.1, 0.14), (100, 0.1): (0.007, 0.01, 0.014),
    (1000, 0.1): (0.0014, 0.002, 0.0028),
    (1, 1.0): (7.0, 10.0, 14.0), (10, 1.0): (4.0, 6.0, 8.0), (100, 1.0): (2.0, 3.0, 4.0),
    (1000, 1.0): (1.4, 2.0, 2.8),
}


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


def _job(key):
    return _steps(*key)


def trend_table(procs=None):
    """{(kappa, alpha, seed): steps} over KAPPAS x ALPHAS x SEEDS, and the mean 1SPSA :
    1.5-SPSA step ratio per (kappa, alpha) over the seeds."""
    procs = procs or min(8, os.cpu_count() or 1)
    steps = trend(_job, KAPPAS, ALPHAS, SEEDS, procs)
    ratios = {}
    for kappa in KAPPAS:
        for alpha in ALPHAS[1:]:
            ratios[(kappa, alpha)] = float(np.mean([steps[(kappa, 0.0, s)] / steps[(kappa, alpha, s)] for s in SEEDS]))
    return steps, ratios


@pytest.fixture(scope="module")
def table():
    return trend_table()


def test_every_run_converges(table):
    steps, _ = table
    for key, n in steps.items():
        assert n is not None and n < MAX_STEPS, key


def test_well_conditioned_matches(table):
    _, ratios = table
    assert 0.5 <= ratios[(1, 1.0)] <= 2.0
    assert 0.5 <= ratios[(1, 0.1)] <= 2.0


def test_advantage_grows_with_condition_number(table):
    """The mean 1SPSA : 1.5-SPSA (alpha = 1) step ratio does not fall as kappa grows and is
    several-fold at kappa = 1000 (the paper: up to 7x on average)."""
    _, ratios = table
    r = [ratios[(k, 1.0)] for k in KAPPAS]
    assert all(b >= a for a, b in zip(r, r[1:])), r
    assert r[-1] >= 4.0, r
    assert ratios[(100, 1.0)] >= 2.0, r


def test_default_alpha_never_loses_much(table):
    """alpha = 0.1 (the paper's default) saturates the curvature weight: it tracks 1SPSA on
    these quadratics, never more than 2x slower."""
    _, ratios = table
    for k in KAPPAS:
        assert ratios[(k, 0.1)] >= 0.5, (k, ratios[(k, 0.1)])


if __name__ == "__main__":
    steps, ratios = trend_table()
    print("kappa  alpha  steps per seed            mean   1SPSA:1.5-SPSA")
    for k in KAPPAS:
        for a in ALPHAS:
            ss = [steps[(k, a, s)] for s in SEEDS]
            r = "" if a == 0.0 else f"{ratios[(k, a)]:.2f}"
            print(f"{k:5d}  {a:5.1f}  {str(ss):24s}  {np.mean(ss):7.1f}  {r}")
