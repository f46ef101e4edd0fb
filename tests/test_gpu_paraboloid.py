"""The stiff paraboloid (section 5.3, appendix A.2) end to end through libzo on the GPU:
perturb schedule, host coefficients and fused update in the library, the quadratic loss
evaluated by torch on the device. Same settings, seeds and bars as the oracle version at
kappa = 1 and 100 (alpha = 0 against alpha = 1), plus agreement of the step counts with the
oracle's on every seed."""

import numpy as np
import pytest
import torch

import paper_2609_38095_amd as zo
import workloads
from paraboloid import best_steps
from test_oracle_paraboloid import D, EPS, K, LRS, MAX_STEPS, SEEDS, TOL, OracleBackend

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


class GpuBackend:
    def __init__(self, A, seed):
        self.A = torch.from_numpy(A).to(DEV)
        self.seed = seed

    def loss(self, x):
        v = x.double()
        return float(v @ (self.A @ v))

    def perturb(self, x, k, e, step):
        zo.zo_perturb(x, k, e, self.seed, step)
        return x

    def coeffs(self, lp, lm, l0, eps, alpha):
        return zo.zo_probe_coeffs_ex(lp, lm, l0, eps, alpha, 1.0)["c"]

    def update(self, x, c, lr, step):
        zo.zo_update(x, c, lr, self.seed, step)
        return x


def _steps(kappa, alpha, seed, gpu):
    def make():
        A, x0 = workloads.stiff_paraboloid(D, kappa, seed)
        if gpu:
            return GpuBackend(A, seed), torch.from_numpy(x0).to(DEV)
        return OracleBackend(A, seed), x0
    return best_steps(make, LRS[(kappa, alpha)], K, EPS, alpha, MAX_STEPS, TOL)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    zo.library()


@pytest.mark.parametrize("kappa,min_ratio,max_ratio", [(1, 0.5, 2.0), (100, 2.0, 1e9)])
def test_paraboloid_through_library(kappa, min_ratio, max_ratio):
    ratios = []
    for seed in SEEDS:
        print(f"paraboloid kappa {kappa} seed {seed}", flush=True)
        s0, s1 = _steps(kappa, 0.0, seed, True), _steps(kappa, 1.0, seed, True)
        assert s0 is not None and s1 is not None
        ratios.append(s0 / s1)
        o0, o1 = _steps(kappa, 0.0, seed, False), _steps(kappa, 1.0, seed, False)
        for g, o in ((s0, o0), (s1, o1)):
            assert abs(g - o) <= max(3, 0.1 * o), (seed, g, o)
    assert min_ratio <= float(np.mean(ratios)) <= max_ratio, ratios
