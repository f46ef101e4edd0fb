"""The oracle's single-device step is Algorithm 1's schedule followed by one fused update."""

import numpy as np

import oracle
import workloads


def test_full_step_tiny_composition():
    w = workloads.WORKLOADS["tiny"]
    th = workloads.tiny_theta(1 << 14)
    K = 4
    lp, lm, l0 = workloads.synthetic_losses(K, 1)
    new, co = oracle.full_step(th, "f32", 0, 0, 0, w.eps, w.lr, lp, lm, l0)
    t = th
    for k in range(K):
        t = oracle.perturb_schedule(t, "f32", 0, 0, 0, k, w.eps)[2]
    np.testing.assert_array_equal(new, oracle.update(t, "f32", 0, 0, 0, co["c"], w.lr))
    # each restore errs by at most 1.5 ulp of magnitudes below |theta| + 2 eps
    bound = 1.5 * K * np.spacing((np.abs(th) + 2 * w.eps).astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(t.astype(np.float64) - th) <= bound)
