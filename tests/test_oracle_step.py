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
    # the restores leave the weights within 1 ulp of the largest intermediate
    assert np.max(np.abs(t.astype(np.float64) - th)) < 1e-9
