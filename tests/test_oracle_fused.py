"""Pins of the oracle's fused transition sweeps (restore of probe k with +eps of probe k+1;
last restore with the update)."""

import numpy as np
import pytest
import torch

import oracle
import workloads


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_perturb2_with_zero_second_scale_is_perturb(dtype):
    th = workloads.normal_f32(3000, 1) if dtype == "f32" else workloads.normal_bf16_bits(3000, 1)
    a = oracle.perturb2(th, dtype, 7, 3, 2, 5, 1e-3, 9, 0.0)
    b = oracle.perturb(th, dtype, 7, 3, 2, 5, 1e-3)
    np.testing.assert_array_equal(a, b)


def test_perturb2_same_probe_doubles_and_cancels():
    th = workloads.normal_f32(3000, 2)
    np.testing.assert_array_equal(oracle.perturb2(th, "f32", 0, 1, 1, 4, 1e-3, 4, 1e-3),
                                  oracle.perturb(th, "f32", 0, 1, 1, 4, 2e-3))
    np.testing.assert_array_equal(oracle.perturb2(th, "f32", 0, 1, 1, 4, 1e-3, 4, -1e-3), th)


def test_perturb2_matches_torch_arithmetic():
    """d = e_a z_a + e_b z_b in fp32 (torch), one fp32 add, torch's bf16 cast."""
    n = 4000
    za = torch.from_numpy(oracle.signs(11, n, 5, 6, 3).astype(np.float32))
    zb = torch.from_numpy(oracle.signs(11, n, 5, 6, 12).astype(np.float32))
    ea, eb = np.float32(1e-3), np.float32(-3.7e-4)
    d = torch.tensor(ea) * za + torch.tensor(eb) * zb
    th = workloads.normal_f32(n, 3)
    np.testing.assert_array_equal(oracle.perturb2(th, "f32", 11, 5, 6, 3, ea, 12, eb), (torch.from_numpy(th) + d).numpy())
    tb = workloads.normal_bf16_bits(n, 3)
    tt = torch.from_numpy(tb.view(np.int16)).view(torch.bfloat16).float()
    want = (tt + d).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle.perturb2(tb, "bf16", 11, 5, 6, 3, ea, 12, eb), want)


def test_perturb2_close_to_sequential():
    """One rounding instead of two: within one ulp of the largest magnitude involved."""
    th = workloads.normal_f32(1 << 15, 4)
    seq = oracle.perturb(oracle.perturb(th, "f32", 0, 2, 2, 6, 1e-3), "f32", 0, 2, 2, 7, 1e-3)
    fus = oracle.perturb2(th, "f32", 0, 2, 2, 6, 1e-3, 7, 1e-3)
    M = np.abs(th) + 2e-3
    assert np.all(np.abs(seq.astype(np.float64) - fus) <= np.spacing(M.astype(np.float32)))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_update_restore_zero_restore_is_update(dtype):
    th = workloads.normal_f32(2000, 5) if dtype == "f32" else workloads.normal_bf16_bits(2000, 5)
    c = np.random.default_rng(0).standard_normal(12).astype(np.float32)
    np.testing.assert_array_equal(oracle.update_restore(th, dtype, 3, 4, 5, c, 1e-3, 11, 0.0),
                                  oracle.update(th, dtype, 3, 4, 5, c, 1e-3))


def test_update_restore_equals_materialised():
    """theta + e_r z_r - lr Z c with Z materialised (dyadic values: every sum exact)."""
    rng = np.random.default_rng(6)
    n, K = 500, 9
    c = (rng.integers(-512, 512, K) / 1024.0).astype(np.float32)
    lr, er = np.float32(2.0 ** -9), np.float32(2.0 ** -10)
    Z = oracle.materialize_Z(40, n, K, 8, 1).astype(np.float64)
    zr = oracle.signs(40, n, 8, 1, K - 1).astype(np.float64)
    th = workloads.normal_f32(n, 6)
    want = ((th.astype(np.float64) + np.float64(er) * zr) - np.float64(lr) * (Z @ c.astype(np.float64))).astype(np.float32)
    np.testing.assert_array_equal(oracle.update_restore(th, "f32", 40, 8, 1, c, lr, K - 1, er), want)


def test_fused_step_sees_the_same_perturbed_weights_and_lands_close():
    """The fused schedule presents each forward pass theta +- eps z_k (within rounding) and
    ends within rounding of the sequential schedule."""
    th = workloads.tiny_theta(1 << 14)
    K, eps, lr = 6, 1e-3, 1e-4
    lp, lm, l0 = workloads.synthetic_losses(K, 1)
    fused, co, seen = oracle.full_step_fused(th, "f32", 0, 0, 0, eps, lr, lp, lm, l0)
    seq, co2 = oracle.full_step(th, "f32", 0, 0, 0, eps, lr, lp, lm, l0)
    np.testing.assert_array_equal(co["c"], co2["c"])
    bound = 8 * np.spacing((np.abs(th) + 3 * eps).astype(np.float32)).astype(np.float64)
    for k, (tp, tm) in enumerate(seen):
        z = oracle.signs(0, th.size, 0, 0, k).astype(np.float64)
        assert np.all(np.abs(tp - (th + eps * z)) <= bound)
        assert np.all(np.abs(tm - (th - eps * z)) <= bound)
    assert np.all(np.abs(fused.astype(np.float64) - seq) <= bound)
