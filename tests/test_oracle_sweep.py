"""Pins of the oracle's perturb and update sweeps."""

import numpy as np
import pytest
import torch

import oracle
import workloads


def _ulp32(x):
    x = np.abs(np.asarray(x, dtype=np.float32))
    return np.spacing(x).astype(np.float64)


def test_perturb_on_zero_weights_is_eps_z():
    n = 1000
    z = oracle.signs(3, n, 11, 2, 5).astype(np.float32)
    out = oracle.perturb(np.zeros(n, np.float32), "f32", 3, 11, 2, 5, 1e-3)
    np.testing.assert_array_equal(out, np.float32(1e-3) * z)
    outb = oracle.perturb(np.zeros(n, np.uint16), "bf16", 3, 11, 2, 5, 1e-3)
    e_b = oracle.bf16_to_f32(oracle.f32_to_bf16(np.float32(1e-3)))
    np.testing.assert_array_equal(oracle.bf16_to_f32(outb), e_b * z)


@pytest.mark.parametrize("eps", [1e-3, -2e-3, 1e-4, 7.5])
def test_perturb_matches_torch_arithmetic(eps):
    """One IEEE fp32 add (torch on CPU), and for bf16 torch's round-to-nearest-even cast."""
    n, off = 5000, 12345
    z = torch.from_numpy(oracle.signs(off, n, 1, 4, 9).astype(np.float32))
    th = workloads.normal_f32(n, 3)
    ref = (torch.from_numpy(th) + torch.tensor(np.float32(eps)) * z).numpy()
    np.testing.assert_array_equal(oracle.perturb(th, "f32", off, 1, 4, 9, eps), ref)
    tb = workloads.normal_bf16_bits(n, 4)
    tt = torch.from_numpy(tb.view(np.int16)).view(torch.bfloat16)
    refb = (tt.float() + torch.tensor(np.float32(eps)) * z).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle.perturb(tb, "bf16", off, 1, 4, 9, eps), refb)


def test_restore_roundtrip_fp32_bound():
    """(+eps, -2 eps, +eps) returns fp32 weights within the rounding bound.

    Each of the three additions errs by at most half an ulp of its result, so the restore
    errs by at most 1.5 ulp of the largest intermediate magnitude M; on the tiny workload
    (theta ~ N(0, 0.02), eps = 1e-3) the observed worst case is within 1 ulp of M.
    """
    th = workloads.tiny_theta()
    tp, tm, tr = oracle.perturb_schedule(th, "f32", 0, 0, 0, 1, 1e-3)
    M = np.maximum.reduce([np.abs(th), np.abs(tp), np.abs(tm), np.abs(tr)])
    err = np.abs(tr.astype(np.float64) - th.astype(np.float64))
    assert np.all(err <= 1.5 * _ulp32(M))
    assert np.all(err <= 1.0 * _ulp32(M))
    # most elements restore exactly
    assert np.mean(tr == th) > 0.5


def _dyadic_c(K, rng):
    return (rng.integers(-512, 512, K) / 1024.0).astype(np.float32)


@pytest.mark.parametrize("K", [1, 3, 8, 9, 16, 21])
def test_update_equals_materialised_Z(K):
    """theta - lr * Z c with Z materialised and a library matmul (all sums exact with dyadic c)."""
    rng = np.random.default_rng(K)
    n, off = 777, 31
    c = _dyadic_c(K, rng)
    lr = np.float32(2.0 ** -9)
    Z = oracle.materialize_Z(off, n, K, 5, 6)
    th = workloads.normal_f32(n, K)
    ref = (th.astype(np.float64) - np.float64(lr) * (Z.astype(np.float64) @ c.astype(np.float64))).astype(np.float32)
    np.testing.assert_array_equal(oracle.update(th, "f32", off, 5, 6, c, lr), ref)
    tb = workloads.normal_bf16_bits(n, K)
    tbt = torch.from_numpy(tb.view(np.int16)).view(torch.bfloat16).double()
    refb64 = tbt.numpy() - np.float64(lr) * (Z.astype(np.float64) @ c.astype(np.float64))
    # torch's float64 -> bf16 cast is a single round-to-nearest-even
    refb = torch.from_numpy(refb64).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle.update(tb, "bf16", off, 5, 6, c, lr), refb)


def test_update_k1_equals_perturb():
    """With one probe the update is a perturbation by -lr*c0 (exact product here)."""
    th = workloads.normal_f32(2000, 9)
    c0, lr = np.float32(0.375), np.float32(2.0 ** -10)
    u = oracle.update(th, "f32", 17, 1, 2, [c0], lr)
    p = oracle.perturb(th, "f32", 17, 1, 2, 0, -lr * c0)
    np.testing.assert_array_equal(u, p)


def test_update_linearity_restores():
    th = workloads.normal_f32(4096, 1)
    c = np.random.default_rng(3).standard_normal(16).astype(np.float32)
    u = oracle.update(th, "f32", 0, 4, 5, c, 1e-4)
    back = oracle.update(u, "f32", 0, 4, 5, -c, 1e-4)
    assert np.all(np.abs(back.astype(np.float64) - th) <= 1.0 * _ulp32(np.maximum(np.abs(th), np.abs(u))))


def test_update_window_consistency():
    th = workloads.normal_f32(3000, 2)
    c = np.random.default_rng(0).standard_normal(12).astype(np.float32)
    full = oracle.update(th, "f32", 100, 8, 1, c, 1e-3)
    for a, b in [(0, 1), (5, 77), (1000, 3000), (2999, 3000)]:
        np.testing.assert_array_equal(oracle.update(th[a:b], "f32", 100 + a, 8, 1, c, 1e-3), full[a:b])


def test_update_chunks_by_k_base():
    """Splitting the probes with k_base gives the same probe sum."""
    c = np.random.default_rng(1).standard_normal(20).astype(np.float32)
    s_all = oracle.probe_sum(40, 500, 2, 3, c)
    s_a = oracle.probe_sum(40, 500, 2, 3, c[:8])
    s_b = oracle.probe_sum(40, 500, 2, 3, c[8:], k_base=8)
    np.testing.assert_allclose(s_a + s_b, s_all, rtol=0, atol=1e-12)
