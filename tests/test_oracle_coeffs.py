"""Pins of the coefficient function: exact quadratic curvature, the paper's special cases."""

import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

EPS = 2.0 ** -10


def _quad_loss_exact(H, x):
    """0.5 x^T H x for integer H and dyadic x, computed exactly, returned as float."""
    xs = [Fraction(float(v)) for v in x]
    n = len(xs)
    s = Fraction(0)
    for i in range(n):
        if xs[i] == 0:
            continue
        row = sum(int(H[i, j]) * xs[j] for j in range(n) if H[i, j] != 0)
        s += xs[i] * row
    v = s / 2
    f = float(v)
    assert Fraction(f) == v  # exactly representable
    return f


def _quadratic_setup(n, K, seed, diagonal):
    rng = np.random.default_rng(seed)
    if diagonal:
        H = np.diag(rng.integers(1, 5, n))
    else:
        A = rng.integers(-2, 3, (n, n))
        H = A + A.T
    theta = rng.integers(-255, 256, n) / 256.0
    Z = oracle.materialize_Z(0, n, K, seed, 0).astype(np.float64)
    L0 = _quad_loss_exact(H, theta)
    Lp = [_quad_loss_exact(H, theta + EPS * Z[:, k]) for k in range(K)]
    Lm = [_quad_loss_exact(H, theta - EPS * Z[:, k]) for k in range(K)]
    return H, theta, Z, L0, Lp, Lm


@pytest.mark.parametrize("diagonal", [True, False])
def test_quadratic_curvature_is_exact(diagonal):
    """Eq. 3 on L = 0.5 theta^T H theta gives z^T H z exactly (zero finite-difference bias),
    which for a diagonal H and Rademacher z is tr(H); and L+ - L- = 2 eps z^T H theta."""
    n, K = 24, 10
    H, theta, Z, L0, Lp, Lm = _quadratic_setup(n, K, 7 + diagonal, diagonal)
    co = oracle.probe_coeffs(Lp, Lm, L0, EPS)
    for k in range(K):
        z = Z[:, k]
        assert co["curv"][k] == float(z @ H @ z)
        if diagonal:
            assert co["curv"][k] == float(np.trace(H))
        assert Lp[k] - Lm[k] == 2 * EPS * float(z @ (H @ theta))


def test_alpha_zero_is_1spsa():
    """alpha = 0 gives w = 1 for any curvature: c_k = (L+ - L-) / (2 K eps)."""
    Lp = [2.0, 5.0, 1e6, -3.0]
    Lm = [1.0, -5.0, 2.0, -3.5]
    co = oracle.probe_coeffs(Lp, Lm, 0.25, 1e-3, alpha=0.0)
    assert np.all(co["w"] == 1.0)
    for k in range(4):
        assert co["c64"][k] == (Lp[k] - Lm[k]) / (2 * 4 * 1e-3)


def test_worked_value_curvature_1e8():
    """Section 6's worked value (tests/golden/curvature_weight_worked_value.txt): a
    three-point curvature of 1e8 with alpha = 0.1 is down-weighted by the printed factor."""
    golden = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "curvature_weight_worked_value.txt")
    row = [ln.split() for ln in open(golden) if ln.strip() and not ln.startswith("#")][0]
    curv, alpha, factor, tol = (float(x) for x in row)
    eps = 1e-3
    # L+ - 2 L0 + L- = curv * eps^2 = 100 with L0 = 1
    co = oracle.probe_coeffs([52.0], [50.0], 1.0, eps, alpha=alpha)
    assert abs(co["curv"][0] - curv) < 1e-3
    assert abs(1.0 / co["w"][0] - factor) < tol


def test_saturation_below_lambda():
    """|chat|^alpha <= lambda_reg = 1 leaves the weight at exactly 1."""
    co = oracle.probe_coeffs([1.0 + 1e-7, 1.0, 1.0 + 5e-7], [1.0 - 1e-7, 1.0, 1.0 - 4e-7], 1.0, 1e-3)
    assert np.all(np.abs(co["curv"]) <= 1.0)
    assert np.all(co["w"] == 1.0)


def test_alpha_one_is_probe_space_newton_step():
    """alpha = 1 and |chat| >= 1: one probe with lr = 1 lands on the minimiser along z."""
    n = 16
    H, theta, Z, L0, Lp, Lm = _quadratic_setup(n, 1, 3, True)
    co = oracle.probe_coeffs(Lp, Lm, L0, EPS, alpha=1.0)
    z = Z[:, 0]
    assert co["w"][0] == 1.0 / float(z @ H @ z)
    new = theta - co["c64"][0] * z
    g_along = float(z @ (H @ new))
    assert abs(g_along) <= 1e-12 * float(np.abs(z @ (H @ theta)) + 1)


def test_eq6_compact_form_with_tied_step():
    """With lr = eps, lr * c_k = eta w_k Delta l_k with eta = 1/(2n) (Eq. 6, Algorithm 1's gamma)."""
    rng = np.random.default_rng(5)
    K = 40
    Lp, Lm = rng.normal(2, 0.05, K), rng.normal(2, 0.05, K)
    L0, eps = 1.97, 1e-4
    co = oracle.probe_coeffs(Lp, Lm, L0, eps)
    gamma = (1.0 / (2 * K)) * (Lp - Lm) * co["w"]
    np.testing.assert_allclose(eps * co["c64"], gamma, rtol=4e-16, atol=0)


def test_update_descends_on_quadratic():
    """Descent sign (Eq. 6 and Algorithm 1 subtract): a step with many probes lowers the loss."""
    n, K = 12, 64
    H, theta, Z, L0, Lp, Lm = _quadratic_setup(n, K, 11, True)
    co = oracle.probe_coeffs(Lp, Lm, L0, EPS)
    new = oracle.update(theta.astype(np.float32), "f32", 0, 11, 0, co["c"], 0.05)
    f = lambda x: 0.5 * float(x @ H @ x)
    assert f(new.astype(np.float64)) < f(theta)


@pytest.mark.parametrize("bad", [
    dict(L_plus=[], L_minus=[]),
    dict(L_plus=[1.0, 2.0], L_minus=[1.0]),
    dict(L_plus=[float("nan")], L_minus=[1.0]),
    dict(L_plus=[1.0], L_minus=[float("inf")]),
    dict(L_clean=float("nan")),
    dict(eps=0.0), dict(eps=-1e-3), dict(eps=float("inf")),
    dict(alpha=-0.1), dict(alpha=1.5), dict(lambda_reg=0.0),
])
def test_invalid_inputs_raise(bad):
    args = dict(L_plus=[1.0], L_minus=[0.9], L_clean=1.0, eps=1e-3, alpha=0.1, lambda_reg=1.0)
    args.update(bad)
    with pytest.raises(ValueError):
        oracle.probe_coeffs(**args)


def test_vanishing_eps_square_is_ieee():
    """eps*eps underflowing to 0 follows IEEE (infinite curvature, zero weight), no exception."""
    co = oracle.probe_coeffs([2.0], [1.0], 1.0, 1e-170)
    assert np.isinf(co["curv"][0]) and co["w"][0] == 0.0 and co["c"][0] == 0.0
