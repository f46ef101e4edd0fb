"""One 1.5-SPSA step on one device, composed from the oracle's sweeps.

TEST INFRASTRUCTURE: part of the CPU oracle.

Algorithm 1 on a single rank: for each probe k apply +eps, -2 eps, +eps around the two
perturbed forward passes, then form the coefficients from the gathered losses and apply
the update. The forward passes are outside the sweep: the losses are inputs here.
"""

from .coeffs import DEFAULT_ALPHA, DEFAULT_LAMBDA_REG, probe_coeffs
from .probes import DEFAULT_ROUNDS
from .sweep import perturb, perturb2, update, update_restore


def full_step(theta, dtype, offset, seed, step, eps, lr, L_plus, L_minus, L_clean,
              alpha=DEFAULT_ALPHA, lambda_reg=DEFAULT_LAMBDA_REG, rounds=DEFAULT_ROUNDS):
    """Return (theta after the step, coefficient dict)."""
    K = len(L_plus)
    t = theta
    for k in range(K):
        t = perturb(t, dtype, offset, seed, step, k, eps, rounds)
        t = perturb(t, dtype, offset, seed, step, k, -2.0 * float(eps), rounds)
        t = perturb(t, dtype, offset, seed, step, k, eps, rounds)
    co = probe_coeffs(L_plus, L_minus, L_clean, eps, alpha, lambda_reg)
    return update(t, dtype, offset, seed, step, co["c"], lr, rounds), co


def full_step_fused(theta, dtype, offset, seed, step, eps, lr, L_plus, L_minus, L_clean,
                    alpha=DEFAULT_ALPHA, lambda_reg=DEFAULT_LAMBDA_REG, rounds=DEFAULT_ROUNDS):
    """The same step in 2K + 1 sweeps: +eps z_0; then per probe -2 eps z_k followed by the
    restore of z_k merged with +eps z_{k+1}, the last restore merged with the update.
    Returns (theta after the step, coefficient dict, list of the weights each perturbed
    forward pass would see as (theta_plus, theta_minus) pairs)."""
    K = len(L_plus)
    e = float(eps)
    seen = []
    t = perturb(theta, dtype, offset, seed, step, 0, e, rounds)
    for k in range(K):
        tp = t
        t = perturb(t, dtype, offset, seed, step, k, -2.0 * e, rounds)
        seen.append((tp, t))
        if k + 1 < K:
            t = perturb2(t, dtype, offset, seed, step, k, e, k + 1, e, rounds)
    co = probe_coeffs(L_plus, L_minus, L_clean, eps, alpha, lambda_reg)
    return update_restore(t, dtype, offset, seed, step, co["c"], lr, K - 1, e, rounds), co, seen
