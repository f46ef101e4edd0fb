"""One 1.5-SPSA step on one device, composed from the oracle's sweeps.

TEST INFRASTRUCTURE: part of the CPU oracle.

Algorithm 1 on a single rank: for each probe k apply +eps, -2 eps, +eps around the two
perturbed forward passes, then form the coefficients from the gathered losses and apply
the update. The forward passes are outside the sweep: the losses are inputs here.
"""

from .coeffs import DEFAULT_ALPHA, DEFAULT_LAMBDA_REG, probe_coeffs
from .probes import DEFAULT_ROUNDS
from .sweep import perturb, update


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
