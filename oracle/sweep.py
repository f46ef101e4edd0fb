"""The two parameter sweeps of 1.5-SPSA: in-place probe perturbation and the fused update.

TEST INFRASTRUCTURE: part of the CPU oracle.

perturb  -- Algorithm 1 applies each probe to the weights three times, with scales
            +eps, -2 eps and +eps around the two perturbed forward passes
            (ApplyPackedPerturbation). One call is theta <- theta + e * z_k.
update   -- section 4.2, Eq. 5 and its compact form Eq. 6, Delta theta = -eta Z W Delta l;
            Algorithm 1 applies it probe by probe. Here the step is
            theta <- theta - lr * sum_k c_k z_k with the coefficients c_k of coeffs.py.
            Reading: the sum is formed first and the weights are rounded to their storage
            type once (the paper's per-probe loop would round once per probe).

Arithmetic (readings; the paper does not fix it):
  * perturb: one IEEE float32 addition of theta (bf16 widened exactly) and e * z,
    which is exact since z = +-1; then bf16 storage rounds to nearest-even.
  * update: the sum over probes is accumulated in float64 from the float32 c_k, and
    theta - lr * sum is rounded once to the storage type.
Weights are float32 numpy arrays, or uint16 arrays of bf16 bit patterns.

Fused transitions (reading; the paper applies them as separate passes): on one device the
restore of probe k (+eps) and the +eps of probe k+1 are consecutive applications, and so are
the last restore and the update. perturb2 and update_restore apply such a pair in one pass:
  perturb2       -- d = fl32(e_a z_a + e_b z_b) (exact when |e_a| = |e_b|), theta + d in one
                    fp32 addition, then bf16 storage rounds to nearest-even;
  update_restore -- theta + e_r z_r - lr * sum_k c_k z_k formed in float64 and rounded once.
"""

import numpy as np

from .numerics import bf16_to_f32, bf16_to_f64, f32_to_bf16, f64_to_bf16, f64_to_f32
from .probes import DEFAULT_ROUNDS, signs

DTYPES = ("f32", "bf16")


def _check_theta(theta, dtype):
    if dtype not in DTYPES:
        raise ValueError("dtype must be 'f32' or 'bf16'")
    want = np.float32 if dtype == "f32" else np.uint16
    theta = np.asarray(theta)
    if theta.dtype != want or theta.ndim != 1:
        raise ValueError(f"{dtype} weights must be a 1-D {np.dtype(want).name} array")
    return theta


def perturb(theta, dtype, offset, seed, step, k, eps, rounds=DEFAULT_ROUNDS):
    """Return theta + eps * z_k over global elements offset .. offset+len(theta)-1."""
    theta = _check_theta(theta, dtype)
    n = theta.shape[0]
    e = np.float32(eps)
    z = signs(offset, n, seed, step, k, rounds)
    delta = np.where(z > 0, e, -e).astype(np.float32)
    with np.errstate(over="ignore", invalid="ignore"):  # IEEE: overflow gives inf, inf - inf NaN
        if dtype == "f32":
            return (theta + delta).astype(np.float32)
        return f32_to_bf16(bf16_to_f32(theta) + delta)


def perturb2(theta, dtype, offset, seed, step, k_a, eps_a, k_b, eps_b, rounds=DEFAULT_ROUNDS):
    """Return theta + (eps_a z_{k_a} + eps_b z_{k_b}), the pair's sum rounded to fp32 first."""
    theta = _check_theta(theta, dtype)
    n = theta.shape[0]
    ea, eb = np.float32(eps_a), np.float32(eps_b)
    da = np.where(signs(offset, n, seed, step, k_a, rounds) > 0, ea, -ea).astype(np.float32)
    db = np.where(signs(offset, n, seed, step, k_b, rounds) > 0, eb, -eb).astype(np.float32)
    with np.errstate(over="ignore", invalid="ignore"):  # IEEE: overflow gives inf, inf - inf NaN
        d = (da + db).astype(np.float32)
        if dtype == "f32":
            return (theta + d).astype(np.float32)
        return f32_to_bf16(bf16_to_f32(theta) + d)


def probe_sum(offset, n, seed, step, c, rounds=DEFAULT_ROUNDS, k_base=0):
    """sum_j c[j] * z_{k_base+j} over the window, in float64 (c taken as float32 values)."""
    c64 = np.asarray(c, dtype=np.float32).astype(np.float64)
    acc = np.zeros(n, dtype=np.float64)
    for j, cj in enumerate(c64):
        acc += cj * signs(offset, n, seed, step, k_base + j, rounds)
    return acc


def update(theta, dtype, offset, seed, step, c, lr, rounds=DEFAULT_ROUNDS, k_base=0):
    """Return round(theta - lr * sum_j c[j] z_{k_base+j}), rounded once to `dtype`."""
    theta = _check_theta(theta, dtype)
    n = theta.shape[0]
    acc = probe_sum(offset, n, seed, step, c, rounds, k_base)
    lr64 = np.float64(np.float32(lr))
    if dtype == "f32":
        return f64_to_f32(theta.astype(np.float64) - lr64 * acc)
    return f64_to_bf16(bf16_to_f64(theta) - lr64 * acc)


def update_restore(theta, dtype, offset, seed, step, c, lr, k_restore, eps_restore,
                   rounds=DEFAULT_ROUNDS, k_base=0):
    """Return round(theta + eps_r z_{k_restore} - lr * sum_j c[j] z_{k_base+j}), rounded once."""
    theta = _check_theta(theta, dtype)
    n = theta.shape[0]
    acc = probe_sum(offset, n, seed, step, c, rounds, k_base)
    er = np.float64(np.float32(eps_restore))
    rz = er * signs(offset, n, seed, step, k_restore, rounds)
    lr64 = np.float64(np.float32(lr))
    if dtype == "f32":
        return f64_to_f32((theta.astype(np.float64) + rz) - lr64 * acc)
    return f64_to_bf16((bf16_to_f64(theta) + rz) - lr64 * acc)


def perturb_schedule(theta, dtype, offset, seed, step, k, eps, rounds=DEFAULT_ROUNDS):
    """Algorithm 1's three applications of probe k: +eps, -2 eps, +eps.

    Returns (theta_plus, theta_minus, theta_restored): the weights seen by the two
    perturbed forward passes and the weights after the restore.
    """
    e = np.float32(eps)
    tp = perturb(theta, dtype, offset, seed, step, k, e, rounds)
    tm = perturb(tp, dtype, offset, seed, step, k, np.float32(-2.0) * e, rounds)
    tr = perturb(tm, dtype, offset, seed, step, k, e, rounds)
    return tp, tm, tr
