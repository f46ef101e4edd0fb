"""Per-probe update coefficients of 1.5-SPSA, from the antithetic and clean losses.

TEST INFRASTRUCTURE: part of the CPU oracle.

Definitions followed:
  * 3-point directional curvature, section 4.1, Eq. 3:
        chat_k = (L(theta + eps z_k) - 2 L(theta) + L(theta - eps z_k)) / eps^2
  * alpha-saturated weight, section 4.1, Eq. 4:
        w_k = 1 / max(lambda_reg, |chat_k|^alpha),   lambda_reg = 1, alpha = 0.1 by default
    (alpha = 0 recovers 1SPSA, alpha = 1 is a Newton step in probe space).
  * update, section 4.2, Eq. 5 / Eq. 6 and Algorithm 1 (gamma_k = (1/2n) (L+ - L-) w_k):
    theta <- theta - lr * sum_k c_k z_k with
        c_k = w_k (L+_k - L-_k) / (2 K eps).
    Reading: with the paper's tie lr = eps (section 3.1) lr * c_k equals Algorithm 1's
    gamma_k exactly, and with alpha = 0 it is the central difference (L+ - L-)/(2 eps)
    averaged over the K probes. Eq. 2's extra factor 1/2 is read as a typo.

Evaluation order is fixed (float64 throughout), so a C implementation that performs the
same operations in the same order with the same libm pow agrees bit for bit:
    d2   = (L+ - 2*L0) + L-
    chat = d2 / (eps*eps)
    a    = pow(|chat|, alpha)
    den  = a if a > lambda_reg else lambda_reg
    w    = 1 / den
    c64  = ((L+ - L-) * w) / ((2*K) * eps)
    c32  = c64 rounded to float32 (nearest, ties to even)
"""

import math

import numpy as np

DEFAULT_ALPHA = 0.1
DEFAULT_LAMBDA_REG = 1.0


def probe_coeffs(L_plus, L_minus, L_clean, eps, alpha=DEFAULT_ALPHA,
                 lambda_reg=DEFAULT_LAMBDA_REG):
    """Return dict with float32 'c', float64 'c64', 'curv' (chat) and 'w', each of length K.

    Raises ValueError for K = 0, mismatched lengths, non-finite inputs, eps <= 0,
    alpha outside [0, 1] (the range section 4.1 gives) or lambda_reg <= 0.
    Arithmetic is IEEE float64 (numpy scalars, so a vanishing eps*eps gives inf rather
    than a Python exception) and pow is the C library's (math.pow).
    """
    Lp = [float(v) for v in L_plus]
    Lm = [float(v) for v in L_minus]
    K = len(Lp)
    if K == 0 or len(Lm) != K:
        raise ValueError("L_plus and L_minus must have the same non-zero length")
    L0, eps, alpha, lam = float(L_clean), float(eps), float(alpha), float(lambda_reg)
    scalars = Lp + Lm + [L0, eps, alpha, lam]
    if not all(math.isfinite(v) for v in scalars):
        raise ValueError("losses, eps, alpha and lambda_reg must be finite")
    if eps <= 0.0:
        raise ValueError("eps must be positive")
    if not (0.0 <= alpha <= 1.0):
        raise ValueError("alpha must lie in [0, 1]")
    if lam <= 0.0:
        raise ValueError("lambda_reg must be positive")
    c64 = np.empty(K, dtype=np.float64)
    curv = np.empty(K, dtype=np.float64)
    w = np.empty(K, dtype=np.float64)
    f = np.float64
    two = f(2.0)
    with np.errstate(all="ignore"):
        for k in range(K):
            d2 = (f(Lp[k]) - two * f(L0)) + f(Lm[k])
            chat = d2 / (f(eps) * f(eps))
            a = f(math.pow(abs(float(chat)), alpha))
            den = a if a > f(lam) else f(lam)
            wk = f(1.0) / den
            c64[k] = ((f(Lp[k]) - f(Lm[k])) * wk) / ((two * f(K)) * f(eps))
            curv[k] = chat
            w[k] = wk
    with np.errstate(over="ignore"):
        c32 = c64.astype(np.float32)
    return {"c": c32, "c64": c64, "curv": curv, "w": w}
