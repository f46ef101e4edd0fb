"""Stiff-paraboloid driver (section 5.3, appendix A.2) over a pluggable sweep backend.

A step is Algorithm 1 on one device with the forward pass J(x) = x^T A x: the clean loss,
then per probe the +eps / -2 eps / +eps applications around the two perturbed losses, the
coefficients, and the fused update. The backend supplies perturb(x, k, e, step),
coeffs(L+, L-, L0, eps, alpha) -> c, update(x, c, lr, step) and loss(x); the same loop
drives the CPU oracle and the GPU library.
"""

import math


def steps_to_converge(backend, x, lr, K, eps, alpha, max_steps, tol):
    """Steps until J < tol * J(x0); None if the run diverges, max_steps if it never gets there."""
    J0 = backend.loss(x)
    for s in range(max_steps):
        L0 = backend.loss(x)
        lp, lm = [], []
        for k in range(K):
            x = backend.perturb(x, k, eps, s)
            lp.append(backend.loss(x))
            x = backend.perturb(x, k, -2.0 * eps, s)
            lm.append(backend.loss(x))
            x = backend.perturb(x, k, eps, s)
        c = backend.coeffs(lp, lm, L0, eps, alpha)
        x = backend.update(x, c, lr, s)
        J = backend.loss(x)
        if not math.isfinite(J) or J > 1e6 * J0:
            return None
        if J < tol * J0:
            return s + 1
    return max_steps


def best_steps(make_backend, lrs, K, eps, alpha, max_steps, tol):
    """Fewest steps over a grid of step sizes (each solver gets its own tuned step size).
    The largest step size runs first and every later run stops once it cannot beat the best
    count so far, which leaves the minimum unchanged. None if every run diverges."""
    best = None
    for lr in sorted(lrs, reverse=True):
        backend, x0 = make_backend()
        n = steps_to_converge(backend, x0, lr, K, eps, alpha, max_steps if best is None else best, tol)
        if n is not None and (best is None or n < best):
            best = n
    return best


def trend(job, kappas, alphas, seeds, procs):
    """{(kappa, alpha, seed): best steps} for every combination, job((kappa, alpha, seed))
    computing one entry, in `procs` forked worker processes."""
    import multiprocessing
    keys = [(k, a, s) for k in kappas for a in alphas for s in seeds]
    # the slowest combinations (large kappa, plain 1SPSA) first, so that the pool stays busy
    keys.sort(key=lambda t: (-t[0], t[1]))
    with multiprocessing.get_context("fork").Pool(procs) as pool:
        return dict(zip(keys, pool.map(job, keys, chunksize=1)))
