"""Philox-4xW counter-based generator, written from its published definition.

TEST INFRASTRUCTURE: part of the CPU oracle. Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import it.

Definition followed: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC'11 (Philox-N x W, N = 4). One round maps the
counter (x0, x1, x2, x3) under the round key (k0, k1) to

    (hi(M1*x2) ^ x1 ^ k0,  lo(M1*x2),  hi(M0*x0) ^ x3 ^ k1,  lo(M0*x0))

where hi/lo are the high and low W-bit halves of the full 2W-bit product, and the key is
bumped by the Weyl constants (W0, W1) after every round (mod 2^W).

The 1.5-SPSA paper does not state which generator produces its packed perturbations
(section 4.3, "Bit-Packed perturbations"; Algorithm 1, PackedPerturbation). Philox4x32
with 10 rounds is the reading taken here; the round count is a parameter.

Pins: at W = 64, R = 10 this function must reproduce numpy.random.Philox bit for bit
(numpy advances the counter by one before each block); at W = 32, R = 10 it must
reproduce rocRAND's Philox4x32-10 engine. Both are independent implementations.
"""

import numpy as np

# (multipliers M0, M1), (Weyl key increments W0, W1), per word width, as published.
CONSTANTS = {
    32: ((0xD2511F53, 0xCD9E8D57), (0x9E3779B9, 0xBB67AE85)),
    64: ((0xD2E7470EE14C6C93, 0xCA5A826395121157),
         (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)),
}

_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(m, x, width):
    """Full product m * x of two width-bit words as (high word, low word), uint64 arrays."""
    x = np.asarray(x, dtype=np.uint64)
    if width == 32:
        p = np.uint64(m) * x  # both factors < 2^32, so the product fits exactly
        return p >> _S32, p & _M32
    # width 64: schoolbook product on 32-bit halves, every partial product exact in uint64
    a1, a0 = np.uint64(m >> 32), np.uint64(m & 0xFFFFFFFF)
    b1, b0 = x >> _S32, x & _M32
    p00, p01, p10, p11 = a0 * b0, a0 * b1, a1 * b0, a1 * b1
    mid = (p00 >> _S32) + (p01 & _M32) + (p10 & _M32)
    lo = (p00 & _M32) | ((mid & _M32) << _S32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    return hi, lo


def philox4(counter, key, width=32, rounds=10):
    """Philox-4 x width with `rounds` rounds.

    counter: four integer arrays (broadcastable), each word < 2^width.
    key: two Python ints, each < 2^width.
    Returns the four output words as uint64 arrays.
    """
    if width not in CONSTANTS:
        raise ValueError("width must be 32 or 64")
    (m0, m1), (w0, w1) = CONSTANTS[width]
    mask = (1 << width) - 1
    x0, x1, x2, x3 = np.broadcast_arrays(*[np.asarray(c, dtype=np.uint64) for c in counter])
    k0, k1 = int(key[0]) & mask, int(key[1]) & mask
    for _ in range(rounds):
        hi0, lo0 = _mulhilo(m0, x0, width)
        hi1, lo1 = _mulhilo(m1, x2, width)
        x0, x1, x2, x3 = (hi1 ^ x1 ^ np.uint64(k0), lo1, hi0 ^ x3 ^ np.uint64(k1), lo0)
        k0 = (k0 + w0) & mask
        k1 = (k1 + w1) & mask
    return x0, x1, x2, x3
