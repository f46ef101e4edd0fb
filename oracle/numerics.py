"""Storage-format helpers for the oracle: bfloat16 as uint16 bit patterns.

TEST INFRASTRUCTURE: part of the CPU oracle.

The paper keeps weights in bf16 (section 4.3, "Bit-Packed perturbations", which compares
against unpacked bf16) and does not discuss rounding. Readings used here:
  * a bf16 value widens to fp32 exactly (the bf16 bits are the high half of the fp32 bits);
  * fp32 -> bf16 and fp64 -> bf16 round to nearest, ties to even, in ONE step;
  * NaN stays NaN (quiet), infinities stay infinite, signed zeros keep their sign.
"""

import numpy as np


def bf16_to_f32(bits):
    """Widen bf16 bit patterns (uint16) to float32 values, exactly."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_to_f64(bits):
    return bf16_to_f32(bits).astype(np.float64)


def f64_to_bf16(x):
    """Round float64 values to bf16 bit patterns: nearest, ties to even, one rounding.

    bf16 keeps 8 significant bits and fp32's exponent range, so a finite x with
    2^(e-1) <= |x| < 2^e (numpy.frexp exponent e) is rounded to a multiple of
    2^(e-8); below the smallest normal 2^-126 the spacing is the subnormal step 2^-133.
    Scaling by a power of two is exact, numpy.rint rounds half to even, and the
    rounded value is exactly representable, so the only rounding is the one intended.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    finite = np.isfinite(x)
    ax = np.abs(np.where(finite, x, 0.0))
    _, e = np.frexp(ax)
    q = np.maximum(e.astype(np.int32) - 8, -133).astype(np.int32)
    r = np.rint(np.ldexp(ax, -q))
    y = np.ldexp(r, q)
    over = y >= 2.0 ** 128
    with np.errstate(over="ignore"):
        y32 = np.where(over, np.inf, y).astype(np.float32)
    y32 = np.copysign(y32, np.where(finite, x, 1.0).astype(np.float32))
    bits = (y32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    out[...] = bits
    # non-finite inputs: infinities keep sign; NaN becomes a quiet NaN with its sign
    sign = np.signbit(x).astype(np.uint16) << np.uint16(15)
    out[np.isinf(x)] = (sign | np.uint16(0x7F80))[np.isinf(x)]
    out[np.isnan(x)] = (sign | np.uint16(0x7FC0))[np.isnan(x)]
    return out


def f32_to_bf16(x):
    """Round float32 values to bf16 bit patterns (nearest, ties to even).

    Every float32 is exactly a float64, so this is f64_to_bf16 of the same value.
    """
    return f64_to_bf16(np.asarray(x, dtype=np.float32).astype(np.float64))


def f64_to_f32(x):
    """Round float64 to float32, nearest with ties to even (numpy's IEEE cast)."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float64).astype(np.float32)
