"""Pins of the oracle's bf16 storage helpers: torch's RNE cast and exact rational rounding."""

from fractions import Fraction

import numpy as np
import torch

import oracle


def _torch_bf16_bits(x32):
    return torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_f32_to_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(200_000).astype(np.float32) * 0.02,
        rng.standard_normal(10_000).astype(np.float32) * 1e30,
        (rng.standard_normal(10_000) * 1e-39).astype(np.float32),      # subnormals
        np.array([0.0, -0.0, 1.0, -1.0, 3.3895314e38, -3.3895314e38, np.inf, -np.inf,
                  1.401298e-45, -1.401298e-45, 1.1754942e-38], dtype=np.float32),
    ])
    # exact ties: low 16 bits equal to 0x8000 with odd and even kept parts
    u = rng.integers(0, 2 ** 31, 10_000, dtype=np.uint64).astype(np.uint32) & np.uint32(0x7F7F0000)
    ties = (u | np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    np.testing.assert_array_equal(oracle.f32_to_bf16(x), _torch_bf16_bits(x))


def test_bf16_to_f32_matches_torch():
    bits = np.arange(0, 2 ** 16, dtype=np.uint32).astype(np.uint16)
    t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()
    mine = oracle.bf16_to_f32(bits)
    finite = np.isfinite(t)
    np.testing.assert_array_equal(mine[finite].view(np.uint32), t[finite].view(np.uint32))
    assert np.array_equal(np.isnan(mine), np.isnan(t))


def _exact_round_bf16(v):
    """Round a finite float64 to bf16 by exact rational arithmetic (brute force)."""
    if v == 0.0:
        return np.float32(v)
    f = Fraction(v)
    a = abs(f)
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    step = Fraction(2) ** (max(e, -126) - 7)
    q = abs(f) / step
    lo = q.numerator // q.denominator
    rem = q - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    r = lo * step
    if r >= Fraction(2) ** 128:
        return np.float32(np.inf if v > 0 else -np.inf)
    return np.float32(float(r) if v > 0 else -float(r))


def test_f64_to_bf16_single_rounding_exact():
    """f64 -> bf16 rounds once; a double rounding through fp32 would differ on crafted values."""
    rng = np.random.default_rng(1)
    vals = list(rng.standard_normal(3000) * 0.02) + list(rng.standard_normal(500) * 1e-38)
    # values just above a bf16 tie that become an exact tie after rounding to fp32
    for m in range(1, 200):
        base = 1.0 + m * 2.0 ** -7 + 2.0 ** -8          # exact bf16 tie between two codes
        vals += [base + 2.0 ** -40, base - 2.0 ** -40, -(base + 2.0 ** -40)]
    vals += [3.3961e38, 3.39e38, 1e-45, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135]
    x = np.array(vals, dtype=np.float64)
    mine = oracle.f64_to_bf16(x)
    ref = np.array([_exact_round_bf16(v) for v in x], dtype=np.float32)
    ref_bits = (ref.view(np.uint32) >> 16).astype(np.uint16)
    np.testing.assert_array_equal(mine, ref_bits)
    # the crafted near-ties really do expose double rounding through fp32
    dbl = oracle.f32_to_bf16(x.astype(np.float32))
    assert np.count_nonzero(dbl != mine) > 100


def test_f64_to_bf16_nonfinite_and_zero_sign():
    out = oracle.f64_to_bf16(np.array([np.inf, -np.inf, np.nan, 0.0, -0.0]))
    assert out[0] == 0x7F80 and out[1] == 0xFF80
    assert (out[2] & 0x7F80) == 0x7F80 and (out[2] & 0x7F) != 0
    assert out[3] == 0x0000 and out[4] == 0x8000
