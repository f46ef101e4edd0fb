"""Rademacher probes z_k regenerated from (seed, step, k, element index).

TEST INFRASTRUCTURE: part of the CPU oracle.

What the paper fixes:
  * probes are Rademacher, z in {-1, +1}^d, so the coordinate-wise inverse is z itself
    (section 2, 1SPSA estimator, Eq. 2);
  * probes are regenerated from a seed rather than stored, and are "8-bit packed"
    (abstract; section 4.3, "Bit-Packed perturbations" and "Seed-Based Distribution");
  * a set bit means +1 and a clear bit means -1, least significant bit first
    (appendix F, the unpack-and-apply kernels).

Readings (the paper does not state the generator or the packing order):
  * element i belongs to tile t = i // 16; one Philox4x32 call per (tile, probe group)
    with counter (t mod 2^32, t // 2^32, step, g) and key (seed mod 2^32, seed // 2^32)
    yields four 32-bit words x0..x3 = 16 bytes;
  * element i's byte is byte (i mod 4) of word x_{(i mod 16) // 4} (little-endian order);
  * one byte carries eight probes of one element: probe k uses group g = k // 8 and
    bit k mod 8 of that byte.
"""

import numpy as np

from .philox import philox4

TILE = 16            # elements per generator call
PROBES_PER_GROUP = 8  # probes carried by one byte
DEFAULT_ROUNDS = 10


def _check_common(seed, step):
    if not (0 <= int(seed) < 2 ** 64):
        raise ValueError("seed must fit in 64 bits")
    if not (0 <= int(step) < 2 ** 32):
        raise ValueError("step must fit in 32 bits")


def tile_words(tiles, seed, step, group, rounds=DEFAULT_ROUNDS):
    """The four Philox output words for each tile index in `tiles` (uint64 arrays)."""
    _check_common(seed, step)
    if not (0 <= int(group) < 2 ** 32):
        raise ValueError("group must fit in 32 bits")
    t = np.asarray(tiles, dtype=np.uint64)
    counter = (t & np.uint64(0xFFFFFFFF), t >> np.uint64(32),
               np.uint64(step), np.uint64(group))
    seed = int(seed)
    return philox4(counter, (seed & 0xFFFFFFFF, seed >> 32), width=32, rounds=rounds)


def tile_bytes(tile_begin, n_tiles, seed, step, group, rounds=DEFAULT_ROUNDS):
    """uint8 array [n_tiles, 16]: byte j of a tile is byte (j mod 4) of word j // 4."""
    tiles = np.uint64(tile_begin) + np.arange(n_tiles, dtype=np.uint64)
    words = tile_words(tiles, seed, step, group, rounds)
    out = np.empty((n_tiles, TILE), dtype=np.uint8)
    for j in range(TILE):
        w = words[j // 4]
        out[:, j] = ((w >> np.uint64(8 * (j % 4))) & np.uint64(0xFF)).astype(np.uint8)
    return out


def element_bytes(offset, n, seed, step, group, rounds=DEFAULT_ROUNDS):
    """The packed byte of probe group `group` for global elements offset .. offset+n-1."""
    if n == 0:
        return np.zeros(0, dtype=np.uint8)
    offset = int(offset)
    t_first = offset // TILE
    t_last = (offset + n - 1) // TILE
    table = tile_bytes(t_first, t_last - t_first + 1, seed, step, group, rounds)
    i = np.uint64(offset) + np.arange(n, dtype=np.uint64)
    return table[(i // np.uint64(TILE) - np.uint64(t_first)).astype(np.int64),
                 (i % np.uint64(TILE)).astype(np.int64)]


def signs(offset, n, seed, step, k, rounds=DEFAULT_ROUNDS):
    """z_k[offset .. offset+n-1] as an int8 array of +1 / -1 (set bit -> +1)."""
    k = int(k)
    if not (0 <= k < 2 ** 32):
        raise ValueError("probe index must fit in 32 bits")
    b = element_bytes(offset, n, seed, step, k // PROBES_PER_GROUP, rounds)
    bit = (b >> np.uint8(k % PROBES_PER_GROUP)) & np.uint8(1)
    return np.where(bit == 1, np.int8(1), np.int8(-1))


def materialize_Z(offset, n, K, seed, step, rounds=DEFAULT_ROUNDS, k_base=0):
    """The probe matrix Z = [z_{k_base} ... z_{k_base+K-1}] of section 4.2 (Eq. 6), as int8 [n, K]."""
    Z = np.empty((n, K), dtype=np.int8)
    for j in range(K):
        Z[:, j] = signs(offset, n, seed, step, k_base + j, rounds)
    return Z
