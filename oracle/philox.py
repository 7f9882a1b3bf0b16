"""Philox4x32-10 counter-based generator, written from its published definition.

Test infrastructure: only the tests, the smoke check and the bench's CPU
baseline may import this module; the GPU library never does.

Definition (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11, the Philox family): a 128-bit counter (c0, c1, c2, c3) and a
64-bit key (k0, k1) go through 10 rounds.  One round multiplies c0 and c2 by
the two round multipliers, splits each 64-bit product into hi/lo halves and
outputs (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0)).
Between rounds the key is bumped by the two Weyl constants.

The paper draws Klein's random roundings without naming a generator.  The
draws here are keyed so a run is reproducible and order-free: the draw for
row i of column j on Klein sample k is Philox(counter=(i, j, k, 0),
key=(seed mod 2^32, seed div 2^32)), turned into a uniform double in [0, 1)
from the first two output words with the 27+26-bit "res53" construction of
Matsumoto and Nishimura (mt19937ar.c, genrand_res53).
"""

from __future__ import annotations

import numpy as np

MASK32 = np.uint64(0xFFFFFFFF)
PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = np.uint64(0x9E3779B9)
PHILOX_W1 = np.uint64(0xBB67AE85)


def philox4x32_10(ctr, key):
    """Vectorised Philox4x32-10.

    ctr: 4 integer arrays (or scalars) with values < 2^32; key: 2 of them.
    Returns the 4 output words as uint64 arrays holding 32-bit values.
    """
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & MASK32 for c in ctr)
    k0, k1 = (np.asarray(k, dtype=np.uint64) & MASK32 for k in key)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = PHILOX_M0 * c0          # < 2^64: exact in uint64
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def uniform53(seed: int, i, j, k):
    """Uniform double in [0, 1) for Klein draw (row i, column j, sample k).

    The words are pinned by the published known-answer vectors; the mapping
    of two words to one double (res53) is a chosen convention, since
    the paper names no generator, and is pinned only by its definition."""
    seed = int(seed)
    i = np.asarray(i, dtype=np.uint64)
    j = np.asarray(j, dtype=np.uint64)
    k = np.asarray(k, dtype=np.uint64)
    zero = np.zeros(np.broadcast(i, j, k).shape, dtype=np.uint64)
    x0, x1, _, _ = philox4x32_10((i + zero, j + zero, k + zero, zero),
                                 (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))
    a = (x0 >> np.uint64(5)).astype(np.float64)   # 27 bits
    b = (x1 >> np.uint64(6)).astype(np.float64)   # 26 bits
    return (a * 67108864.0 + b) / 9007199254740992.0
