"""Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11), written in numpy from
that paper's definition.

TEST INFRASTRUCTURE ONLY.  This file belongs to the CPU oracle: only the test
suite, the smoke check and the benchmark's CPU-baseline leg may use it.

Definition.  The state is four 32-bit words (c0, c1, c2, c3) and the key two
words (k0, k1).  One round multiplies c0 and c2 by fixed 32-bit constants,
splits each 64-bit product into high and low halves and outputs
    (hi(c2*M1) ^ c1 ^ k0,  lo(c2*M1),  hi(c0*M0) ^ c3 ^ k1,  lo(c0*M0)).
Between rounds the key is advanced by two Weyl increments: the 32-bit
fractions of the golden ratio and of sqrt(3).  Ten rounds make one output
block of four 32-bit words.

How the method uses it (streams, counter layout) is in ``oracle.bmlp``.
"""
from __future__ import annotations

import numpy as np

MASK32 = 0xFFFFFFFF
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9  # floor(2^32 * (golden ratio - 1))
PHILOX_W1 = 0xBB67AE85  # floor(2^32 * (sqrt(3) - 1))
ROUNDS = 10


def philox4x32(c0, c1, c2, c3, k0: int, k1: int, rounds: int = ROUNDS):
    """Apply Philox4x32 with ``rounds`` rounds.

    c0..c3 are integer arrays (or scalars) broadcast against each other;
    k0, k1 are Python ints (the key is the same for every counter here).
    Returns four uint32 arrays.
    """
    c = [np.asarray(v, dtype=np.uint64) & np.uint64(MASK32) for v in (c0, c1, c2, c3)]
    c0, c1, c2, c3 = np.broadcast_arrays(*c)
    m32 = np.uint64(MASK32)
    m0 = np.uint64(PHILOX_M0)
    m1 = np.uint64(PHILOX_M1)
    sh = np.uint64(32)
    k0 = int(k0) & MASK32
    k1 = int(k1) & MASK32
    for r in range(rounds):
        p0 = c0 * m0  # exact: both factors < 2^32, product < 2^64
        p1 = c2 * m1
        n0 = (p1 >> sh) ^ c1 ^ np.uint64(k0)
        n1 = p1 & m32
        n2 = (p0 >> sh) ^ c3 ^ np.uint64(k1)
        n3 = p0 & m32
        c0, c1, c2, c3 = n0, n1, n2, n3
        k0 = (k0 + PHILOX_W0) & MASK32
        k1 = (k1 + PHILOX_W1) & MASK32
    return tuple(v.astype(np.uint32) for v in (c0, c1, c2, c3))


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Philox4x32-10 (the ten-round default)."""
    return philox4x32(c0, c1, c2, c3, k0, k1, ROUNDS)
