"""Philox4x32-10 counter-based generator, written from its published definition
(Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
SC 2011): a 4 x 32-bit counter and a 2 x 32-bit key go through 10 rounds; each
round multiplies words 0 and 2 by fixed 32-bit constants, keeps both halves of
the 64-bit products, and mixes the high halves with words 1 and 3 and the
round key; the key is advanced by two Weyl constants between rounds.

TEST INFRASTRUCTURE: part of the CPU oracle.  Only the tests, the smoke check
and the benchmark's CPU-baseline leg may import this module.

This is the oracle's own implementation.  It is pinned by the tests against an
independently written, installed open-source implementation (PyTorch's
header-only Philox engine, compiled on the host for the test).
"""

from __future__ import annotations

import numpy as np

MASK32 = np.uint64(0xFFFFFFFF)
M0 = np.uint64(0xD2511F53)  # multiplier for word 0
M1 = np.uint64(0xCD9E8D57)  # multiplier for word 2
W0 = 0x9E3779B9             # key increment, word 0
W1 = 0xBB67AE85             # key increment, word 1


def philox4x32_10(c0, c1, c2, c3, k0, k1, rounds: int = 10):
    """Vectorised Philox4x32.  Counter words ``c0..c3`` are arrays (or scalars)
    of values < 2**32; ``k0, k1`` are the two key words (Python ints).
    Returns four uint32 arrays (the output words x0..x3)."""
    x0, x1, x2, x3 = (np.asarray(c, dtype=np.uint64) & MASK32 for c in (c0, c1, c2, c3))
    x0, x1, x2, x3 = np.broadcast_arrays(x0, x1, x2, x3)
    ka, kb = int(k0) & 0xFFFFFFFF, int(k1) & 0xFFFFFFFF
    for r in range(rounds):
        if r > 0:
            ka = (ka + W0) & 0xFFFFFFFF
            kb = (kb + W1) & 0xFFFFFFFF
        p0 = M0 * x0  # < 2**64: both factors are below 2**32
        p1 = M1 * x2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        x0, x1, x2, x3 = (hi1 ^ x1 ^ np.uint64(ka), lo1, hi0 ^ x3 ^ np.uint64(kb), lo0)
    return tuple(v.astype(np.uint32) for v in (x0, x1, x2, x3))
