"""Philox4x32-10 counter-based generator -- TEST INFRASTRUCTURE ONLY.

Written from its published definition (J. K. Salmon, M. A. Moraes, R. O. Dror,
D. E. Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011, the
Philox-4x32 bijection with 10 rounds): a 128-bit counter (c0, c1, c2, c3) and a
64-bit key (k0, k1).  One round multiplies c0 and c2 by two fixed odd
constants, keeping the high and low 32-bit halves of the products, and mixes
them with c1, c3 and the key; the key is advanced by two Weyl increments
before every round after the first.  Vectorised over numpy uint64 arrays that
hold 32-bit values.  Used by the oracle to draw the Gumbel noise of Gumbel
top-k retrieval; the GPU side has its own implementation of the same
definition and shares no code with this one.
"""

import numpy as np

M0 = 0xD2511F53
M1 = 0xCD9E8D57
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK = 0xFFFFFFFF


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """The four 32-bit output words for counters (c0..c3) and key (k0, k1);
    arguments broadcast (any integer arrays or scalars < 2^32)."""
    c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) & MASK for x in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=np.uint64) & MASK
    k1 = np.asarray(k1, dtype=np.uint64) & MASK
    for r in range(10):
        if r > 0:
            k0 = (k0 + W0) & MASK
            k1 = (k1 + W1) & MASK
        p0 = c0 * np.uint64(M0)          # < 2^64: exact in uint64
        p1 = c2 * np.uint64(M1)
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3
