"""Philox4x32-10 counter-based generator, vectorised over NumPy arrays.

Written from the published definition (Salmon, Moraes, Dror and Shaw,
"Parallel Random Numbers: As Easy as 1, 2, 3", SC'11, Sec. 4): a 128-bit
counter (c0, c1, c2, c3) and a 64-bit key (k0, k1) go through ten rounds of

    (hi0, lo0) = M0 * c0          (hi1, lo1) = M1 * c2          (64-bit products)
    c' = (hi1 ^ c1 ^ k0,  lo1,  hi0 ^ c3 ^ k1,  lo0)

with the key bumped by the Weyl constants (W0, W1) between rounds.  Every
output word is a pure function of (key, counter), so any element of a
synthetic data set can be regenerated on its own.  The HIP generator in
``synth/csrc`` implements the same definition; neither side holds any of the
search method's arithmetic.
"""
from __future__ import annotations

import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = np.uint32(0x9E3779B9)
W1 = np.uint32(0xBB67AE85)
_MASK32 = np.uint64(0xFFFFFFFF)
_SH32 = np.uint64(32)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Apply Philox4x32-10 elementwise.

    All arguments are broadcastable uint32 arrays (or scalars).  Returns the
    four uint32 output words as a tuple of arrays.
    """
    c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(c, dtype=np.uint32) for c in (c0, c1, c2, c3)))
    # words held in uint64 (values below 2^32), so the 32x32 -> 64 products
    # need no conversions
    c0, c1, c2, c3 = (c.astype(np.uint64) for c in (c0, c1, c2, c3))
    k0 = int(k0) & 0xFFFFFFFF
    k1 = int(k1) & 0xFFFFFFFF
    for rnd in range(10):
        p0 = M0 * c0
        p1 = M1 * c2
        c0, c1, c2, c3 = ((p1 >> _SH32) ^ c1) ^ np.uint64(k0), p1 & _MASK32, \
            ((p0 >> _SH32) ^ c3) ^ np.uint64(k1), p0 & _MASK32
        k0 = (k0 + int(W0)) & 0xFFFFFFFF
        k1 = (k1 + int(W1)) & 0xFFFFFFFF
    c0, c1, c2, c3 = (c.astype(np.uint32) for c in (c0, c1, c2, c3))
    return c0, c1, c2, c3
