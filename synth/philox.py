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
    c0 = np.asarray(c0, dtype=np.uint32)
    c1 = np.asarray(c1, dtype=np.uint32)
    c2 = np.asarray(c2, dtype=np.uint32)
    c3 = np.asarray(c3, dtype=np.uint32)
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    c0 = c0.astype(np.uint32)
    c1 = c1.astype(np.uint32)
    c2 = c2.astype(np.uint32)
    c3 = c3.astype(np.uint32)
    k0 = np.uint32(k0)
    k1 = np.uint32(k1)
    with np.errstate(over="ignore"):
        for rnd in range(10):
            p0 = M0 * c0.astype(np.uint64)
            p1 = M1 * c2.astype(np.uint64)
            hi0 = (p0 >> _SH32).astype(np.uint32)
            lo0 = (p0 & _MASK32).astype(np.uint32)
            hi1 = (p1 >> _SH32).astype(np.uint32)
            lo1 = (p1 & _MASK32).astype(np.uint32)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
            if rnd != 9:
                k0 = np.uint32(k0 + W0)
                k1 = np.uint32(k1 + W1)
    return c0, c1, c2, c3
