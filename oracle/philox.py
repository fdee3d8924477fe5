"""Philox4x64-10, the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel Random Numbers: As Easy as 1, 2, 3" (SC 2011), written out in numpy.

TEST INFRASTRUCTURE (part of the oracle): only tests, the smoke check and the
benchmark's CPU-baseline leg may use this module.

The paper draws the NCA's stochastic update mask with PyTorch's generator
(supplement S3; supplement S6, Listing 3), which cannot be reproduced across
devices.  Here the mask bit of a cell is a pure function of
(seed, level, step, cell index), so the GPU and this oracle draw the same
mask; see ``oracle.octree_nca.fire_mask``.

Pinned by: known answers of ``numpy.random.Philox`` (an independent
implementation of the same generator) in tests/test_oracle_philox.py.
"""
from __future__ import annotations

import numpy as np

# Multipliers and Weyl key increments of Philox4x64 (Salmon et al., 2011).
M0 = np.uint64(0xD2E7470EE14C6C93)
M1 = np.uint64(0xCA5A826395121157)
W0 = np.uint64(0x9E3779B97F4A7C15)
W1 = np.uint64(0xBB67AE8584CAA73B)
ROUNDS = 10

_LO32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def mulhilo64(a: np.ndarray, b: np.uint64):
    """Full 128-bit product of uint64 ``a`` (array) and ``b`` (scalar):
    returns (high 64 bits, low 64 bits), from 32-bit partial products."""
    a = np.asarray(a, dtype=np.uint64)
    a0, a1 = a & _LO32, a >> _S32
    b0, b1 = b & _LO32, b >> _S32
    p00 = a0 * b0
    p01 = a0 * b1
    p10 = a1 * b0
    p11 = a1 * b1
    mid = (p00 >> _S32) + (p01 & _LO32) + (p10 & _LO32)   # < 3 * 2^32, no overflow
    lo = (p00 & _LO32) | ((mid & _LO32) << _S32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    return hi, lo


def philox4x64(counter, key, rounds: int = ROUNDS):
    """Apply the Philox4x64 bijection to ``counter`` = (c0, c1, c2, c3) under
    ``key`` = (k0, k1).  Every element may be a numpy uint64 array (broadcast
    together).  Returns the four 64-bit output words.

    One round: multiply words 0 and 2 by the two multipliers; the new word 0 is
    hi(M1*c2) ^ c1 ^ k0, word 1 is lo(M1*c2), word 2 is hi(M0*c0) ^ c3 ^ k1 and
    word 3 is lo(M0*c0).  The key is bumped by the Weyl constants between
    rounds."""
    with np.errstate(over="ignore"):
        x0, x1, x2, x3 = (np.asarray(c, dtype=np.uint64) for c in counter)
        k0, k1 = (np.asarray(k, dtype=np.uint64) for k in key)
        for r in range(rounds):
            hi0, lo0 = mulhilo64(x0, M0)
            hi1, lo1 = mulhilo64(x2, M1)
            x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
            if r + 1 < rounds:
                k0 = k0 + W0
                k1 = k1 + W1
        return x0, x1, x2, x3
