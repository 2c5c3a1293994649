"""Philox4x64-10, the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3" (SC'11), written from that
paper's description: a 4-word counter and 2-word key; each of ten rounds
multiplies words 0 and 2 by fixed odd constants, swaps and xors the high
halves with the other words and the round key; the key is bumped by two
Weyl constants between rounds.

Test infrastructure (see the package docstring).  Two forms are given: a
scalar one on Python integers (obviously correct, slow) and a vectorised one
on numpy uint64 arrays.  Both are pinned against the Random123 known-answer
vectors and against numpy.random.Philox, an independent implementation.
"""
from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1
# Multipliers and Weyl key increments of Philox4x64 (Salmon et al., SC'11).
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15  # golden ratio
PHILOX_W1 = 0xBB67AE8584CAA73B  # sqrt(3) - 1
ROUNDS = 10


def philox4x64_scalar(ctr, key, rounds: int = ROUNDS):
    """One block: ctr is 4 ints, key is 2 ints (each < 2**64); returns 4 ints."""
    x0, x1, x2, x3 = (int(c) & MASK64 for c in ctr)
    k0, k1 = (int(k) & MASK64 for k in key)
    for r in range(rounds):
        if r > 0:
            k0 = (k0 + PHILOX_W0) & MASK64
            k1 = (k1 + PHILOX_W1) & MASK64
        p0 = PHILOX_M0 * x0  # exact 128-bit products on Python ints
        p1 = PHILOX_M1 * x2
        x0, x1, x2, x3 = ((p1 >> 64) ^ x1 ^ k0, p1 & MASK64,
                          (p0 >> 64) ^ x3 ^ k1, p0 & MASK64)
    return x0, x1, x2, x3


_U32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(a: np.ndarray, b: int):
    """(hi, lo) 64-bit halves of the 128-bit product a*b, a uint64 array.

    Split into 32-bit limbs so every partial product fits in uint64."""
    b = np.uint64(b)
    a_lo, a_hi = a & _U32, a >> _S32
    b_lo, b_hi = b & _U32, b >> _S32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> _S32) + (lh & _U32) + (hl & _U32)
    hi = hh + (lh >> _S32) + (hl >> _S32) + (mid >> _S32)
    lo = a * b  # wraps modulo 2**64
    return hi, lo


def philox4x64(c0, c1, c2, c3, k0, k1, rounds: int = ROUNDS):
    """Vectorised Philox4x64: arguments broadcast as uint64 arrays."""
    with np.errstate(over="ignore"):
        x0, x1, x2, x3 = np.broadcast_arrays(*(np.asarray(c, dtype=np.uint64)
                                               for c in (c0, c1, c2, c3)))
        x0, x1, x2, x3 = (np.array(v, dtype=np.uint64) for v in (x0, x1, x2, x3))
        k0 = np.uint64(int(k0) & MASK64)
        k1 = np.uint64(int(k1) & MASK64)
        for r in range(rounds):
            if r > 0:
                k0 = np.uint64((int(k0) + PHILOX_W0) & MASK64)
                k1 = np.uint64((int(k1) + PHILOX_W1) & MASK64)
            hi0, lo0 = _mulhilo(x0, PHILOX_M0)
            hi1, lo1 = _mulhilo(x2, PHILOX_M1)
            x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return x0, x1, x2, x3
