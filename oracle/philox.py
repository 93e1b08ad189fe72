"""Philox4x64-10, written from its published definition (oracle side).

TEST INFRASTRUCTURE ONLY (see the package header).

The paper draws one i.i.d. Uniform(0,1) score per candidate, per KV head, at
every eviction (Section 3) and makes the draw reproducible with a per-request
seed (Appendix H, "Statistics and randomness").  It names no generator; the
reading adopted here is Philox4x64 with 10 rounds from Salmon, Moraes, Dror
and Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11): a keyed
bijection on four 64-bit counter words, so any draw is a pure function of
(counter, key) and needs no sequential state.

One round maps counter (c0, c1, c2, c3) under key (k0, k1) to
    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))
where hi/lo are the upper/lower 64 bits of the 128-bit product; between
rounds the key is advanced by the Weyl constants (W0, W1).

Parity: pinned.  ``philox4x64_10`` (exact Python integers) is checked against
``numpy.random.Philox``, an independent implementation of the same published
generator; ``philox4x64_10_np`` (vectorised) is checked against it.
"""

import numpy as np

# Multipliers and Weyl key increments of Philox4x64 (Salmon et al., SC'11).
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15
PHILOX_W1 = 0xBB67AE8584CAA73B
ROUNDS = 10

_MASK64 = (1 << 64) - 1


def philox4x64_10(counter, key):
    """One Philox4x64-10 block with exact Python integers.

    counter: 4 ints in [0, 2^64); key: 2 ints in [0, 2^64).
    Returns the 4 output words as Python ints.
    """
    c0, c1, c2, c3 = (int(x) & _MASK64 for x in counter)
    k0, k1 = (int(x) & _MASK64 for x in key)
    for rnd in range(ROUNDS):
        if rnd:
            k0 = (k0 + PHILOX_W0) & _MASK64
            k1 = (k1 + PHILOX_W1) & _MASK64
        p0 = PHILOX_M0 * c0          # exact 128-bit products
        p1 = PHILOX_M1 * c2
        c0, c1, c2, c3 = ((p1 >> 64) ^ c1 ^ k0, p1 & _MASK64,
                          (p0 >> 64) ^ c3 ^ k1, p0 & _MASK64)
    return c0, c1, c2, c3


_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(a, b):
    """Upper and lower 64 bits of a*b for a uint64 constant a and array b.

    The 128-bit product is assembled from four 32x32->64 partial products.
    """
    a = np.uint64(a)
    a_lo, a_hi = a & _M32, a >> _S32
    b_lo, b_hi = b & _M32, b >> _S32
    p00 = a_lo * b_lo
    p01 = a_lo * b_hi
    p10 = a_hi * b_lo
    p11 = a_hi * b_hi
    mid = (p00 >> _S32) + (p01 & _M32) + (p10 & _M32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    lo = (mid << _S32) | (p00 & _M32)
    return hi, lo


def philox4x64_10_np(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x64-10 over numpy uint64 arrays (all broadcast).

    Returns four uint64 arrays, the output words of each block.
    """
    with np.errstate(over="ignore"):
        c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(x, dtype=np.uint64)
                                               for x in (c0, c1, c2, c3)))
        k0 = np.asarray(k0, dtype=np.uint64)
        k1 = np.asarray(k1, dtype=np.uint64)
        for rnd in range(ROUNDS):
            if rnd:
                k0 = k0 + np.uint64(PHILOX_W0)
                k1 = k1 + np.uint64(PHILOX_W1)
            hi0, lo0 = _mulhilo(PHILOX_M0, c0)
            hi1, lo1 = _mulhilo(PHILOX_M1, c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3
