"""Philox4x64-10 counter-based generator, vectorised over numpy uint64 arrays.

TEST INFRASTRUCTURE ONLY: part of the CPU oracle.  Only tests, the smoke check
and the benchmark's CPU-baseline leg may import it; the product path never does.

Algorithm: Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11 -- the Philox-4x64 bijection with 10 rounds.  Each round
multiplies counter words 0 and 2 by two fixed odd constants, keeping the full
128-bit products, and mixes the high halves with the other two words and the
round key; the key is advanced by two Weyl constants between rounds.

Pinned against ``numpy.random.Philox`` (an independent library implementation
of the same published generator) in the tests.
"""
import numpy as np

_MASK32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)
PHILOX_M0 = np.uint64(0xD2E7470EE14C6C93)
PHILOX_M1 = np.uint64(0xCA5A826395121157)
PHILOX_W0 = np.uint64(0x9E3779B97F4A7C15)   # golden ratio
PHILOX_W1 = np.uint64(0xBB67AE8584CAA73B)   # sqrt(3) - 1


def _u64(a):
    return np.asarray(a, dtype=np.uint64)


def mulhilo64(a, b):
    """Full 128-bit product of two uint64 arrays as (high, low) words."""
    a = _u64(a)
    b = _u64(b)
    lo = a * b
    a0, a1 = a & _MASK32, a >> _S32
    b0, b1 = b & _MASK32, b >> _S32
    p00 = a0 * b0
    p01 = a0 * b1
    p10 = a1 * b0
    p11 = a1 * b1
    mid = (p00 >> _S32) + (p01 & _MASK32) + (p10 & _MASK32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    return hi, lo


def philox4x64_10(ctr, key):
    """ctr: 4 broadcastable uint64 arrays; key: 2 uint64 arrays.  Returns 4 arrays."""
    c0, c1, c2, c3 = (_u64(c).copy() for c in np.broadcast_arrays(*[_u64(c) for c in ctr]))
    k0, k1 = (_u64(k) for k in key)
    with np.errstate(over="ignore"):
        for r in range(10):
            if r > 0:
                k0 = k0 + PHILOX_W0
                k1 = k1 + PHILOX_W1
            hi0, lo0 = mulhilo64(PHILOX_M0, c0)
            hi1, lo1 = mulhilo64(PHILOX_M1, c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3
