"""Pins of the oracle's Philox4x64-10 and of the uniform / Gumbel mapping."""
import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle.philox import philox4x64_10, mulhilo64
from oracle import gdp_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _numpy_philox_block(ctr, key):
    """numpy.random.Philox advances its 256-bit counter by one before producing
    each block of four words, so a state of (ctr - 1) yields the block of ctr."""
    c = [int(x) for x in ctr]
    # subtract one with borrow across the four 64-bit words
    val = sum(w << (64 * i) for i, w in enumerate(c)) - 1
    val %= 1 << 256
    prev = np.array([(val >> (64 * i)) & ((1 << 64) - 1) for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=prev)
    return bg.random_raw(4)


@pytest.mark.parametrize("ctr,key", [
    ((1, 0, 0, 0), (0, 0)),
    ((7, 3, 2, 0), (1005, 0)),
    ((51999, 63, 2, 0), (2004, 0)),
    ((0, 1, 0, 0), (2**64 - 1, 2**63 + 5)),            # borrow path in the numpy state
    ((2**64 - 1, 2**64 - 1, 12345, 2**40), (0xDEADBEEF, 0x1234)),
])
def test_philox_matches_numpy(ctr, key):
    ours = philox4x64_10(tuple(np.uint64(c) for c in ctr), tuple(np.uint64(k) for k in key))
    ref = _numpy_philox_block(ctr, key)
    assert [int(x) for x in ours] == [int(x) for x in ref]


def test_philox_vectorised_matches_numpy_many():
    rng = np.random.default_rng(0)
    ctrs = rng.integers(1, 2**63, size=(64, 4), dtype=np.uint64)
    key = (np.uint64(99), np.uint64(7))
    ours = philox4x64_10(tuple(ctrs[:, i] for i in range(4)), key)
    for r in range(ctrs.shape[0]):
        ref = _numpy_philox_block(ctrs[r], (99, 7))
        assert [int(o[r]) for o in ours] == [int(x) for x in ref]


def test_philox_known_answer():
    path = os.path.join(GOLDEN, "philox4x64_10_kat.txt")
    n = 0
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        f = [int(t, 16) for t in line.split()]
        out = philox4x64_10(tuple(np.uint64(x) for x in f[:4]), tuple(np.uint64(x) for x in f[4:6]))
        assert [int(o) for o in out] == f[6:10]
        n += 1
    assert n >= 1


def test_mulhilo_against_python_ints():
    rng = np.random.default_rng(1)
    a = rng.integers(0, 2**64, size=1000, dtype=np.uint64, endpoint=False)
    b = rng.integers(0, 2**64, size=1000, dtype=np.uint64, endpoint=False)
    hi, lo = mulhilo64(a, b)
    for i in range(0, 1000, 37):
        p = int(a[i]) * int(b[i])
        assert int(hi[i]) == p >> 64 and int(lo[i]) == p & ((1 << 64) - 1)
    for x, y in [(2**64 - 1, 2**64 - 1), (2**63, 2), (0, 5)]:
        h, l = mulhilo64(np.array([x], np.uint64), np.array([y], np.uint64))
        assert int(h[0]) == (x * y) >> 64 and int(l[0]) == (x * y) & ((1 << 64) - 1)


def test_uniforms_layout_and_exactness():
    u = O.gumbel_uniforms(seed=77, n_nodes=50, k_samples=3, n_devices=12)
    assert u.shape == (3, 50, 12)
    assert (u > 0).all() and (u < 1).all()
    # exactly representable in float32
    assert np.array_equal(u.astype(np.float32).astype(np.float64), u)
    # spot-check the counter layout (v, k, 2, j >> 3) and the half selection
    for (k, v, j) in [(0, 0, 0), (2, 49, 7), (1, 13, 9), (2, 3, 11)]:
        w = philox4x64_10((np.uint64(v), np.uint64(k), np.uint64(2), np.uint64(j >> 3)),
                          (np.uint64(77), np.uint64(0)))[(j & 7) >> 1]
        half = (int(w) >> 32) if (j & 1) else (int(w) & 0xFFFFFFFF)
        assert u[k, v, j] == (2 * (half >> 9) + 1) * 2.0 ** -24


def test_uniforms_chi2():
    u = O.gumbel_uniforms(seed=5, n_nodes=4000, k_samples=8, n_devices=8).ravel()
    hist, _ = np.histogram(u, bins=64, range=(0, 1))
    p = stats.chisquare(hist).pvalue
    assert p > 1e-3
