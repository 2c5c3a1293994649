"""Pins for the oracle's Philox4x64-10 (CPU only).

Two independent anchors: the Random123 known-answer vectors, and
numpy.random.Philox (a third-party implementation).  numpy advances its
counter by one before producing a block, so numpy(counter=c) yields the
block at counter c + 1.
"""
import os

import numpy as np
import pytest

from oracle import philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x64_10_kat.txt")
M64 = (1 << 64) - 1


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([int(v, 16) for v in line.split()])
    return rows


def test_known_answer_vectors_scalar_and_vector():
    rows = _kat_rows()
    assert len(rows) == 3
    for r in rows:
        ctr, key, want = r[0:4], r[4:6], tuple(r[6:10])
        assert philox.philox4x64_scalar(ctr, key) == want
        got = philox.philox4x64(*[np.array([c], dtype=np.uint64) for c in ctr], *key)
        assert tuple(int(w[0]) for w in got) == want


def test_known_answer_vectors_agree_with_numpy():
    # The stored vectors are themselves checked against the third-party
    # implementation, so the fixture cannot carry a transcription error.
    for r in _kat_rows():
        assert _numpy_block(r[0:4], r[4:6]) == tuple(r[6:10])


def _numpy_block(ctr, key):
    """Block at `ctr` from numpy's independent Philox (pre-increment)."""
    c = ctr[0] | (ctr[1] << 64) | (ctr[2] << 128) | (ctr[3] << 192)
    c = (c - 1) % (1 << 256)
    words = np.array([(c >> (64 * j)) & M64 for j in range(4)], dtype=np.uint64)
    bg = np.random.Philox(counter=words, key=np.array(key, dtype=np.uint64))
    return tuple(int(v) for v in bg.random_raw(4))


def test_against_numpy_philox_random_counters():
    rng = np.random.default_rng(1234)
    for _ in range(200):
        ctr = [int(v) for v in rng.integers(0, 2**63, size=4, dtype=np.int64)]
        ctr = [c * 2 + int(rng.integers(0, 2)) for c in ctr]
        key = [int(v) * 2 + 1 for v in rng.integers(0, 2**62, size=2, dtype=np.int64)]
        assert philox.philox4x64_scalar(ctr, key) == _numpy_block(ctr, key)


@pytest.mark.parametrize("ctr", [[1, 0, 0, 0], [M64, 5, 0, 0], [7, M64, 3, 2],
                                 [123456789, 63, 199, 1]])
def test_against_numpy_philox_edges(ctr):
    for key in ([0, 0], [M64, M64], [42, 0]):
        assert philox.philox4x64_scalar(ctr, key) == _numpy_block(ctr, key)


def test_vectorised_matches_scalar():
    rng = np.random.default_rng(5)
    n = 300
    cols = [rng.integers(0, 2**63, size=n, dtype=np.int64).astype(np.uint64) * np.uint64(2)
            + rng.integers(0, 2, size=n, dtype=np.int64).astype(np.uint64) for _ in range(4)]
    k0, k1 = 0x0123456789ABCDEF, 0xFEDCBA9876543210
    out = philox.philox4x64(*cols, k0, k1)
    for j in range(n):
        want = philox.philox4x64_scalar([int(c[j]) for c in cols], [k0, k1])
        assert tuple(int(w[j]) for w in out) == want


def test_mulhilo_limbs_exact():
    rng = np.random.default_rng(9)
    a = rng.integers(0, 2**63, size=1000, dtype=np.int64).astype(np.uint64) * np.uint64(2) + np.uint64(1)
    for b in (philox.PHILOX_M0, philox.PHILOX_M1, M64, 1):
        with np.errstate(over="ignore"):
            hi, lo = philox._mulhilo(a, b)
        for j in range(0, 1000, 37):
            p = int(a[j]) * b
            assert int(hi[j]) == p >> 64 and int(lo[j]) == p & M64
