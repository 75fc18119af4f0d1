"""Pins for the oracle's Philox4x64-10: the published known answers and NumPy's
independent implementation."""

import os

import numpy as np
import pytest

from oracle import philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x64_10_kat.txt")


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            v = [int(x, 16) for x in line.split()]
            rows.append((tuple(v[0:4]), tuple(v[4:6]), tuple(v[6:10])))
    return rows


@pytest.mark.parametrize("ctr,key,out", _kat_rows())
def test_known_answers(ctr, key, out):
    assert philox.block(ctr, key) == out


def _numpy_block(ctr, key):
    # numpy advances the 256-bit counter before producing each block, so the
    # block for counter c comes from a generator positioned at c - 1.
    c = ctr[0] | (ctr[1] << 64) | (ctr[2] << 128) | (ctr[3] << 192)
    c = (c - 1) % (1 << 256)
    words = np.array([(c >> (64 * k)) & ((1 << 64) - 1) for k in range(4)], dtype=np.uint64)
    g = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=words)
    return tuple(int(x) for x in g.random_raw(4))


def test_matches_numpy_philox():
    rng = np.random.default_rng(1234)
    for _ in range(200):
        ctr = tuple(int(x) for x in rng.integers(0, 2**63, size=4, dtype=np.int64))
        ctr = (ctr[0] * 2 + 1, ctr[1], ctr[2], 0)
        key = tuple(int(x) for x in rng.integers(0, 2**63, size=2, dtype=np.int64))
        assert philox.block(ctr, key) == _numpy_block(ctr, key)
    # small counters as used by the schedule (step, learner, mini-batch)
    for step in range(3):
        for i in range(4):
            for j in range(3):
                assert philox.block((step, i, j, 0), (0, 1)) == _numpy_block((step, i, j, 0), (0, 1))


def test_u01_open_interval_and_bounded():
    assert 0.0 < philox.u01(0) < 1e-15
    assert 1.0 - 1e-15 < philox.u01((1 << 64) - 1) < 1.0
    for k in (1, 2, 3, 47, 48, 1000):
        assert philox.bounded(0, k) == 0
        assert philox.bounded((1 << 64) - 1, k) == k - 1
    # uniformity of the bounded map over Philox words (chi-square, 6 bins)
    counts = np.zeros(6)
    for t in range(6000):
        counts[philox.bounded(philox.word(7, 2, 0, t), 6)] += 1
    chi2 = ((counts - 1000.0) ** 2 / 1000.0).sum()
    assert chi2 < 20.5  # p ~ 0.001 at 5 degrees of freedom
