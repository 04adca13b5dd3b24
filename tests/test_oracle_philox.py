"""Pins of the oracle's Philox4x64-10 against numpy's independent
implementation, plus properties of the U24 uniforms."""

import numpy as np
import pytest
from numpy.random import Philox
from scipy import stats

from oracle.philox import draw_words, philox4x64_10, u24

MASK256 = (1 << 256) - 1


def numpy_block(counter_words, key_words):
    """numpy's Philox increments its 256-bit counter before producing a
    block, so the block for counter c is obtained from a generator set to
    c - 1 (mod 2^256)."""
    c = sum(int(w) << (64 * i) for i, w in enumerate(counter_words))
    k = int(key_words[0]) | (int(key_words[1]) << 64)
    g = Philox(counter=(c - 1) & MASK256, key=k)
    return [int(x) for x in g.random_raw(4)]


def test_matches_numpy_random_blocks():
    rng = np.random.default_rng(7)
    for _ in range(200):
        ctr = [int(x) for x in rng.integers(0, 2**64, size=4, dtype=np.uint64)]
        key = [int(x) for x in rng.integers(0, 2**64, size=2, dtype=np.uint64)]
        ours = [int(x) for x in philox4x64_10(np.array(ctr, np.uint64), np.array(key, np.uint64))]
        assert ours == numpy_block(ctr, key)


@pytest.mark.parametrize("ctr,key", [
    ((0, 0, 0, 0), (0, 0)),
    ((1, 0, 0, 0), (0, 0)),
    ((2**64 - 1, 2**64 - 1, 2**64 - 1, 2**64 - 1), (2**64 - 1, 2**64 - 1)),
    ((5, 3, 7, 0), (123456789, 0)),
])
def test_matches_numpy_edge_words(ctr, key):
    ours = [int(x) for x in philox4x64_10(np.array(ctr, np.uint64), np.array(key, np.uint64))]
    assert ours == numpy_block(ctr, key)


def test_draw_words_layout():
    seed, off = 987654321, 42
    rows = np.array([0, 3, 1000])
    steps = np.arange(4)
    w = draw_words(seed, rows, steps, off)
    assert w.shape == (3, 4, 4)
    for a, b in enumerate(rows):
        for s in steps:
            assert [int(x) for x in w[a, s]] == numpy_block((b, s, off, 0), (seed, 0))


def test_u24_grid_and_range():
    w = np.array([0, 1, (1 << 40) - 1, 1 << 40, 2**64 - 1], dtype=np.uint64)
    u = u24(w)
    assert list(u) == [0.0, 0.0, 0.0, 2.0**-24, 1.0 - 2.0**-24]
    assert np.all(u.astype(np.float32).astype(np.float64) == u)


def test_u24_uniform_chi_square():
    w = draw_words(3, np.arange(1 << 14), np.arange(4), 0)
    u = u24(w[..., :2]).ravel()
    assert u.min() >= 0.0 and u.max() < 1.0
    hist = np.histogram(u, bins=64, range=(0.0, 1.0))[0]
    p = stats.chisquare(hist).pvalue
    assert p > 1e-3, p
