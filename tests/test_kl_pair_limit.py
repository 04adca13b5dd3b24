"""The two facts the CE / forward-KL pair limit rests on, checked on random
rows in float64 (no GPU):

* the difference of the two rows' log2 partition sums taken relative to each
  row's largest logit equals log2(max q / max p);
* where |log2(max q / max p)| exceeds a limit t, the row's largest |q - p| is
  at least (1 - 2^-t) times the larger of max q and max p, so an error e in
  that difference (which moves each q - p by at most about e ln2 max(p, q))
  stays within e ln2 / (1 - 2^-t) of the row's largest gradient.
"""

import numpy as np
import pytest


def _softmax(z, T):
    a = z / T
    e = np.exp(a - a.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def _lam(z, T):
    """log2 of the partition sum relative to the row's largest logit."""
    a = z / T
    return np.log2(np.exp(a - a.max(axis=-1, keepdims=True)).sum(axis=-1))


@pytest.mark.parametrize("seed", range(4))
def test_normaliser_gap_is_the_ratio_of_the_largest_probabilities(seed):
    rng = np.random.default_rng(seed)
    R, V = 64, 3000
    s = rng.uniform(0.5, 8.0, size=(R, 1))
    zt = rng.standard_normal((R, V)) * s
    zd = zt + rng.standard_normal((R, V)) * rng.uniform(0.01, 3.0, size=(R, 1))
    T = float(rng.uniform(0.5, 1.5))
    p, q = _softmax(zt, T), _softmax(zd, T)
    gap = _lam(zt, T) - _lam(zd, T)
    np.testing.assert_allclose(gap, np.log2(q.max(axis=-1) / p.max(axis=-1)), rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_beyond_the_limit_the_largest_gradient_is_bounded_below(seed):
    rng = np.random.default_rng(100 + seed)
    R, V = 256, 2000
    s = rng.uniform(0.5, 8.0, size=(R, 1))
    zt = rng.standard_normal((R, V)) * s
    zd = zt + rng.standard_normal((R, V)) * np.logspace(-3, 0.5, R)[:, None]
    p, q = _softmax(zt, 1.0), _softmax(zd, 1.0)
    gap = np.abs(np.log2(q.max(axis=-1) / p.max(axis=-1)))
    largest = np.abs(q - p).max(axis=-1)
    top = np.maximum(q.max(axis=-1), p.max(axis=-1))
    for t in (1.0 / 64, 0.5):
        beyond = gap > t
        assert beyond.sum() >= 10 and (~beyond).sum() >= 10  # both sides are exercised
        assert np.all(largest[beyond] >= (1.0 - 2.0 ** -t) * top[beyond] * (1.0 - 1e-12))
    # it holds at every gap (with equality where the largest |q - p| sits at
    # the larger maximum); 1 - 2^-gap by expm1, which keeps its digits at small gaps
    assert np.all(largest >= -np.expm1(-gap * np.log(2.0)) * top * (1.0 - 1e-9))
