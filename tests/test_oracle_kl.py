"""Pins of the CE / forward-KL / reverse-KL oracle against scipy's entropy,
relative-entropy and xlogy routines, central finite differences of the
losses, the identity CE = H(p) + KL(p||q), Pinsker's inequality (Sec. 4.3),
and the q = p special case."""

import numpy as np
import pytest
from scipy import special, stats

from oracle.kl import KIND_CE, KIND_FORWARD, KIND_REVERSE, kl_ref, log_softmax_t
from paper_2606_12370_amd import workloads as W

KINDS = [KIND_FORWARD, KIND_CE, KIND_REVERSE]


def _rows(seed, N=3, K=2, V=40, noise=1.0):
    rng = np.random.default_rng(seed)
    zt = rng.normal(0, 2, size=(N, K, V))
    zd = zt + rng.normal(0, noise, size=(N, K, V))
    return zt, zd


def test_log_softmax_matches_scipy():
    zt, _ = _rows(0)
    for T in (0.7, 1.3):
        np.testing.assert_allclose(log_softmax_t(zt, T), special.log_softmax(zt / T, axis=-1), rtol=1e-13)
    # shift invariance with logits far outside exp's range
    np.testing.assert_allclose(log_softmax_t(zt + 1000.0, 0.5), special.log_softmax(zt / 0.5, axis=-1), rtol=1e-9)


@pytest.mark.parametrize("T", [1.0, 0.6])
def test_losses_against_scipy(T):
    zt, zd = _rows(1)
    fk = kl_ref(zt, zd, T, KIND_FORWARD)["per_step"]
    ce = kl_ref(zt, zd, T, KIND_CE)["per_step"]
    rk = kl_ref(zt, zd, T, KIND_REVERSE)["per_step"]
    for n in range(zt.shape[0]):
        for k in range(zt.shape[1]):
            p = special.softmax(zt[n, k] / T)
            q = special.softmax(zd[n, k] / T)
            np.testing.assert_allclose(fk[n, k], stats.entropy(p, q), rtol=1e-11)
            np.testing.assert_allclose(fk[n, k], special.rel_entr(p, q).sum(), rtol=1e-11)
            np.testing.assert_allclose(rk[n, k], stats.entropy(q, p), rtol=1e-11)
            np.testing.assert_allclose(ce[n, k], -special.xlogy(p, q).sum(), rtol=1e-11)
            np.testing.assert_allclose(ce[n, k], stats.entropy(p) + stats.entropy(p, q), rtol=1e-11)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("K,T", [(1, 1.0), (3, 0.7)])
def test_gradient_matches_finite_differences(kind, K, T):
    zt, zd = _rows(2, N=2, K=K, V=12)
    scale = 1.7
    out = kl_ref(zt, zd, T, kind, scale)
    h = 1e-6
    fd = np.zeros_like(zd)
    for idx in np.ndindex(zd.shape):
        zp = zd.copy(); zp[idx] += h
        zm = zd.copy(); zm[idx] -= h
        fd[idx] = (kl_ref(zt, zp, T, kind, scale)["loss"] - kl_ref(zt, zm, T, kind, scale)["loss"]) / (2 * h)
    np.testing.assert_allclose(out["grad"], fd, rtol=1e-6, atol=1e-8)
    # softmax is shift invariant: every gradient row sums to 0
    np.testing.assert_allclose(out["grad"].sum(axis=-1), 0.0, atol=1e-13)


def test_forward_and_ce_share_the_gradient_and_reduce_at_q_equals_p():
    zt, zd = _rows(3)
    a = kl_ref(zt, zd, 0.9, KIND_FORWARD)
    b = kl_ref(zt, zd, 0.9, KIND_CE)
    np.testing.assert_allclose(a["grad"], b["grad"], rtol=0, atol=0)
    same = [kl_ref(zt, zt, 0.9, kind) for kind in KINDS]
    np.testing.assert_allclose(same[0]["per_step"], 0.0, atol=1e-13)
    np.testing.assert_allclose(same[2]["per_step"], 0.0, atol=1e-13)
    H = np.array([[stats.entropy(special.softmax(zt[n, k] / 0.9)) for k in range(zt.shape[1])]
                  for n in range(zt.shape[0])])
    np.testing.assert_allclose(same[1]["per_step"], H, rtol=1e-12)
    for s in same:
        np.testing.assert_allclose(s["grad"], 0.0, atol=1e-15)


def test_pinsker_bound():
    """Sec. 4.3 (Eq. pinsker): d_TV(p, q) <= sqrt(KL(p||q) / 2)."""
    zt, zd = _rows(4, N=50, K=1, V=30, noise=2.0)
    kl = kl_ref(zt, zd, 1.0, KIND_FORWARD)["per_step"][:, 0]
    p = special.softmax(zt[:, 0], axis=-1)
    q = special.softmax(zd[:, 0], axis=-1)
    tv = 0.5 * np.abs(p - q).sum(axis=-1)
    assert np.all(tv <= np.sqrt(kl / 2) + 1e-15)


def test_loss_reduction_and_zero_weights():
    d = W.tv_inputs_numpy(5, 3, 64, W.F32, 6)
    out = kl_ref(d["target"], d["draft"], 1.0, KIND_FORWARD, scale=0.5)
    np.testing.assert_allclose(out["loss"], 0.5 * out["per_step"].mean(axis=1).sum(), rtol=1e-14)
    # p_v = 0 contributes nothing to forward KL or CE; q_v = 0 nothing to reverse KL
    zt = np.zeros((1, 1, 4)); zt[0, 0, 0] = -np.inf
    zd = np.zeros((1, 1, 4)); zd[0, 0, 1] = -np.inf
    f = kl_ref(zt, np.zeros((1, 1, 4)), 1.0, KIND_FORWARD)
    r = kl_ref(np.zeros((1, 1, 4)), zd, 1.0, KIND_REVERSE)
    assert np.isfinite(f["per_step"]).all() and np.isfinite(r["per_step"]).all()
    assert np.all(np.isfinite(r["grad"]))
    np.testing.assert_allclose(f["per_step"][0, 0], stats.entropy([0, 1 / 3, 1 / 3, 1 / 3], [0.25] * 4), rtol=1e-13)


def _case_dominant_1e8(rng):
    # one token holding all but about 4e-10 of both distributions
    V = 64
    zt = rng.normal(0.0, 1.0, size=(1, 1, V))
    zt[0, 0, 17] = 16.0
    zd = zt + rng.normal(0.0, 0.3, size=(1, 1, V))
    zd[0, 0, 17] = zt[0, 0, 17] + 0.4
    return zt, zd, 0.7


def _case_dominant_1e14(rng):
    # all but about 1e-14 on one token, the draft's top logit shifted
    V = 1024
    zt = rng.normal(0.0, 4.0, size=(1, 1, V))
    zt[0, 0, 300] = zt.max() + 19.0
    zd = zt + rng.normal(0.0, 1.3, size=(1, 1, V))
    zd[0, 0, 300] = zd.max() + 18.0
    return zt, zd, 0.6


def _case_two_tokens_shifted(rng):
    # two tokens sharing the mass (about 0.6 / 0.4); the draft's logits of
    # both are the target's plus one constant, the rest are noise far below:
    # q - p of the two is the small difference of the log partition sums
    V = 1024
    zt = rng.normal(0.0, 3.0, size=(1, 1, V))
    zd = zt + rng.normal(0.0, 1.8, size=(1, 1, V))
    top = zt.max()
    zt[0, 0, 668] = top + 12.0
    zt[0, 0, 281] = top + 11.75
    zd[0, 0, 668] = zt[0, 0, 668] + 0.875
    zd[0, 0, 281] = zt[0, 0, 281] + 0.875
    return zt, zd, 0.53


def _case_equal_log_ratios_far_below_target(rng):
    # the draft holds nearly all its mass on two tokens (q about 1 and
    # e^-12) whose log ratios log q - log p agree exactly, both rated about
    # e^-50 below the target's largest: log q - log p - L of the second token
    # is a difference of two numbers near 53 that agree to about 1e-19
    V = 1024
    zt = rng.normal(0.0, 2.0, size=(1, 1, V))
    zd = rng.normal(0.0, 2.0, size=(1, 1, V))
    zt[0, 0, 100], zd[0, 0, 100] = -20.0, 30.0
    zt[0, 0, 700], zd[0, 0, 700] = -26.0, 24.0
    return zt, zd, 0.5


@pytest.mark.parametrize("case", [_case_dominant_1e8, _case_dominant_1e14, _case_two_tokens_shifted,
                                  _case_equal_log_ratios_far_below_target])
def test_near_coincident_gradients_against_50_digit_arithmetic(case):
    """Rows where the gradient is a small difference of nearly equal
    quantities: one token holding all but 4e-10 or 1e-14 of both
    distributions ((q - p) / T of that token is a difference of two numbers
    that close to 1), and two tokens sharing the mass with the draft's two
    logits shifted by one constant (log q - log p of each is the small
    difference of the two log partition functions), and two draft tokens
    whose log ratios agree exactly, far below the target's mass (reverse KL's
    log q - log p - L of the lesser one cancels to 1e-19).  The oracle's forward-KL
    and reverse-KL gradients equal an evaluation in 50-digit arithmetic
    (mpmath), element by element, to 1e-9 of the row's largest gradient."""
    mpmath = pytest.importorskip("mpmath")
    mpmath.mp.dps = 50
    zt, zd, T = case(np.random.default_rng(5))
    for kind in (KIND_FORWARD, KIND_REVERSE):
        g = kl_ref(zt, zd, T, kind)["grad"][0, 0]
        a = [mpmath.mpf(float(x)) / mpmath.mpf(T) for x in zt[0, 0]]
        b = [mpmath.mpf(float(x)) / mpmath.mpf(T) for x in zd[0, 0]]
        la = mpmath.log(mpmath.fsum(mpmath.exp(x) for x in a))
        lb = mpmath.log(mpmath.fsum(mpmath.exp(x) for x in b))
        lp = [x - la for x in a]
        lq = [x - lb for x in b]
        q = [mpmath.exp(x) for x in lq]
        if kind == KIND_FORWARD:
            exact = [(mpmath.exp(y) - mpmath.exp(x)) / mpmath.mpf(T) for x, y in zip(lp, lq)]
        else:
            L = mpmath.fsum(qi * (y - x) for qi, x, y in zip(q, lp, lq))
            exact = [qi * (y - x - L) / mpmath.mpf(T) for qi, x, y in zip(q, lp, lq)]
        exact = np.array([float(e) for e in exact])
        scale = np.abs(exact).max()
        assert np.abs(g - exact).max() <= 1e-9 * scale, (kind, np.abs(g - exact).max() / scale)
