"""The TV comparison used by the GPU tests accepts exactly the freedom the
method leaves and nothing more.

At an element with p = q the TV integrand min(p, q) has a kink; either
indicator value gives a valid subgradient and moves S = sum 1[q <= p] q by that
element's mass.  Two oracle evaluations on each side of a planted heavy tie
must pass the comparison although every gradient element of the row differs,
while planted mistakes (a sign, a dropped S term, one wrong element, an S shift
beyond the tied mass, an S error of 1e-3 in rows without ties, a wrong loss)
must fail it."""

import numpy as np
import pytest
import torch

from oracle import tv_ref
from oracle.tv import MODE_E2E, MODE_PER_STEP, MODE_PROD
from paper_2606_12370_amd import workloads as W
from tests.parity import compare_tv

T = 0.8


def tied_logits(seed, N=2, K=2, V=24):
    """Random logits with element j0 of row (0, 0) tied (p = q) and heavy."""
    rng = np.random.default_rng(seed)
    zd = rng.normal(0, 1.5, size=(N, K, V))
    zt = zd + rng.normal(0, 0.7, size=(N, K, V))
    j0 = 5
    zd[0, 0, j0] += 6.0
    q = np.exp(zd[0, 0] / T - np.logaddexp.reduce(zd[0, 0] / T))
    rest = np.delete(zt[0, 0] / T, j0)
    # p_j0 = e / (e + A) equals q_j0 when e = q_j0 A / (1 - q_j0)
    zt[0, 0, j0] = T * (np.log(q[j0]) - np.log1p(-q[j0]) + np.logaddexp.reduce(rest))
    return zt, zd, j0, q[j0]


def as_gpu(ref, grad=None, loss=None):
    return (torch.tensor([ref["loss"] if loss is None else loss]),
            torch.tensor(ref["overlap"]),
            torch.tensor(ref["grad"] if grad is None else grad))


@pytest.mark.parametrize("mode", [MODE_E2E, MODE_PROD, MODE_PER_STEP])
def test_either_side_of_a_heavy_tie_is_accepted(mode):
    zt, zd, j0, qj = tied_logits(1 + mode)
    assert qj > 0.3
    eps = 1e-9
    above, below = zt.copy(), zt.copy()
    above[0, 0, j0] += eps
    below[0, 0, j0] -= eps
    ra = tv_ref(above, zd, T, mode, scale=0.7)
    rb = tv_ref(below, zd, T, mode, scale=0.7)
    assert ra["tie_margin"][0, 0, j0] <= 1e-6
    # the two sides really differ: S moves by q_j0 and so does every element
    assert abs(ra["S"][0, 0] - rb["S"][0, 0]) > 0.9 * qj
    assert np.abs(ra["grad"][0, 0] - rb["grad"][0, 0]).max() > 1e-2 * np.abs(ra["grad"][0, 0]).max()
    rep = compare_tv(*as_gpu(rb), ra, W.F32)
    assert rep["rows_with_shifted_S"] >= 1
    compare_tv(*as_gpu(ra), rb, W.F32)


def test_planted_mistakes_are_rejected():
    zt, zd, j0, qj = tied_logits(7)
    ref = tv_ref(zt, zd, T, MODE_E2E, scale=0.7)
    compare_tv(*as_gpu(ref), ref, W.F32)
    g = ref["grad"]
    w = ref["grad_weight"]
    untied_rows = np.ones(g.shape[:2], dtype=bool)
    untied_rows[0, 0] = False
    ind = np.where(ref["grad_weight"] != 0, g / np.where(w != 0, w, 1) + ref["S"][..., None], 0)
    bad = {
        "sign": -g,
        "dropped S": w * ind,
        "one element": g + np.where(np.arange(g.shape[-1]) == 3, 0.1 * np.abs(g).max(), 0.0),
        "S beyond tied mass": g - w * (2.5 * qj),
        "S off by 1e-3 in the untied rows": g - np.where(untied_rows[..., None], w * 1e-3, 0.0),
    }
    for name, gb in bad.items():
        with pytest.raises(AssertionError):
            compare_tv(*as_gpu(ref, grad=gb), ref, W.F32)
            pytest.fail("accepted: " + name)


def test_loss_floor_near_zero_and_relative_elsewhere():
    rng = np.random.default_rng(3)
    z = rng.normal(0, 1, size=(2, 3, 16))
    ref0 = tv_ref(z, z, 1.0, MODE_E2E, scale=1.0)
    assert ref0["loss"] < 1e-12
    compare_tv(*as_gpu(ref0, loss=3e-7), ref0, W.F32)
    with pytest.raises(AssertionError):
        compare_tv(*as_gpu(ref0, loss=1e-4), ref0, W.F32)
    zt, zd, _, _ = tied_logits(4)
    ref = tv_ref(zt, zd, T, MODE_E2E, scale=1.0)
    with pytest.raises(AssertionError):
        compare_tv(*as_gpu(ref, loss=ref["loss"] * (1 + 1e-3)), ref, W.F32)



def dominant_tie_logits(seed, N=2, K=2, V=24, m=1e-7, delta=1e-4):
    """Logits whose row (0, 0) has q_0 = p_0 = 1 - m (a tie) and all but
    delta m of the other mass on tokens with p = q (1 - delta); the last
    three tokens, holding delta m of q, take the surplus of p, so they alone
    have q < p and S = sum 1[q <= p] q off the tie is delta m.  The other
    rows are random."""
    rng = np.random.default_rng(seed)
    zd = rng.normal(0, 1.5, size=(N, K, V))
    zt = zd + rng.normal(0, 0.7, size=(N, K, V))
    q = np.empty(V)
    q[0] = 1 - m
    big = rng.uniform(0.5, 1.5, size=V - 4)
    big *= (1 - delta) * m / big.sum()
    q[1:V - 3] = big
    q[V - 3:] = (m - big.sum()) / 3
    p = q.copy()
    p[1:V - 3] *= 1 - delta
    p[V - 3:] += delta * big.sum() / 3
    assert abs(p.sum() - 1) < 1e-15
    zd[0, 0] = T * np.log(q)
    zt[0, 0] = T * np.log(p)
    return zt, zd, 0, 1 - m


def test_dominant_tied_token_with_float32_q_errors():
    """A tied token that holds all but 1e-7 of q: on the side of the tie that
    leaves it out of S the row's gradient is of the order of the small mass
    with q <= p, on the other of the q_j themselves.  The second side, with
    each q_j off by a relative error inside its float32 bound, is accepted
    against the first; one element off by 1e-3 of its own size is not."""
    zt, zd, j0, qj = dominant_tie_logits(11)
    # log p_j0 moves by (1 - p_j0) / T per unit of its logit and every other
    # log p_v by -p_j0 / T: a nudge that puts log q_j0 - log p_j0 at +-1e-13
    # moves the other ratios by 1e-6, well inside delta
    eps = 1e-13 * T / (1 - qj)
    above, below = zt.copy(), zt.copy()
    above[0, 0, j0] += eps
    below[0, 0, j0] -= eps
    for mode in (MODE_E2E, MODE_PER_STEP):
        ra = tv_ref(above, zd, T, mode, scale=1.0)
        rb = tv_ref(below, zd, T, mode, scale=1.0)
        assert ra["tie_margin"][0, 0, j0] < 1e-12 and rb["tie_margin"][0, 0, j0] < 1e-12
        small, large = (ra, rb) if ra["S"][0, 0] < rb["S"][0, 0] else (rb, ra)
        gs, gl = np.abs(small["grad"][0, 0]).max(), np.abs(large["grad"][0, 0]).max()
        assert gl > 30 * gs
        qerr = 2e-6 + 2.0 ** -22 * large["tie_condition"]
        rng = np.random.default_rng(5 + mode)
        noisy = large["grad"] * (1 + 0.5 * qerr * rng.uniform(-1, 1, size=qerr.shape))
        compare_tv(*as_gpu(large, grad=noisy), small, W.F32)
        compare_tv(*as_gpu(small, grad=small["grad"]), large, W.F32)
        bad = large["grad"].copy()
        v = int(np.argmax(np.where(np.arange(bad.shape[-1]) == j0, 0.0, np.abs(bad[0, 0]))))
        bad[0, 0, v] *= 1 + 1e-3
        with pytest.raises(AssertionError):
            compare_tv(*as_gpu(large, grad=bad), small, W.F32)
            pytest.fail("accepted an element off by 1e-3")
