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
