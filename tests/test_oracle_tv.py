"""Pins of the TV-loss oracle: central finite differences of its own loss
(pins the gradient formula and the chain rule of every mode), the invariants
the paper proves (bounded gradient, zero row sum, q = p stationary point),
closed forms of the multi-step losses and hand-worked fixtures."""

import json
import os

import numpy as np
import pytest

from oracle import tv_ref
from oracle.tv import MODE_E2E, MODE_PER_STEP, MODE_PROD, chain_factors
from paper_2606_12370_amd import workloads as W

MODES = [MODE_E2E, MODE_PROD, MODE_PER_STEP]


def random_logits(rng, N, K, V, scale=2.0):
    zt = rng.normal(0, scale, size=(N, K, V))
    zd = zt + rng.normal(0, 0.8, size=(N, K, V))
    return zt, zd


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("K", [1, 2, 3])
@pytest.mark.parametrize("T", [1.0, 0.7])
def test_gradient_matches_finite_differences(mode, K, T):
    rng = np.random.default_rng(100 + 10 * mode + K)
    N, V = 2, 13
    zt, zd = random_logits(rng, N, K, V)
    out = tv_ref(zt, zd, T, mode, scale=0.5)
    # a perturbation of h moves log q - log p by at most 2h/T: stay off the kink
    assert np.min(out["tie_margin"]) > 20 * 1e-6
    h = 1e-6
    fd = np.zeros_like(zd)
    for idx in np.ndindex(zd.shape):
        zp = zd.copy()
        zm = zd.copy()
        zp[idx] += h
        zm[idx] -= h
        fd[idx] = (tv_ref(zt, zp, T, mode, 0.5, False)["loss"]
                   - tv_ref(zt, zm, T, mode, 0.5, False)["loss"]) / (2 * h)
    np.testing.assert_allclose(out["grad"], fd, rtol=1e-6, atol=1e-9)


def test_gradient_row_sum_and_bound():
    rng = np.random.default_rng(1)
    zt, zd = random_logits(rng, 5, 3, 400, scale=4.0)
    for mode in MODES:
        for T in (0.6, 1.0, 1.3):
            out = tv_ref(zt, zd, T, mode)
            g = out["grad"]
            np.testing.assert_allclose(g.sum(axis=-1), 0.0, atol=1e-15)
            q = np.exp(zd / T - out["logz_draft"][..., None])
            bound = np.abs(out["g"])[..., None] * q / T
            assert np.all(np.abs(g) <= bound * (1 + 1e-12) + 1e-300)


def test_q_equals_p_is_stationary():
    rng = np.random.default_rng(2)
    zt = rng.normal(0, 3, size=(3, 2, 200))
    for mode in MODES:
        out = tv_ref(zt, zt.copy(), 1.0, mode)
        np.testing.assert_allclose(out["overlap"], 1.0, atol=1e-13)
        np.testing.assert_allclose(out["S"], 1.0, atol=1e-13)
        assert np.max(np.abs(out["grad"])) < 1e-14  # 1 - S is a rounding residue only


def test_single_step_losses_are_tv():
    rng = np.random.default_rng(3)
    zt, zd = random_logits(rng, 4, 1, 300)
    p = np.exp(zt - np.log(np.exp(zt).sum(-1, keepdims=True)))
    q = np.exp(zd - np.log(np.exp(zd).sum(-1, keepdims=True)))
    tv = 0.5 * np.abs(p - q).sum(-1)[:, 0]
    np.testing.assert_allclose(tv_ref(zt, zd, 1.0, MODE_E2E)["loss_per_position"], tv, atol=1e-13)
    np.testing.assert_allclose(tv_ref(zt, zd, 1.0, MODE_PER_STEP)["loss_per_position"], tv, atol=1e-13)
    np.testing.assert_allclose(tv_ref(zt, zd, 1.0, MODE_PROD)["loss_per_position"], tv - 1.0, atol=1e-13)


def test_e2e_loss_is_one_minus_normalised_acceptance_length():
    rng = np.random.default_rng(4)
    zt, zd = random_logits(rng, 6, 3, 100)
    out = tv_ref(zt, zd, 1.0, MODE_E2E)
    a = out["overlap"]
    EL = a[:, 0] + a[:, 0] * a[:, 1] + a[:, 0] * a[:, 1] * a[:, 2]
    np.testing.assert_allclose(out["loss_per_position"], 1.0 - EL / 3.0, atol=1e-14)


def test_chain_factors_with_zero_alpha():
    alpha = np.array([[0.0, 0.5, 0.25], [0.3, 0.0, 0.0]])
    g, L = chain_factors(alpha, MODE_PROD)
    np.testing.assert_allclose(g, [[-0.125, 0.0, 0.0], [0.0, 0.0, 0.0]])
    g, L = chain_factors(alpha, MODE_E2E)
    # d/d a0 of 1 - (a0 + a0 a1 + a0 a1 a2)/3 = -(1 + a1 + a1 a2)/3
    np.testing.assert_allclose(g[0], [-(1 + 0.5 + 0.125) / 3, 0.0, 0.0])
    np.testing.assert_allclose(L, [1.0, 1.0 - 0.3 / 3])


def test_golden_closed_form(golden_dir):
    gld = json.load(open(os.path.join(golden_dir, "tv_closed_form_v3.json")))
    p = np.array(gld["target_probs"])
    q = np.array(gld["draft_probs"])
    e = gld["expected"]
    out = tv_ref(np.log(p)[None, None], np.log(q)[None, None], 1.0, MODE_PER_STEP)
    assert abs(out["overlap"][0, 0] - e["alpha"]) < 1e-12
    assert abs(out["S"][0, 0] - e["S"]) < 1e-12
    # PER_STEP with K = 1: g = -1, so grad = -d alpha / dz
    np.testing.assert_allclose(-out["grad"][0, 0], e["d_alpha_d_zdraft"], atol=1e-12)
    ms = gld["multi_step"]
    a = np.array([ms["alphas"]])
    for mode, lk, gk in ((MODE_E2E, "e2e_loss", "e2e_chain"), (MODE_PROD, "prod_loss", "prod_chain"),
                         (MODE_PER_STEP, "per_step_loss", "per_step_chain")):
        g, L = chain_factors(a, mode)
        assert abs(L[0] - ms[lk]) < 1e-12
        np.testing.assert_allclose(g[0], ms[gk], atol=1e-12)
    al = gld["acceptance_length"]
    a = np.array([al["alphas"]])
    _, L = chain_factors(a, MODE_E2E)
    assert abs((1.0 - L[0]) * 3 - al["expected_length"]) < 1e-12


def test_tiled_passes_match_untiled():
    """The two-pass, BLOCK_V-tiled organisation of the fused kernels (App. F,
    Alg. tv_fwd / tv_bwd: max and exp-sum first, then per-tile overlap and S,
    then the per-tile gradient q (S - 1 + 1[q > p]) g) gives the same
    numbers as the whole-vector oracle."""
    rng = np.random.default_rng(5)
    zt, zd = random_logits(rng, 1, 1, 1000)
    out = tv_ref(zt, zd, 1.0, MODE_PER_STEP)
    z, lp = zd[0, 0], zt[0, 0] - np.log(np.exp(zt[0, 0]).sum())
    m = z.max()
    D = np.exp(z - m).sum()
    overlap = S = 0.0
    BV = 128
    for s in range(0, z.size, BV):
        qq = np.exp(z[s:s + BV] - m) / D
        pp = np.exp(lp[s:s + BV])
        overlap += np.minimum(qq, pp).sum()
        S += (qq * (qq <= pp)).sum()
    assert abs(overlap - out["overlap"][0, 0]) < 1e-13 and abs(S - out["S"][0, 0]) < 1e-13
    gout = out["g"][0, 0]
    grad = np.concatenate([
        (np.exp(z[s:s + BV] - m) / D) * (S - 1 + (np.exp(z[s:s + BV] - m) / D > np.exp(lp[s:s + BV]))) * gout
        for s in range(0, z.size, BV)])
    # Alg. tv_bwd differentiates L_TV = 1 - alpha; the oracle's g already holds d L / d alpha
    np.testing.assert_allclose(-grad, out["grad"][0, 0], atol=1e-15)


def test_bf16_workload_shapes():
    d = W.tv_inputs_numpy(3, 3, 4096, W.BF16, 5)
    zt = W.to_float64(d["target"], W.BF16)
    zd = W.to_float64(d["draft"], W.BF16)
    out = tv_ref(zt, zd, 1.0, MODE_PROD)
    assert out["grad"].shape == (3, 3, 4096) and np.all(np.isfinite(out["grad"]))
    assert np.all((out["overlap"] > 0) & (out["overlap"] < 1))
