"""Pins of the oracle's target-only verification, draft-stage sampler and
per-step diagnostics against what the paper and the mathematics fix: the
reduction of target-only verification to rejection sampling with a
point-mass draft, unbiasedness (chi-square), acceptance statistics, numpy's
Philox, scipy's softmax / logsumexp / entropy, the TV identity and the
decision boundary of App. E, brute force on tiny vocabularies, and special
cases."""

import numpy as np
import pytest
from numpy.random import Philox
from scipy import special, stats

from oracle import verify_ref
from oracle.variants import (DIAG_COLUMNS, diagnostics_ref, sample_ref, sampler_words,
                             verify_target_only_ref)
from paper_2606_12370_amd import workloads as W


def _chisq(counts, probs):
    probs = np.asarray(probs, dtype=np.float64)
    keep = probs > 0
    assert counts[~keep].sum() == 0
    exp = probs[keep] / probs[keep].sum() * counts.sum()
    return stats.chisquare(counts[keep], exp).pvalue


def _logits(p):
    with np.errstate(divide="ignore"):
        return np.log(np.asarray(p, dtype=np.float64))


def _shared(rows, B):
    z = np.asarray(rows, dtype=np.float64)
    return np.broadcast_to(z, (B,) + z.shape)


# ----------------------------------------------------------------------------
# target-only verification (Sec. 2.2, Eq. target_only)

@pytest.mark.parametrize("gen,K,V,seed", [("rollout", 3, 700, 41), ("rollout_t", 2, 1500, 42), ("tiny", 1, 64, 43)])
def test_target_only_is_rejection_sampling_with_point_mass_draft(gen, K, V, seed):
    """With q_i = delta(x_i) the rejection test u q(x) < p(x) becomes u < p(x)
    and the residual max(0, p - q) is p with x removed: the rejection-sampling
    oracle on point-mass drafts must give the same outcome, bit for bit."""
    d = W.verify_inputs_numpy(24, K, V, W.F32, gen, seed)
    ids = W.greedy_ids(d["draft"], W.F32)
    zd = np.full((24, K, V), -np.inf)
    np.put_along_axis(zd, ids[..., None].astype(np.int64), 0.0, axis=-1)
    for s in (0, 5, 123456789):
        to = verify_target_only_ref(d["target"], ids, d["temperature"], s, 3)
        rs = verify_ref(d["target"], zd, ids, d["temperature"], s, 3)
        for k in ("accept_len", "emitted", "p_at_draft", "logz_target", "u_accept", "u_resample"):
            np.testing.assert_array_equal(to[k], rs[k], err_msg=k)
        assert np.all(rs["q_at_draft"] == 1.0)


def test_target_only_first_token_is_distributed_as_target():
    rng = np.random.default_rng(50)
    B, V = 60000, 8
    p0, p1 = rng.dirichlet(np.full(V, 0.8)), rng.dirichlet(np.full(V, 0.8))
    x = int(np.argsort(p0)[-2])                       # the draft's greedy token, not the target's top-1
    ids = np.full((B, 1), x, np.int32)
    out = verify_target_only_ref(_shared([_logits(p0), _logits(p1)], B), ids, 1.0, 9)
    assert _chisq(np.bincount(out["emitted"][:, 0], minlength=V), p0) > 1e-3
    acc = out["accept_len"] == 1
    assert _chisq(np.bincount(out["emitted"][acc, 1], minlength=V), p1) > 1e-3
    # given a rejection the token is never x and follows p restricted to v != x
    rej = out["emitted"][~acc, 0]
    assert np.all(rej != x)
    r = p0.copy()
    r[x] = 0.0
    assert _chisq(np.bincount(rej, minlength=V), r) > 1e-3


def test_target_only_acceptance_rate_is_p_of_greedy_token():
    rng = np.random.default_rng(51)
    B, V, K = 40000, 12, 3
    P = [rng.dirichlet(np.full(V, 0.6)) for _ in range(K + 1)]
    x = [int(rng.integers(V)) for _ in range(K)]
    ids = np.tile(np.array(x, np.int32), (B, 1))
    out = verify_target_only_ref(_shared([_logits(pi) for pi in P], B), ids, 1.0, 10)
    a = np.array([P[i][x[i]] for i in range(K)])
    rate = np.mean(out["accept_len"] >= 1)
    assert abs(rate - a[0]) < 5 * np.sqrt(a[0] * (1 - a[0]) / B)
    n = out["accept_len"].astype(np.float64)
    expect = sum(np.prod(a[: j + 1]) for j in range(K))
    assert abs(n.mean() - expect) < 5 * n.std() / np.sqrt(B), (n.mean(), expect)
    np.testing.assert_allclose(out["p_at_draft"][0], a, rtol=1e-13)


def test_target_only_special_cases():
    V = 10
    one_hot = np.full(V, -np.inf)
    one_hot[3] = 0.0
    flat = np.zeros(V)
    zero_at_3 = np.zeros(V)
    zero_at_3[3] = -np.inf
    B = 500
    # p(x) = 1 at every step: every draft accepted, the bonus comes from p_K
    out = verify_target_only_ref(_shared([one_hot, one_hot, one_hot], B), np.full((B, 2), 3, np.int32), 1.0, 1)
    assert np.all(out["accept_len"] == 2) and np.all(out["emitted"] == 3)
    # p(x) = 0: always rejected at step 0, never re-emitted
    out = verify_target_only_ref(_shared([zero_at_3, flat], B), np.full((B, 1), 3, np.int32), 1.0, 2)
    assert np.all(out["accept_len"] == 0)
    assert np.all(out["emitted"][:, 0] != 3) and np.all(out["emitted"][:, 1] == -1)
    assert np.all(out["p_at_draft"] == 0.0)
    # V = 1: the only token has p = 1
    out = verify_target_only_ref(np.zeros((4, 3, 1)), np.zeros((4, 2), np.int32), 0.7, 3)
    assert np.all(out["accept_len"] == 2) and np.all(out["emitted"] == 0)


def test_target_only_row_errors():
    d = W.verify_inputs_numpy(6, 2, 50, W.F32, "tiny", 44)
    ids = W.greedy_ids(d["draft"], W.F32)
    zt = d["target"].astype(np.float64)
    T = d["temperature"].astype(np.float64)
    zt[0, 1, 7] = np.nan
    zt[1, 2, :] = -np.inf
    ids[2, 1] = 50
    T[3] = 0.0
    zt[4, 0, 0] = np.inf
    out = verify_target_only_ref(zt, ids, T, 0)
    assert list(out["row_error"]) == [True, True, True, True, True, False]
    assert np.all(out["accept_len"][:5] == -1) and np.all(out["emitted"][:5] == -1)
    assert np.all(np.isnan(out["p_at_draft"][:5]))
    assert out["accept_len"][5] >= 0


# ----------------------------------------------------------------------------
# draft-stage sampler (App. G.1, draft stage)

def test_sampler_stream_is_philox_with_word3_one():
    seed, off = 987654321, 17
    rows = np.array([0, 1, 5, 1000])
    w = sampler_words(seed, rows, off)
    for a, r in enumerate(rows):
        c = int(r) + (off << 128) + (1 << 192)
        ref = Philox(counter=c - 1, key=seed).random_raw(4)
        assert [int(v) for v in w[a]] == [int(v) for v in ref]
    out = sample_ref(np.zeros((4, 3)), 1.0, seed, off, rows=rows)
    np.testing.assert_array_equal(out["u"], (w[:, 0] >> np.uint64(40)).astype(np.float64) * 2.0 ** -24)


def test_sampler_is_inverse_cdf_of_scipy_softmax():
    rng = np.random.default_rng(60)
    z = rng.normal(0, 3, size=(40, 257))
    z[:, :5] = -np.inf
    T = rng.uniform(0.5, 1.5, size=40)
    out = sample_ref(z, T, 3, 1)
    p = special.softmax(z / T[:, None], axis=-1)
    for r in range(40):
        assert out["token"][r] == np.searchsorted(np.cumsum(p[r]), out["u"][r], side="right")
    np.testing.assert_allclose(out["logz"], special.logsumexp(z / T[:, None], axis=-1), rtol=1e-13)
    assert np.all(out["token"] >= 5)


def test_sampler_frequencies_follow_softmax():
    B, V, T = 50000, 9, 0.8
    z = np.linspace(-2.0, 1.5, V)
    z[4] = -np.inf
    out = sample_ref(_shared(z, B), T, 21)
    assert _chisq(np.bincount(out["token"], minlength=V), special.softmax(z / T)) > 1e-3


def test_sampler_greedy_rows_and_errors():
    z = np.array([[1.0, 3.0, 3.0, 2.0],
                  [-np.inf, -5.0, -5.0, -np.inf],
                  [0.0, 0.0, 0.0, 0.0],
                  [1.0, np.nan, 0.0, 0.0],
                  [-np.inf] * 4,
                  [0.0, 1.0, 2.0, 3.0],
                  [0.0, 1.0, 2.0, 3.0],
                  [0.0, np.inf, 2.0, 3.0]])
    T = np.array([0.0, 0.0, 0.0, 1.0, 1.0, -1.0, np.inf, 0.0])
    out = sample_ref(z, T, 0)
    assert list(out["token"]) == [1, 1, 0, -1, -1, -1, -1, -1]
    assert np.all(np.isnan(out["logz"][:3]))
    # a very low temperature concentrates all mass on the maximum
    zz = np.array([[0.0, 1.0, 0.5, 0.99]])
    assert sample_ref(np.repeat(zz, 64, 0), 1e-3, 4)["token"].tolist() == [1] * 64


# ----------------------------------------------------------------------------
# per-step diagnostics (Sec. 3, App. E)

def _brute_alphas(p, q):
    gt = ge = 0.0
    for v in range(len(p)):
        if p[v] > q[v]:
            gt += q[v]
        else:
            ge += p[v]
    return gt, ge


def test_diagnostics_against_scipy_and_brute_force():
    rng = np.random.default_rng(70)
    R, K, V = 5, 3, 40
    zt = rng.normal(0, 2, size=(R, K + 1, V))
    zd = zt[:, :K] + rng.normal(0, 1, size=(R, K, V))
    zt[0, 0, :3] = -np.inf
    T = rng.uniform(0.6, 1.4, size=R)
    out = diagnostics_ref(zt, zd, T)
    for r in range(R):
        for i in range(K):
            p = special.softmax(zt[r, i] / T[r])
            q = special.softmax(zd[r, i] / T[r])
            np.testing.assert_allclose(out["entropy_target"][r, i], stats.entropy(p), rtol=1e-12)
            np.testing.assert_allclose(out["entropy_draft"][r, i], stats.entropy(q), rtol=1e-12)
            np.testing.assert_allclose(out["max_p"][r, i], p.max(), rtol=1e-13)
            # App. E: alpha^RS = 1 - d_TV with d_TV = half the L1 distance
            np.testing.assert_allclose(out["alpha_rs"][r, i], 1 - 0.5 * np.abs(p - q).sum(), rtol=1e-12)
            g = max(range(V), key=lambda v: (zd[r, i, v], -v))
            assert out["greedy_draft"][r, i] == g
            np.testing.assert_allclose(out["alpha_to"][r, i], p[g], rtol=1e-13)
            gt, ge = _brute_alphas(p, q)
            np.testing.assert_allclose(out["alpha_p_gt_q"][r, i], gt, rtol=1e-12, atol=1e-15)
            np.testing.assert_allclose(out["alpha_q_ge_p"][r, i], ge, rtol=1e-12, atol=1e-15)
            dtv = 0.5 * np.abs(p - q).sum()
            assert out["rs_preferred"][r, i] == (dtv < 1 - p[g])
    np.testing.assert_allclose(out["alpha_p_gt_q"] + out["alpha_q_ge_p"], out["alpha_rs"], rtol=1e-13)


def test_diagnostics_entropy_bound_and_special_cases():
    rng = np.random.default_rng(71)
    V = 64
    z = rng.normal(0, 3, size=(200, 1, V))
    out = diagnostics_ref(z, z + rng.normal(0, 1, size=z.shape), 1.0)
    # Prop. to_entropy: max p >= exp(-H(p))
    assert np.all(out["max_p"] >= np.exp(-out["entropy_target"]) * (1 - 1e-12))
    # uniform p: equality, H = log V
    flat = diagnostics_ref(np.zeros((1, 1, V)), np.arange(V, dtype=np.float64)[None, None], 1.0)
    np.testing.assert_allclose(flat["entropy_target"], np.log(V), rtol=1e-14)
    np.testing.assert_allclose(flat["max_p"], np.exp(-flat["entropy_target"]), rtol=1e-13)
    assert flat["greedy_draft"][0, 0] == V - 1
    # q = p: full overlap, nothing where p > q
    same = diagnostics_ref(z[:3], z[:3], 0.9)
    np.testing.assert_allclose(same["alpha_rs"], 1.0, rtol=1e-13)
    assert np.all(same["alpha_p_gt_q"] == 0.0)
    assert np.all(same["rs_preferred"] == (same["max_p"] < 1.0))
    # target one-hot on the draft's greedy token: target-only accepts surely
    zt = np.full((1, 1, 5), -np.inf)
    zt[0, 0, 2] = 0.0
    oh = diagnostics_ref(zt, np.array([[[0.0, 0.5, 2.0, 1.0, 0.0]]]), 1.0)
    assert oh["alpha_to"][0, 0] == 1.0 and not oh["rs_preferred"][0, 0]
    assert oh["entropy_target"][0, 0] == 0.0
    # App. E's inequality is strict: at alpha^RS = alpha^TO (here both 1/2) RS is not preferred
    eq = diagnostics_ref(np.zeros((1, 1, 2)), np.array([[[0.0, -np.inf]]]), 1.0)
    assert eq["alpha_rs"][0, 0] == 0.5 and eq["alpha_to"][0, 0] == 0.5 and not eq["rs_preferred"][0, 0]
    # greedy ties go to the first index
    tie = diagnostics_ref(np.zeros((1, 1, 4)), np.array([[[0.0, 2.0, 2.0, 1.0]]]), 1.0)
    assert tie["greedy_draft"][0, 0] == 1


def test_diagnostics_match_simulated_acceptance():
    """alpha^RS and alpha^TO are the acceptance rates of the two verification
    procedures: simulate both with one shared (p, q) and compare."""
    rng = np.random.default_rng(72)
    B, V = 40000, 16
    p, q = rng.dirichlet(np.full(V, 0.7)), rng.dirichlet(np.full(V, 0.7))
    zt, zd = _shared([_logits(p), _logits(p)], B), _shared([_logits(q)], B)
    dg = diagnostics_ref(zt[:1], zd[:1], 1.0)
    ids_rs = rng.choice(V, size=(B, 1), p=q).astype(np.int32)
    rs = verify_ref(zt, zd, ids_rs, 1.0, 31)
    ids_to = np.full((B, 1), dg["greedy_draft"][0, 0], np.int32)
    to = verify_target_only_ref(zt, ids_to, 1.0, 32)
    for out, a in ((rs, dg["alpha_rs"][0, 0]), (to, dg["alpha_to"][0, 0])):
        rate = np.mean(out["accept_len"] == 1)
        assert abs(rate - a) < 5 * np.sqrt(a * (1 - a) / B), (rate, a)


def test_diagnostics_tie_mass_and_row_errors():
    z = np.zeros((3, 1, 6))
    zd = np.zeros((3, 1, 6))
    zd[:, 0, 0] = 1.0
    zd[1, 0, 2] = np.nan
    out = diagnostics_ref(z, zd, np.array([1.0, 1.0, -1.0]))
    assert list(out["row_error"]) == [False, True, True]
    assert np.all(np.isnan(out["alpha_rs"][1:])) and np.all(out["greedy_draft"][1:] == -1)
    # tokens 1..5 have equal p and equal q but p != q; no tie
    assert out["tie_mass"][0, 0] == 0.0
    exact = diagnostics_ref(z[:1], z[:1], 1.0)
    np.testing.assert_allclose(exact["tie_mass"], 1.0, rtol=1e-14)
    assert set(DIAG_COLUMNS) <= set(out)
