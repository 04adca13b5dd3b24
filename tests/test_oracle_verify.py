"""Pins of the verification oracle against what the paper and the
mathematics fix: library routines (scipy softmax / logsumexp, numpy
searchsorted), the TV identity, the unbiasedness theorem of speculative
sampling (chi-square tests and exact enumeration), acceptance statistics,
special cases and hand-worked fixtures."""

import json
import os

import numpy as np
import pytest
from scipy import special, stats

from oracle import verify_ref
from oracle.verify import inverse_cdf, residual_sample, softmax_t
from paper_2606_12370_amd import workloads as W


def logits_from_probs(p):
    p = np.asarray(p, dtype=np.float64)
    with np.errstate(divide="ignore"):
        return np.log(p)


def shared_batch(target_row_probs, draft_row_probs, B, rng, K=None):
    """B rows all sharing the same target [K+1, V] and draft [K, V]
    distributions, with draft ids x ~ q drawn independently per row."""
    zt = logits_from_probs(target_row_probs)
    zd = logits_from_probs(draft_row_probs)
    K = zd.shape[0]
    q = np.asarray(draft_row_probs, dtype=np.float64)
    ids = np.stack([rng.choice(q.shape[1], size=B, p=q[i] / q[i].sum()) for i in range(K)], axis=1)
    return (np.broadcast_to(zt, (B,) + zt.shape), np.broadcast_to(zd, (B,) + zd.shape),
            ids.astype(np.int32))


def random_probs(rng, V, conc=1.0):
    return rng.dirichlet(np.full(V, conc))


# ----------------------------------------------------------------------------
# library pins

def test_softmax_matches_scipy():
    rng = np.random.default_rng(0)
    z = rng.normal(0, 5, size=(6, 300))
    z[0, :10] = -np.inf
    for T in (0.6, 1.0, 1.7):
        p, lz = softmax_t(z, T)
        np.testing.assert_allclose(p, special.softmax(z / T, axis=-1), rtol=1e-13, atol=1e-300)
        np.testing.assert_allclose(lz, special.logsumexp(z / T, axis=-1), rtol=1e-13)


def test_inverse_cdf_matches_searchsorted():
    rng = np.random.default_rng(1)
    r = rng.random((50, 37)) * (rng.random((50, 37)) < 0.5)
    r[:, 0] += 1e-3
    t = rng.random(50) * r.sum(axis=1)
    idx, C = inverse_cdf(r, t)
    for i in range(50):
        assert idx[i] == np.searchsorted(C[i], t[i], side="right")
        assert r[i, idx[i]] > 0  # strict '>' never lands on a zero-mass token


# ----------------------------------------------------------------------------
# closed forms and identities

def test_overlap_is_one_minus_tv():
    rng = np.random.default_rng(2)
    d = W.verify_inputs_numpy(8, 3, 2048, W.F32, "tiny", 11)
    out = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 0)
    p, _ = softmax_t(d["target"].astype(np.float64)[:, :3], 1.0)
    q, _ = softmax_t(d["draft"].astype(np.float64), 1.0)
    tv = 0.5 * np.abs(p - q).sum(axis=-1)
    np.testing.assert_allclose(out["overlap"], 1.0 - tv, rtol=0, atol=1e-13)
    del rng


def test_residual_mass_is_one_minus_alpha():
    rng = np.random.default_rng(3)
    p = np.stack([random_probs(rng, 100) for _ in range(20)])
    q = np.stack([random_probs(rng, 100) for _ in range(20)])
    _, Z, _, zero = residual_sample(p, q, rng.random(20))
    assert not zero.any()
    np.testing.assert_allclose(Z, 1.0 - np.minimum(p, q).sum(axis=1), atol=1e-14)


def test_golden_ranking_flip(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "ranking_flip.json")))
    p, q, e = g["target_probs"], g["draft_probs"], g["expected"]
    zt = logits_from_probs([p, p])[None]
    zd = logits_from_probs([q])[None]
    out = verify_ref(zt, zd, np.array([[0]]), 1.0, 0)
    assert abs(out["overlap"][0, 0] - e["alpha_rs"]) < 1e-12
    assert abs(0.5 * np.abs(np.subtract(p, q)).sum() - e["tv_distance"]) < 1e-12
    top1_q = int(np.argmax(q))
    assert abs(q[top1_q] - e["alpha_to_before"]) < 1e-12
    assert abs(p[top1_q] - e["alpha_to_after"]) < 1e-12
    tv = 1.0 - out["overlap"][0, 0]
    assert abs((1.0 - p[top1_q]) - e["rs_boundary_rhs"]) < 1e-12
    assert (tv < 1.0 - p[top1_q]) == e["rs_preferred"]


def test_golden_closed_form(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "tv_closed_form_v3.json")))
    p = np.array(g["target_probs"])
    q = np.array(g["draft_probs"])
    e = g["expected"]
    out = verify_ref(logits_from_probs([p, p])[None], logits_from_probs([q])[None],
                     np.array([[2]]), 1.0, 0)
    assert abs(out["overlap"][0, 0] - e["alpha"]) < 1e-12
    for u, tok in e["inverse_cdf"]:
        y, Z, _, _ = residual_sample(p[None], q[None], np.array([u]))
        assert int(y[0]) == tok
        assert abs(Z[0] - e["residual_mass"]) < 1e-12


# ----------------------------------------------------------------------------
# special cases

def test_q_equals_p_accepts_every_draft():
    d = W.verify_inputs_numpy(65536, 1, 8, W.F32, "exact", 1002, q_equals_p=True)
    out = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 0)
    assert np.all(out["accept_len"] == 1)
    assert np.all(out["emitted"][:, 0] == d["ids"][:, 0])
    np.testing.assert_allclose(out["overlap"], 1.0, atol=1e-13)
    d = W.verify_inputs_numpy(16, 3, 1024, W.F32, "rollout", 5, q_equals_p=True)
    out = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 9)
    assert np.all(out["accept_len"] == 3)


def test_zero_target_probability_always_rejects():
    rng = np.random.default_rng(4)
    B, V = 64, 16
    q = random_probs(rng, V)
    p = random_probs(rng, V)
    p0 = p.copy()
    p0[5] = 0.0
    p0 /= p0.sum()
    zt, zd, ids = shared_batch([p0, p], [q], B, rng)
    ids = np.full_like(ids, 5)
    out = verify_ref(zt, zd, ids, 1.0, 1)
    assert np.all(out["accept_len"] == 0)
    assert np.all(out["emitted"][:, 0] != 5)


def test_draft_below_target_always_accepts():
    rng = np.random.default_rng(5)
    B, V = 256, 12
    p = random_probs(rng, V)
    q = random_probs(rng, V)
    zt, zd, ids = shared_batch([p, p], [q], B, rng)
    ok = q <= p
    out = verify_ref(zt, zd, ids, 1.0, 2)
    acc = out["accept_len"] == 1
    assert np.all(acc[ok[ids[:, 0]]])


def test_one_hot_bonus_and_v1():
    B, V = 32, 9
    zt = np.full((B, 2, V), -np.inf)
    zt[:, :, 4] = 0.0
    zd = zt[:, :1].copy()
    out = verify_ref(zt, zd, np.full((B, 1), 4), 1.0, 3)
    assert np.all(out["accept_len"] == 1) and np.all(out["emitted"] == 4)
    out = verify_ref(np.zeros((5, 3, 1)), np.zeros((5, 2, 1)), np.zeros((5, 2), int), 0.7, 4)
    assert np.all(out["accept_len"] == 2) and np.all(out["emitted"] == 0)


def test_row_errors():
    d = W.verify_inputs_numpy(6, 2, 64, W.F32, "tiny", 12)
    zt, zd = d["target"].astype(np.float64), d["draft"].astype(np.float64)
    ids, T = d["ids"].copy(), d["temperature"].astype(np.float64).copy()
    zt[0, 1, 3] = np.nan
    zd[1, 0, 0] = np.inf
    zt[2, 2, :] = -np.inf
    ids[3, 1] = 64
    T[4] = 0.0
    zt[5, 0, :10] = -np.inf  # legal: masked tokens
    out = verify_ref(zt, zd, ids, T, 0)
    assert list(out["row_error"]) == [True] * 5 + [False]
    assert np.all(out["accept_len"][:5] == -1) and np.all(out["emitted"][:5] == -1)
    assert np.all(np.isnan(out["overlap"][:5])) and out["accept_len"][5] >= 0


def test_rows_subset_and_determinism():
    d = W.verify_inputs_numpy(12, 3, 500, W.F32, "rollout", 13)
    full = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 77, 5)
    again = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 77, 5)
    sel = np.array([2, 7, 11])
    part = verify_ref(d["target"][sel], d["draft"][sel], d["ids"][sel], d["temperature"][sel],
                      77, 5, rows=sel)
    for k in ("accept_len", "emitted"):
        assert np.array_equal(full[k], again[k])
        assert np.array_equal(full[k][sel], part[k])
    other = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 77, 6)
    assert not np.array_equal(full["u_accept"], other["u_accept"])


# ----------------------------------------------------------------------------
# distributional pins (fixed seeds: deterministic pass/fail)

def test_step0_acceptance_is_alpha_binomial():
    rng = np.random.default_rng(6)
    B, V = 40000, 10
    p = random_probs(rng, V, 0.7)
    q = random_probs(rng, V, 0.7)
    zt, zd, ids = shared_batch([p, p], [q], B, rng)
    out = verify_ref(zt, zd, ids, 1.0, 5)
    alpha = np.minimum(p, q).sum()
    rate = np.mean(out["accept_len"] >= 1)
    sd = np.sqrt(alpha * (1 - alpha) / B)
    assert abs(rate - alpha) < 5 * sd, (rate, alpha, sd)


def test_mean_accept_length_is_sum_of_prefix_products():
    rng = np.random.default_rng(7)
    B, V, K = 40000, 10, 3
    P = [random_probs(rng, V, 0.8) for _ in range(K + 1)]
    Q = [random_probs(rng, V, 0.8) for _ in range(K)]
    zt, zd, ids = shared_batch(P, Q, B, rng)
    out = verify_ref(zt, zd, ids, 1.0, 6)
    a = [np.minimum(P[i], Q[i]).sum() for i in range(K)]
    expect = sum(np.prod(a[: j + 1]) for j in range(K))
    n = out["accept_len"].astype(np.float64)
    assert abs(n.mean() - expect) < 5 * n.std() / np.sqrt(B), (n.mean(), expect)


def _chisq(counts, probs):
    probs = np.asarray(probs, dtype=np.float64)
    keep = probs > 0
    assert counts[~keep].sum() == 0
    exp = probs[keep] / probs[keep].sum() * counts.sum()
    return stats.chisquare(counts[keep], exp).pvalue


def test_first_token_distribution_equals_target_shared():
    """65536 rows, V = 8, one shared target/draft pair: the first emitted
    token (accepted draft or residual resample) is distributed as p_0."""
    d = W.verify_inputs_numpy(65536, 1, 8, W.F32, "exact", 1002, shared_target=True)
    out = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 0)
    p0, _ = softmax_t(d["target"][0, 0].astype(np.float64), 1.0)
    counts = np.bincount(out["emitted"][:, 0], minlength=8)
    assert _chisq(counts, p0) > 1e-3


def test_first_token_distribution_per_row_targets():
    d = W.verify_inputs_numpy(65536, 1, 8, W.F32, "exact", 1002)
    out = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 0)
    p, _ = softmax_t(d["target"][:, 0].astype(np.float64), 1.0)
    counts = np.bincount(out["emitted"][:, 0], minlength=8)
    assert _chisq(counts, p.sum(axis=0)) > 1e-3


def test_bonus_and_residual_conditionals():
    rng = np.random.default_rng(8)
    B, V = 60000, 8
    p0, p1, q0 = random_probs(rng, V), random_probs(rng, V), random_probs(rng, V)
    zt, zd, ids = shared_batch([p0, p1], [q0], B, rng)
    out = verify_ref(zt, zd, ids, 1.0, 11)
    acc = out["accept_len"] == 1
    bonus = np.bincount(out["emitted"][acc, 1], minlength=V)
    assert _chisq(bonus, p1) > 1e-3
    rej = ~acc
    resid = np.maximum(0.0, p0 - q0)
    res = np.bincount(out["emitted"][rej, 0], minlength=V)
    assert _chisq(res, resid) > 1e-3


def test_exact_enumeration_of_emitted_distribution():
    """Brute force over every draft token x and both branches, with the
    accept probability counted on the 2^-24 uniform grid and the residual
    sample taken through the oracle's inverse CDF on a fine uniform grid:
    P(first emitted = v) must equal p(v) up to the grid resolution."""
    rng = np.random.default_rng(9)
    V = 6
    for _ in range(5):
        p, q = random_probs(rng, V), random_probs(rng, V)
        grid = (np.arange(1 << 12) + 0.5) / (1 << 12)
        tok, _, _, _ = residual_sample(np.broadcast_to(p, (grid.size, V)).copy(),
                                       np.broadcast_to(q, (grid.size, V)).copy(), grid)
        r_emp = np.bincount(tok, minlength=V) / grid.size
        prob = np.zeros(V)
        for x in range(V):
            # accept iff u * q(x) < p(x) with u = k 2^-24, k = 0 .. 2^24 - 1
            k_acc = min(1 << 24, int(np.ceil(p[x] / q[x] * (1 << 24))))
            a = k_acc / float(1 << 24)
            prob[x] += q[x] * a
            prob += q[x] * (1 - a) * r_emp
        np.testing.assert_allclose(prob, p, atol=4e-4)
        # and the exact identity with the continuous uniform (no grid)
        a = np.minimum(1.0, p / q)
        r = np.maximum(0, p - q) / np.maximum(0, p - q).sum()
        exact = q * a + (q * (1 - a)).sum() * r
        np.testing.assert_allclose(exact, p, atol=1e-12)


@pytest.mark.parametrize("T", [0.6, 1.2])
def test_temperature_enters_both_distributions(T):
    d = W.verify_inputs_numpy(4, 2, 300, W.F32, "tiny", 21)
    out = verify_ref(d["target"], d["draft"], d["ids"], T, 0)
    zt, zd = d["target"].astype(np.float64) / T, d["draft"].astype(np.float64) / T
    p, lzt = special.softmax(zt, axis=-1), special.logsumexp(zt, axis=-1)
    q, lzd = special.softmax(zd, axis=-1), special.logsumexp(zd, axis=-1)
    np.testing.assert_allclose(out["overlap"], np.minimum(p[:, :2], q).sum(-1), atol=1e-13)
    np.testing.assert_allclose(out["logz_target"], lzt, rtol=1e-13)
    np.testing.assert_allclose(out["logz_draft"], lzd, rtol=1e-13)


def test_inverse_cdf_strict_inequality_skips_zero_mass_prefix():
    r = np.array([[0.0, 0.0, 0.5, 0.5], [0.25, 0.0, 0.0, 0.75]])
    idx, _ = inverse_cdf(r, np.array([0.0, 0.25]))
    assert list(idx) == [2, 3]


def test_random_stream_definition():
    """u_i is U24 of word 0 of Philox((b, i, offset, 0); (seed, 0)) and the
    resample uniform is U24 of word 1 of the block at the emitting step n;
    checked against numpy's Philox."""
    from numpy.random import Philox
    d = W.verify_inputs_numpy(6, 3, 256, W.F32, "rollout", 31)
    seed, off = 1234567, 9
    rows = np.array([3, 10, 11, 12, 40, 41])
    out = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], seed, off, rows=rows)
    for a, b in enumerate(rows):
        for i in range(3):
            c = int(b) + (i << 64) + (off << 128)
            w = Philox(counter=c - 1, key=seed).random_raw(4)
            assert out["u_accept"][a, i] == (int(w[0]) >> 40) * 2.0 ** -24
        n = int(out["accept_len"][a])
        c = int(b) + (n << 64) + (off << 128)
        w = Philox(counter=c - 1, key=seed).random_raw(4)
        assert out["u_resample"][a] == (int(w[1]) >> 40) * 2.0 ** -24
