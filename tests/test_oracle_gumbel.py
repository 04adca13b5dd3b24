"""Pins of the Gumbel-max oracle (App. G.2, Alg. rs_gumbel) against numpy's
Philox, scipy's Gumbel distribution, brute-force argmax loops, the
multinomial oracle's acceptance decisions, and the unbiasedness of the
emitted tokens (chi-square)."""

import math

import numpy as np
import pytest
from numpy.random import Philox
from scipy import special, stats

from oracle import verify_ref
from oracle.gumbel import (TAG_SAMPLE, TAG_VERIFY, gumbel_noise, gumbel_uniforms, sample_gumbel_ref,
                           verify_gumbel_ref)
from oracle.verify import softmax_t
from paper_2606_12370_amd import workloads as W


def _chisq(counts, probs):
    probs = np.asarray(probs, dtype=np.float64)
    keep = probs > 0
    assert counts[~keep].sum() == 0
    return stats.chisquare(counts[keep], probs[keep] / probs[keep].sum() * counts.sum()).pvalue


def test_uniform_layout_against_numpy_philox():
    seed, off, V = 2024, 5, 37
    rows = np.array([0, 3, 1000])
    for tag in (TAG_VERIFY, TAG_SAMPLE):
        U = gumbel_uniforms(seed, rows, V, off, tag)
        for a, r in enumerate(rows):
            for v in range(V):
                c = int(r) + ((v // 8) << 64) + (off << 128) + (tag << 192)
                w = int(Philox(counter=c - 1, key=seed).random_raw(4)[(v // 2) % 4])
                bits = (w >> 40) if v % 2 == 0 else (w >> 8) & 0xFFFFFF
                assert U[a, v] == (bits + 0.5) / 2 ** 24, (tag, r, v)
    assert not np.array_equal(gumbel_uniforms(seed, rows, V, off, 2), gumbel_uniforms(seed, rows, V, off, 3))


def test_gumbel_noise_distribution():
    U = gumbel_uniforms(7, np.array([0]), 200000, 0, TAG_VERIFY)[0]
    assert U.min() > 0.0 and U.max() < 1.0
    G = gumbel_noise(U)
    assert stats.kstest(G, stats.gumbel_r.cdf).pvalue > 1e-3
    assert np.all(np.isfinite(G))


def test_sample_gumbel_brute_force_and_greedy():
    rng = np.random.default_rng(3)
    z = rng.normal(0, 2, size=(6, 50))
    z[1, :10] = -np.inf
    T = np.array([1.0, 0.7, 1.3, 0.0, 2.0, 0.5])
    out = sample_gumbel_ref(z, T, 99, 4)
    U = gumbel_uniforms(99, np.arange(6), 50, 4, TAG_SAMPLE)
    for r in range(6):
        if T[r] == 0:
            assert out["token"][r] == int(np.argmax(z[r]))
            continue
        best, arg = -math.inf, -1
        for v in range(50):
            sc = z[r, v] / T[r] - math.log(-math.log(U[r, v]))
            if sc > best:
                best, arg = sc, v
        assert out["token"][r] == arg
    assert out["token"][1] >= 10


def test_sample_gumbel_frequencies_follow_softmax():
    B, V, T = 60000, 8, 0.7
    z = np.linspace(-1.5, 2.0, V)
    z[2] = -np.inf
    out = sample_gumbel_ref(np.broadcast_to(z, (B, V)), T, 11)
    assert _chisq(np.bincount(out["token"], minlength=V), special.softmax(z / T)) > 1e-3


def test_sample_gumbel_row_errors():
    z = np.zeros((4, 5))
    z[0, 1] = np.nan
    z[1, :] = -np.inf
    out = sample_gumbel_ref(z, np.array([1.0, 1.0, -1.0, np.inf]), 0)
    assert list(out["token"]) == [-1, -1, -1, -1]


@pytest.mark.parametrize("gen,K,V", [("rollout", 3, 900), ("rollout_t", 2, 3000), ("tiny", 1, 64)])
def test_acceptance_equals_multinomial_oracle(gen, K, V):
    d = W.verify_inputs_numpy(20, K, V, W.F32, gen, V + K)
    a = verify_gumbel_ref(d["target"], d["draft"], d["ids"], d["temperature"], 8, 2)
    b = verify_ref(d["target"], d["draft"], d["ids"], d["temperature"], 8, 2)
    np.testing.assert_array_equal(a["accept_len"], b["accept_len"])
    np.testing.assert_array_equal(a["overlap"], b["overlap"])
    for r in range(20):
        n = b["accept_len"][r]
        np.testing.assert_array_equal(a["emitted"][r, :n], b["emitted"][r, :n])
        assert np.all(a["emitted"][r, n + 1:] == -1)


def test_emitted_tokens_follow_target_shared():
    """65536 rows sharing one (target, draft) pair, draft ids drawn from q:
    the first emitted token follows p_0; given a rejection it follows
    max(0, p - q); given acceptance the bonus follows p_1."""
    d = W.verify_inputs_numpy(65536, 1, 8, W.F32, "exact", 1002, shared_target=True)
    out = verify_gumbel_ref(d["target"], d["draft"], d["ids"], d["temperature"], 17)
    p0, _ = softmax_t(d["target"][0, 0].astype(np.float64), 1.0)
    q0, _ = softmax_t(d["draft"][0, 0].astype(np.float64), 1.0)
    p1, _ = softmax_t(d["target"][0, 1].astype(np.float64), 1.0)
    assert _chisq(np.bincount(out["emitted"][:, 0], minlength=8), p0) > 1e-3
    acc = out["accept_len"] == 1
    assert _chisq(np.bincount(out["emitted"][~acc, 0], minlength=8), np.maximum(0, p0 - q0)) > 1e-3
    assert _chisq(np.bincount(out["emitted"][acc, 1], minlength=8), p1) > 1e-3


def test_bonus_follows_tempered_target():
    """q = p accepts every draft; the bonus then follows softmax(z_K / T)."""
    d = W.verify_inputs_numpy(65536, 1, 8, W.F32, "exact", 1003, shared_target=True, q_equals_p=True)
    T = 0.6
    out = verify_gumbel_ref(d["target"], d["draft"], d["ids"], T, 23)
    assert np.all(out["accept_len"] == 1)
    p1, _ = softmax_t(d["target"][0, 1].astype(np.float64), T)
    assert _chisq(np.bincount(out["emitted"][:, 1], minlength=8), p1) > 1e-3


def test_bonus_brute_force_and_row_errors():
    d = W.verify_inputs_numpy(6, 2, 40, W.F32, "tiny", 5, q_equals_p=True)
    d["temperature"][:] = [0.5, 1.0, 1.5, 0.9, 1.1, 0.0]
    out = verify_gumbel_ref(d["target"], d["draft"], d["ids"], d["temperature"], 3, 1)
    U = gumbel_uniforms(3, np.arange(6), 40, 1, TAG_VERIFY)
    for r in range(5):
        assert out["accept_len"][r] == 2
        sc = [d["target"][r, 2, v] / np.float64(d["temperature"][r]) - math.log(-math.log(U[r, v])) for v in range(40)]
        assert out["emitted"][r, 2] == int(np.argmax(sc))
    assert out["accept_len"][5] == -1 and np.all(out["emitted"][5] == -1)
