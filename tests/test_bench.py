"""bench.py's host logic, on the CPU: the one-GPU refusal, the parity
summary's classification of rows, the algorithmic byte count of the
headline call, the quantiles of the per-call distribution and the
counter-traffic lookup tied to the kernel sources."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_headline_algorithmic_bytes():
    # every logit read once: 256 x (2*3+1) x 151936 bf16 values, plus ids,
    # temperatures, accept lengths, emitted ids and overlaps
    assert bench.verify_bytes(256, 3, 151936) - 544538624 == 256 * 3 * 4 + 256 * 4 + 256 * 4 * 4 + 256 * 4 + 256 * 3 * 4


def _ref(acc, em, ov, u, ratio, margin):
    return [{"accept_len": np.array(acc, np.int32), "emitted": np.array(em, np.int32),
             "overlap": np.array(ov, np.float64), "u_accept": np.array(u, np.float64),
             "ratio": np.array(ratio, np.float64), "resample_margin": np.array(margin, np.float64)}]


def test_parity_summary_classifies_rows():
    K = 2
    # row 0: identical; row 1: accept decision differs at step 1 with u within 1e-6 of p/q;
    # row 2: same accept length, resampled token differs with the uniform on a CDF step;
    # row 3: differs with the uniform far from p/q; row 4: the GPU reports a row error
    acc_r = [2, 2, 0, 1, 1]
    em_r = [[5, 6, 7], [5, 6, 9], [3, -1, -1], [4, 8, -1], [1, 2, -1]]
    ov_r = [[0.5, 0.25]] * 5
    u = [[0.1, 0.2], [0.1, 0.4000004], [0.9, 0.1], [0.1, 0.7], [0.1, 0.1]]
    ratio = [[0.5, 0.5], [0.6, 0.4], [0.2, 0.3], [0.5, 0.1], [0.5, 0.01]]
    margin = [0.3, 0.2, 5e-7, 0.2, 0.2]
    acc_g = np.array([2, 1, 0, 2, -1], np.int32)
    em_g = np.array([[5, 6, 7], [5, 11, -1], [4, -1, -1], [4, 8, 3], [-1, -1, -1]], np.int32)
    ov_g = np.array(ov_r, np.float32) * np.float32(1 + 2e-7)
    out = bench.parity_summary((acc_g, em_g, ov_g), _ref(acc_r, em_r, ov_r, u, ratio, margin), K)
    assert out["rows"] == 5
    assert out["exact"] == 1
    assert out["boundary_draws"] == 2
    assert out["mismatches"] == 2
    assert 1e-7 < out["max_rel_overlap"] < 1e-6


def test_traffic_is_reported_only_for_the_profiled_sources(tmp_path, monkeypatch):
    h = bench.kernel_source_hash()
    rec = {"w": {"hbm_bytes_per_launch": 123, "source_hash": h}, "old": {"hbm_bytes_per_launch": 7, "source_hash": "x"}}
    (tmp_path / "traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.measured_traffic("w", 0) == 123
    assert bench.measured_traffic("old", 0) is None
    assert bench.measured_traffic("missing", 0) is None
    assert bench.hbm_roofline(8e9, 1.0, None)["traffic"] is None
    assert bench.hbm_roofline(8e9, 1.0, None)["frac"] == pytest.approx(1.0)


def test_quantiles_of_the_per_call_distribution():
    vals = sorted([4.0, 1.0, 3.0, 2.0, 5.0])
    assert bench.quantile(vals, 0.5) == 3.0
    assert bench.quantile(vals, 0.0) == 1.0 and bench.quantile(vals, 1.0) == 5.0
    assert bench.quantile(vals, 0.1) == pytest.approx(1.4)  # linear between the first two
    assert bench.quantile(vals, 0.9) == pytest.approx(4.6)
    assert bench.quantile([7.0], 0.9) == 7.0
    assert bench.quantile([], 0.5) is None
    # agrees with numpy's default (linear) quantile
    rng = np.random.default_rng(3)
    x = sorted(rng.random(101).tolist())
    for q in (0.1, 0.5, 0.9):
        assert bench.quantile(x, q) == pytest.approx(float(np.quantile(x, q)))


def test_all_cores_baseline_on_a_tiny_batch():
    """The all-cores oracle leg on a tiny bf16 batch, two spawned workers:
    every row is covered and the throughput is positive."""
    rng = np.random.default_rng(0)
    B, K, V = 6, 2, 64
    f32 = rng.standard_normal((B, K + 1, V)).astype(np.float32)
    tgt = (f32.view(np.uint32) >> 16).astype(np.uint16)
    drf = (f32[:, :K].view(np.uint32) >> 16).astype(np.uint16)
    ids = rng.integers(0, V, size=(B, K)).astype(np.int32)
    T = np.ones(B, np.float64)
    r = bench.cpu_baseline_all_cores((tgt, drf, ids, T), K, budget_s=0.3, workers=2)
    assert r["cores"] == 2 and r["kind"] == "oracle" and r["value"] > 0
    assert r["host_cpus"] == os.cpu_count()
    assert int(r["sample"].split()[0]) >= B


def test_tv_three_pass_floor():
    """The TV loss's three-pass floor at the measured ceilings: the two
    tensors read twice (plus the indicator words written), then the draft
    and the words read and the float32 gradient written."""
    N, K, V = 16384, 3, 151936
    logits = N * K * V * 2
    words = N * K * 10 * 256 * 8
    expect = (4 * logits + words) / bench.STREAM_READ_GBS / 1e6 + (logits + words + 2 * logits) / bench.COPY_GBS / 1e6
    assert bench.tv_three_pass_floor_ms(N, K, V) == pytest.approx(expect, rel=1e-12)
    assert 17.5 < expect < 19.0
