"""Randomized shapes, fixed generator: spec_verify and target-only
verification against the oracle on 300 cases drawn from bf16 / fp32,
K = 1..8, V from 1 to 40000 plus the sub-chunk edges (4096, 8191, 8192,
8193, 16384 + a few), per-row temperatures, random seeds and offsets, and
masked vocabularies.  Every row must match the oracle exactly or be a
boundary draw (the comparison helpers raise otherwise).  The TV loss and its
gradient on 200 cases: bf16 / fp32, all three modes, K = 1..8, V up to 30000
plus chunk edges, temperatures 0.5..1.5, three loss scales, draft noise from
nearly equal to far apart, and q = p controls."""

import numpy as np
import pytest
import torch

import oracle
from oracle.variants import verify_target_only_ref
from paper_2606_12370_amd import binding
from paper_2606_12370_amd import workloads as W
from tests.parity import compare_target_only, compare_tv, compare_verify, device_inputs
from tests.test_gpu_tv import MODES

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    binding.load_library()
    yield
    torch.cuda.synchronize()


def random_cases(n, seed):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        dt = W.BF16 if rng.random() < 0.6 else W.F32
        K = int(rng.integers(1, 9))
        V = int(rng.choice([int(rng.integers(1, 40000)), 8191, 8192, 8193, 4096, 16384 + int(rng.integers(0, 64))]))
        B = int(rng.integers(1, max(2, min(48, 2_000_000 // (V * (2 * K + 1))))))
        seed_, offset = int(rng.integers(0, 2**63)), int(rng.integers(0, 2**40))
        masked = bool(rng.random() < 0.3 and V >= 16384)
        gen_seed = int(rng.integers(0, 2**31))
        yield dt, B, K, V, seed_, offset, masked, gen_seed


def test_random_shapes_verify_and_target_only():
    boundary = 0
    for dt, B, K, V, seed, offset, masked, gen_seed in random_cases(300, 20261202):
        d = (W.masked_verify_inputs_numpy(B, K, V, dt, gen_seed) if masked
             else W.verify_inputs_numpy(B, K, V, dt, "rollout_t", gen_seed))
        tgt, drf = device_inputs(d)
        T = torch.from_numpy(d["temperature"]).cuda()
        out = binding.verify(tgt, drf, torch.from_numpy(d["ids"]).cuda(), T, seed, offset, want_debug=True)
        ids = W.greedy_ids(d["draft"], dt)
        out_to = binding.verify_target_only(tgt, torch.from_numpy(ids).cuda(), T, seed, offset, want_debug=True)
        torch.cuda.synchronize()
        zt, zd = W.to_float64(d["target"], dt), W.to_float64(d["draft"], dt)
        T64 = d["temperature"].astype(np.float64)
        rep = compare_verify(out, oracle.verify_ref(zt, zd, d["ids"], T64, seed, offset), dt)
        boundary += rep["boundary_rows"]
        compare_target_only(out_to, verify_target_only_ref(zt, ids, T64, seed, offset), dt)
    print("boundary rows", boundary)


def test_random_shapes_tv_loss_and_gradient():
    rng = np.random.default_rng(20261203)
    shifted = 0
    for _ in range(200):
        dt = W.BF16 if rng.random() < 0.6 else W.F32
        K = int(rng.integers(1, 9))
        V = int(rng.choice([int(rng.integers(1, 30000)), 16383, 16384, 16385, 1024]))
        N = int(rng.integers(1, max(2, min(24, 600_000 // (V * 2 * K)))))
        mode = str(rng.choice(list(MODES)))
        T = float(rng.uniform(0.5, 1.5))
        scale = float(rng.choice([1.0, 1.0 / N, 0.25]))
        gen_seed = int(rng.integers(0, 2**31))
        noise = float(rng.uniform(0.05, 2.0))
        qp = bool(rng.random() < 0.05)
        d = W.tv_inputs_numpy(N, K, V, dt, gen_seed, noise=noise, q_equals_p=qp)
        tgt, drf = device_inputs(d)
        loss, ov, grad = binding.tv_loss_fwd_bwd(tgt, drf, T, mode, scale, want_grad=True)
        torch.cuda.synchronize()
        ref = oracle.tv_ref(W.to_float64(d["target"], dt), W.to_float64(d["draft"], dt),
                            float(np.float32(T)), MODES[mode], float(np.float32(scale)), want_grad=True)
        shifted += compare_tv(loss, ov, grad, ref, dt)["rows_with_shifted_S"]
    print("rows with a float32 S shift", shifted)
