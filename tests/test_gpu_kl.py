"""GPU parity of spec_kl_loss_fwd_bwd (CE, forward KL, reverse KL and their
gradients) against the float64 oracle, through the C ABI."""

import numpy as np
import pytest
import torch

from oracle.kl import KIND_CE, KIND_FORWARD, KIND_REVERSE, kl_ref
from paper_2606_12370_amd import binding
from paper_2606_12370_amd import workloads as W
from tests.parity import compare_kl, device_inputs, host_logits

pytestmark = pytest.mark.gpu
KINDS = {"forward": KIND_FORWARD, "ce": KIND_CE, "reverse": KIND_REVERSE}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    binding.load_library()
    yield
    torch.cuda.synchronize()


def run_case(d, kind, T=1.0, scale=1.0, want_grad=True):
    tgt, drf = device_inputs(d)
    loss, ps, grad = binding.kl_loss_fwd_bwd(tgt, drf, T, kind, scale, want_grad=want_grad)
    torch.cuda.synchronize()
    ref = kl_ref(W.to_float64(d["target"], d["dtype"]), W.to_float64(d["draft"], d["dtype"]), float(np.float32(T)),
                 KINDS[kind], float(np.float32(scale)))
    return loss, ps, grad, ref


@pytest.mark.parametrize("kind", ["forward", "ce", "reverse"])
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("T", [1.0, 0.7])
def test_small_all_kinds(kind, dtype, T):
    d = W.tv_inputs_numpy(4, 3, 5000, dtype, 3)
    loss, ps, grad, ref = run_case(d, kind, T, scale=0.5)
    print(kind, dtype, T, compare_kl(loss, ps, grad, ref, dtype))


@pytest.mark.parametrize("kind", ["forward", "reverse"])
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("N,K,V", [(3, 1, 1), (2, 2, 7), (3, 3, 1023), (2, 8, 8197), (5, 2, 20480 + 3),
                                   (1, 1, 256 * 8192 + 8195)])
def test_ragged(kind, dtype, N, K, V):
    d = W.tv_inputs_numpy(N, K, V, dtype, 13 + V)
    loss, ps, grad, ref = run_case(d, kind)
    print(kind, dtype, N, K, V, compare_kl(loss, ps, grad, ref, dtype))


@pytest.mark.parametrize("noise", [0.05, 0.3])
def test_nearly_equal_distributions(noise):
    """Small KL: the self-normalised sums keep it accurate."""
    d = W.tv_inputs_numpy(4, 2, 60000, W.F32, 21, noise=noise)
    for kind in ("forward", "reverse", "ce"):
        loss, ps, grad, ref = run_case(d, kind)
        rep = compare_kl(loss, ps, grad, ref, W.F32)
        print(kind, noise, rep, "min KL", float(ref["per_step"].min()))


PAIR_LIMIT = {W.BF16: 1.0 / 64, W.F32: 0.5}


@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
@pytest.mark.parametrize("seed", [31, 32])
def test_pairwise_limit_both_sides(dtype, seed):
    """Forward KL and CE sum the partition-function difference pairwise only
    for pairs whose largest probabilities lie within a limit of each other
    (|log2(max q / max p)| at most 1/64 for bfloat16 logits, 1/2 for float32);
    beyond it they take the difference of the two normalisers.  Positions with
    draft noise from 0.003 to 2 put pairs on both sides of the limit."""
    N = 48
    d = W.tv_inputs_numpy(N, 2, 6000, dtype, seed, noise=np.logspace(-2.5, 0.3, N))
    zt, zd = W.to_float64(d["target"], dtype), W.to_float64(d["draft"], dtype)
    lam = lambda z: np.log2(np.exp(z - z.max(-1, keepdims=True)).sum(-1))
    dl = np.abs(lam(zt) - lam(zd))
    lim = PAIR_LIMIT[dtype]
    assert ((dl > lim / 2) & (dl <= lim)).sum() >= 2 and ((dl > lim) & (dl <= 2 * lim)).sum() >= 2
    for kind in ("forward", "ce"):
        loss, ps, grad, ref = run_case(d, kind)
        rep = compare_kl(loss, ps, grad, ref, dtype)
        print(kind, dtype, seed, rep)


def dominant_pair_inputs(dtype, seed, N=6, K=2, V=1024):
    """Rows whose draft puts nearly all its mass on two tokens a, b that the
    target rates about e^-27 below its largest, with log ratios
    d = log q - log p that differ by only eps / T between a and b (d itself
    about 27 / T): the reverse-KL gradient q (d - mu) of both is then a small
    difference of two large log ratios.  eps is exact in the storage type;
    row (n, 5) holds an exact tie of the two draft logits."""
    rng = np.random.default_rng(seed)
    zt = (rng.standard_normal((N, K, V)) * 2.0).astype(np.float32)
    zd = (rng.standard_normal((N, K, V)) * 2.0).astype(np.float32)
    eps = [0.01, 0.001, 0.03, 0.1, 0.0, 0.02] if dtype == W.F32 else [0.125, 0.25, 0.0, 0.5, 0.125, 0.25]
    for n in range(N):
        for k in range(K):
            a, b = rng.choice(V, 2, replace=False)
            gap = [1.0, 2.0, 3.0, 4.0, 6.0, 0.0][n]
            e = eps[(n + k) % len(eps)]
            zt[n, k, a], zd[n, k, a] = -20.0, 30.0
            zt[n, k, b], zd[n, k, b] = -20.0 - gap - e, 30.0 - gap
    store = (lambda x: W.f32_to_bf16_bits(x)) if dtype == W.BF16 else (lambda x: x)
    return dict(target=store(zt), draft=store(zd), dtype=dtype, N=N, K=K, V=V)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("T", [1.0, 0.5])
def test_reverse_kl_dominant_tokens_with_close_log_ratios(dtype, T):
    d = dominant_pair_inputs(dtype, 41 if T == 1.0 else 42)
    for kind in ("reverse", "forward"):
        loss, ps, grad, ref = run_case(d, kind, T)
        print(kind, dtype, T, compare_kl(loss, ps, grad, ref, dtype))


def test_forward_only_q_equals_p_and_determinism():
    d = W.tv_inputs_numpy(6, 3, 30000, W.BF16, 4)
    loss, ps, grad, ref = run_case(d, "ce", want_grad=False)
    assert grad is None
    compare_kl(loss, ps, None, ref, W.BF16)
    d = W.tv_inputs_numpy(3, 2, 30000, W.F32, 5, q_equals_p=True)
    for kind in ("forward", "reverse"):
        loss, ps, grad, ref = run_case(d, kind)
        assert float(ps.abs().max()) < 1e-6
        assert float(grad.abs().max()) < 1e-7
    tgt, drf = device_inputs(W.tv_inputs_numpy(8, 3, 40000, W.BF16, 6))
    a = binding.kl_loss_fwd_bwd(tgt, drf, 0.9, "reverse", 0.25)
    b = binding.kl_loss_fwd_bwd(tgt, drf, 0.9, "reverse", 0.25)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_training_workload_sampled_positions():
    """N=16384 positions x 3 steps x V=151936 (bf16), forward KL (CE's
    gradient): sampled positions against the oracle, the total loss against
    the float64 sum of the kernel's own per-step values."""
    cfg = W.CONFIGS["tv_bf16_n16384_k3_v151936"]
    d = W.tv_inputs_torch(cfg["N"], cfg["K"], cfg["V"], cfg["dtype"], cfg["seed"])
    for kind in ("forward", "reverse"):
        loss, ps, grad = binding.kl_loss_fwd_bwd(d["target"], d["draft"], 1.0, kind, 1.0)
        torch.cuda.synchronize()
        pos = np.sort(np.random.default_rng(cfg["seed"]).choice(cfg["N"], size=4, replace=False))
        pi = torch.as_tensor(pos, device="cuda")
        ref = kl_ref(host_logits(d["target"][pi], W.BF16), host_logits(d["draft"][pi], W.BF16), 1.0, KINDS[kind])
        rep = compare_kl(loss, ps, grad, ref, W.BF16, positions=pos, loss_exact=False)
        total = ps.cpu().numpy().astype(np.float64).mean(axis=1).sum()
        lg = float(loss.cpu().numpy()[0])
        assert abs(lg - total) <= 1e-5 * abs(total)
        print(kind, "training workload", rep, "loss", lg)
        del grad
        torch.cuda.empty_cache()


def masked_inputs(dtype, seed, N=3, K=2, V=5000):
    """Logits with a masked vocabulary: the same 5 % of positions and the last
    37 tokens are -inf in both the target and the draft row (p = q = 0)."""
    d = W.tv_inputs_numpy(N, K, V, dtype, seed)
    rng = np.random.default_rng(seed + 1)
    mask = rng.random((N, K, V)) < 0.05
    mask[..., V - 37:] = True
    neg = W.f32_to_bf16_bits(np.array([-np.inf], np.float32))[0] if dtype == W.BF16 else np.float32(-np.inf)
    for key in ("target", "draft"):
        arr = d[key].copy()
        arr[mask] = neg
        d[key] = arr
    return d


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("T", [1.0, 0.8])
def test_masked_vocabulary(dtype, T):
    d = masked_inputs(dtype, 61 if T == 1.0 else 62)
    for kind in ("forward", "ce", "reverse"):
        loss, ps, grad, ref = run_case(d, kind, T)
        assert np.all(np.isfinite(ref["grad"])) and np.all(np.isfinite(ref["per_step"]))
        g = grad.cpu().numpy()
        tm = W.to_float64(d["target"], dtype)
        assert np.all(g[np.isneginf(tm)] == 0.0)
        print(kind, dtype, T, compare_kl(loss, ps, grad, ref, dtype))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_target_masked_tokens_forward_and_ce(dtype):
    """Tokens the target masks (-inf) but the draft does not: p = 0 < q, so
    they add nothing to forward KL or CE and their gradient is q (reverse KL
    is infinite there).  Positions with draft noise from 0.003 to 2 put pairs
    on both sides of the pair limit."""
    N, K, V = 24, 2, 4000
    d = W.tv_inputs_numpy(N, K, V, dtype, 81, noise=np.logspace(-2.5, 0.3, N))
    mask = np.random.default_rng(82).random((N, K, V)) < 0.05
    neg = W.f32_to_bf16_bits(np.array([-np.inf], np.float32))[0] if dtype == W.BF16 else np.float32(-np.inf)
    arr = d["target"].copy()
    arr[mask] = neg
    d["target"] = arr
    for kind in ("forward", "ce"):
        loss, ps, grad, ref = run_case(d, kind, 0.9)
        assert np.all(np.isfinite(ref["grad"])) and np.all(np.isfinite(ref["per_step"]))
        print(kind, dtype, compare_kl(loss, ps, grad, ref, dtype))
