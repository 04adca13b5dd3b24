"""GPU parity of spec_verify_gumbel and spec_sample_gumbel against the
float64 oracle (App. G.2, Alg. rs_gumbel), through the C ABI."""

import numpy as np
import pytest
import torch
from scipy import stats

import oracle
from oracle.gumbel import sample_gumbel_ref, verify_gumbel_ref
from paper_2606_12370_amd import binding
from paper_2606_12370_amd import workloads as W
from tests.parity import compare_sample_gumbel, compare_verify_gumbel, device_inputs, host_logits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    binding.load_library()
    yield
    torch.cuda.synchronize()


def run_case(d, seed=0, offset=0, T=None, want_overlap=True):
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    if T is None:
        Tg, Tr = torch.from_numpy(d["temperature"]).cuda(), d["temperature"].astype(np.float64)
    else:
        Tg, Tr = float(T), float(np.float32(T))
    out = binding.verify(tgt, drf, ids, Tg, seed, offset, want_debug=True, want_overlap=want_overlap, gumbel=True)
    torch.cuda.synchronize()
    ref = verify_gumbel_ref(W.to_float64(d["target"], d["dtype"]), W.to_float64(d["draft"], d["dtype"]), d["ids"],
                            Tr, seed, offset)
    return out, ref


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("B,K,V", [(4, 1, 1024), (6, 3, 20000), (3, 2, 2049), (5, 1, 1023), (4, 4, 7), (3, 1, 1),
                                   (2, 8, 9000), (3, 3, 65536 + 24), (2, 2, 256 * 8192 + 8195)])
def test_verify_gumbel_ragged(dtype, B, K, V):
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", 500 + B + K + V)
    out, ref = run_case(d, seed=19, offset=4)
    print(dtype, B, K, V, compare_verify_gumbel(out, ref, dtype))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_verify_gumbel_without_overlap(dtype):
    d = W.verify_inputs_numpy(24, 3, 50000, dtype, "rollout_t", 78)
    full, ref = run_case(d, seed=6, offset=1)
    lean, _ = run_case(d, seed=6, offset=1, want_overlap=False)
    assert "overlap" not in lean
    for k in lean:
        assert torch.equal(full[k], lean[k]), k
    compare_verify_gumbel(lean, ref, dtype)


def test_verify_gumbel_chi_square_and_tempered_bonus():
    cfg = W.CONFIGS["exact_f32_b65536_k1_v8"]
    d = W.verify_inputs_numpy(cfg["B"], 1, 8, W.F32, "exact", cfg["seed"], shared_target=True)
    out, ref = run_case(d, seed=321)
    print("shared", compare_verify_gumbel(out, ref, W.F32))
    p, _ = oracle.softmax_t(d["target"][0, 0].astype(np.float64), 1.0)
    counts = np.bincount(out["emitted"][:, 0].cpu().numpy(), minlength=8)
    pval = stats.chisquare(counts, p * counts.sum()).pvalue
    print("first token chi-square p-value", pval)
    assert pval > 1e-3
    d = W.verify_inputs_numpy(cfg["B"], 1, 8, W.F32, "exact", cfg["seed"] + 1, shared_target=True, q_equals_p=True)
    out, ref = run_case(d, seed=5, T=0.6)
    compare_verify_gumbel(out, ref, W.F32)
    assert bool((out["accept_len"] == 1).all())
    p1, _ = oracle.softmax_t(d["target"][0, 1].astype(np.float64), float(np.float32(0.6)))
    counts = np.bincount(out["emitted"][:, 1].cpu().numpy(), minlength=8)
    pval = stats.chisquare(counts, p1 * counts.sum()).pvalue
    print("bonus chi-square p-value", pval)
    assert pval > 1e-3


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_verify_gumbel_row_errors(dtype):
    d = W.verify_inputs_numpy(8, 2, 3000, dtype, "rollout", 10)
    tgt = W.to_float64(d["target"], dtype).astype(np.float32)
    drf = W.to_float64(d["draft"], dtype).astype(np.float32)
    tgt[0, 1, 3] = np.nan
    drf[1, 0, 0] = np.inf
    tgt[2, 2, :] = -np.inf
    d["ids"][3, 1] = 3000
    d["temperature"][4] = 0.0
    tgt[5, 0, :100] = -np.inf
    d["ids"][6, 0] = -1
    d["target"] = W.f32_to_bf16_bits(tgt) if dtype == W.BF16 else tgt
    d["draft"] = W.f32_to_bf16_bits(drf) if dtype == W.BF16 else drf
    out, ref = run_case(d)
    assert list(ref["row_error"]) == [True, True, True, True, True, False, True, False]
    compare_verify_gumbel(out, ref, dtype)


def test_verify_gumbel_benchmark_batch_sampled_rows():
    cfg = W.CONFIGS["verify_bf16_b256_k3_v151936"]
    d = W.verify_inputs_torch(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"])
    out = binding.verify(d["target"], d["draft"], d["ids"], d["temperature"], 3, 0, want_debug=True, gumbel=True)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(4).choice(cfg["B"], size=24, replace=False))
    ri = torch.as_tensor(rows, device="cuda")
    ref = verify_gumbel_ref(host_logits(d["target"][ri], W.BF16), host_logits(d["draft"][ri], W.BF16),
                            d["ids"][ri].cpu().numpy(), d["temperature"][ri].cpu().numpy().astype(np.float64), 3, 0,
                            rows=rows)
    print(compare_verify_gumbel(out, ref, W.BF16, rows=rows))


# ----------------------------------------------------------------------------
# Gumbel-max draft sampler

def _store(x32, dtype):
    return W.f32_to_bf16_bits(x32) if dtype == W.BF16 else np.ascontiguousarray(x32, np.float32)


def _dev(arr, dtype):
    if dtype == W.BF16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("R,V", [(40, 1024), (9, 20000), (17, 2049), (5, 7), (4, 1), (6, 65536 + 24),
                                 (2, 256 * 8192 + 8195)])
def test_sample_gumbel_ragged(dtype, R, V):
    rng = np.random.default_rng(R * 7 + V)
    z = _store((rng.standard_normal((R, V)) * rng.uniform(1, 8, size=(R, 1))).astype(np.float32), dtype)
    T = rng.uniform(0.6, 1.2, size=R).astype(np.float32)
    T[::4] = 0.0
    out = binding.sample_gumbel(_dev(z, dtype), torch.from_numpy(T).cuda(), 41, 2)
    torch.cuda.synchronize()
    ref = sample_gumbel_ref(W.to_float64(z, dtype), T.astype(np.float64), 41, 2)
    print(dtype, R, V, compare_sample_gumbel(out["tokens"], ref))


def test_sample_gumbel_chi_square_errors_and_strides():
    B, V = 65536, 8
    z = np.broadcast_to(np.linspace(-2, 1.5, V).astype(np.float32), (B, V)).copy()
    z[:, 4] = -np.inf
    out = binding.sample_gumbel(torch.from_numpy(z).cuda(), 0.8, 7)
    torch.cuda.synchronize()
    ref = sample_gumbel_ref(z.astype(np.float64), float(np.float32(0.8)), 7)
    compare_sample_gumbel(out["tokens"], ref)
    counts = np.bincount(out["tokens"].cpu().numpy(), minlength=V)
    p = np.exp(z[0].astype(np.float64) / np.float64(np.float32(0.8)))
    pval = stats.chisquare(counts[p > 0], (p / p.sum() * B)[p > 0]).pvalue
    print("chi-square p-value", pval)
    assert pval > 1e-3 and counts[4] == 0
    zz = np.zeros((6, 40000), np.float32)
    zz[0, [5, 20000, 39999]] = 3.0
    zz[1, 100] = np.nan
    zz[2, :] = -np.inf
    zz[3, 7] = np.inf
    T = np.array([0, 1, 1, 1, -1, 0.5], np.float32)
    out = binding.sample_gumbel(torch.from_numpy(zz).cuda(), torch.from_numpy(T).cuda(), 3)
    torch.cuda.synchronize()
    tok = out["tokens"].cpu().numpy()
    assert list(tok[:5]) == [5, -1, -1, -1, -1] and tok[5] >= 0
    ref = sample_gumbel_ref(zz.astype(np.float64), T.astype(np.float64), 3)
    compare_sample_gumbel(out["tokens"], ref)
    R, V2 = 11, 3001
    x = (np.random.default_rng(5).standard_normal((R, V2)) * 3).astype(np.float32)
    big = torch.zeros((R, V2 + 5), dtype=torch.float32, device="cuda")
    big[:, 1:V2 + 1] = torch.from_numpy(x).cuda()
    out = binding.sample_gumbel(big[:, 1:V2 + 1], 1.1, 8)
    torch.cuda.synchronize()
    compare_sample_gumbel(out["tokens"], sample_gumbel_ref(x.astype(np.float64), float(np.float32(1.1)), 8))


def test_sample_gumbel_benchmark_draft_rows():
    cfg = W.CONFIGS["verify_bf16_b256_k3_v151936"]
    d = W.verify_inputs_torch(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"])
    flat = d["draft"].reshape(-1, cfg["V"])
    T = d["temperature"].repeat_interleave(cfg["K"]).contiguous()
    out = binding.sample_gumbel(flat, T, 9, 4)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(3).choice(flat.shape[0], size=32, replace=False))
    ri = torch.as_tensor(rows, device="cuda")
    ref = sample_gumbel_ref(host_logits(flat[ri], W.BF16), T[ri].cpu().numpy().astype(np.float64), 9, 4, rows=rows)
    print(compare_sample_gumbel(out["tokens"], ref, rows=rows))
