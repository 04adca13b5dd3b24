"""GPU parity of spec_verify_target_only, spec_sample and spec_diagnostics
against the float64 oracle (through the C ABI): small cases on every row,
ragged multi-chunk vocabularies, special cases and row errors, and the
benchmark-sized batch on sampled rows."""

import numpy as np
import pytest
import torch
from scipy import stats

from oracle.variants import diagnostics_ref, sample_ref, verify_target_only_ref
from paper_2606_12370_amd import binding
from paper_2606_12370_amd import workloads as W
from tests.parity import (compare_diagnostics, compare_sample, compare_target_only, device_inputs,
                          host_logits)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    binding.load_library()
    yield
    torch.cuda.synchronize()


def _store(x32, dtype):
    return W.f32_to_bf16_bits(x32) if dtype == W.BF16 else np.ascontiguousarray(x32, np.float32)


def _to_device(arr, dtype):
    if dtype == W.BF16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


# ----------------------------------------------------------------------------
# target-only verification

def run_to(d, ids, seed=0, offset=0):
    tgt = _to_device(d["target"], d["dtype"])
    out = binding.verify_target_only(tgt, torch.from_numpy(ids).cuda(), torch.from_numpy(d["temperature"]).cuda(),
                                     seed, offset, want_debug=True)
    torch.cuda.synchronize()
    ref = verify_target_only_ref(W.to_float64(d["target"], d["dtype"]), ids,
                                 d["temperature"].astype(np.float64), seed, offset)
    return out, ref


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("B,K,V", [(4, 1, 1024), (6, 3, 20000), (3, 2, 2049), (5, 1, 1023), (4, 4, 7), (3, 1, 1),
                                   (2, 8, 9000), (3, 3, 65536 + 24), (2, 2, 256 * 8192 + 8195),
                                   (3, 2, 4096), (3, 2, 8192), (3, 2, 8193)])
def test_target_only_ragged(dtype, B, K, V):
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", 100 + B + K + V)
    ids = W.greedy_ids(d["draft"], dtype)
    out, ref = run_to(d, ids, seed=13, offset=2)
    rep = compare_target_only(out, ref, dtype)
    print(dtype, B, K, V, rep)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_target_only_forced_rejections(dtype):
    """Draft ids that are not the target's top token, on peaked targets: most
    rows reject, often with the rejected token holding most of its chunk's
    mass, so the residual's chunk masses are exercised where a difference of
    statistics would cancel."""
    B, K, V = 64, 3, 50000
    rng = np.random.default_rng(5)
    z = rng.normal(0, 1, size=(B, K + 1, V)).astype(np.float32)
    top = rng.integers(0, V, size=(B, K + 1))
    for b in range(B):
        for i in range(K + 1):
            z[b, i, top[b, i]] += rng.uniform(2.0, 14.0)  # p(top) from about 1e-3 to almost 1
    ids = top[:, :K].astype(np.int32).copy()
    flip = rng.random((B, K)) < 0.3
    ids[flip] = rng.integers(0, V, size=flip.sum())
    d = dict(target=_store(z, dtype), temperature=rng.uniform(0.6, 1.2, size=B).astype(np.float32), dtype=dtype)
    out, ref = run_to(d, ids, seed=3)
    rep = compare_target_only(out, ref, dtype)
    n = ref["accept_len"]
    print(dtype, rep, "accept_len histogram", np.bincount(n, minlength=K + 1))
    assert (n < K).sum() > 10 and (n == K).sum() > 0


def test_target_only_special_rows():
    V = 20000
    z = np.zeros((6, 3, V), np.float32)
    ids = np.zeros((6, 2), np.int32)
    z[0, :, :] = -np.inf; z[0, :, 17] = 0.0; ids[0] = 17        # one-hot on the draft: accept, bonus 17
    z[1, 0, 5] = -np.inf; ids[1] = 5                            # p(x) = 0: reject at step 0
    z[2, 0, :] = -np.inf; z[2, 0, [3, 19999]] = 0.0; ids[2] = 3  # p(x) = 1/2, the rest in the last chunk
    z[3, 0, :16384] = -np.inf; z[3, 0, 16384] = 0.0; ids[3] = 16384  # x alone in its chunk's mass
    z[4, 1, 7] = np.nan; ids[4] = 1                            # row error
    ids[5] = [0, V]                                            # draft id out of range
    d = dict(target=z, temperature=np.ones(6, np.float32), dtype=W.F32)
    out, ref = run_to(d, ids, seed=8)
    compare_target_only(out, ref, W.F32)
    acc = out["accept_len"].cpu().numpy()
    em = out["emitted"].cpu().numpy()
    assert acc[0] == 2 and list(em[0]) == [17, 17, 17]
    assert acc[1] == 0 and em[1, 0] != 5
    assert acc[4] == -1 and acc[5] == -1


def test_target_only_chi_square():
    """65536 rows sharing one target: the GPU's first emitted token follows p_0."""
    B, V = 65536, 8
    rng = np.random.default_rng(2)
    p = rng.dirichlet(np.full(V, 0.8), size=2)
    z = np.broadcast_to(np.log(p).astype(np.float32), (B, 2, V)).copy()
    ids = np.full((B, 1), int(np.argsort(p[0])[-2]), np.int32)
    d = dict(target=z, temperature=np.ones(B, np.float32), dtype=W.F32)
    out, ref = run_to(d, ids, seed=77)
    compare_target_only(out, ref, W.F32)
    counts = np.bincount(out["emitted"][:, 0].cpu().numpy(), minlength=V)
    p0 = np.exp(z[0, 0].astype(np.float64))
    pval = stats.chisquare(counts, p0 / p0.sum() * B).pvalue
    print("chi-square p-value", pval)
    assert pval > 1e-3


def test_target_only_strided_view_and_scalar_temperature():
    B, K, V = 3, 2, 4099
    d = W.verify_inputs_numpy(B, K, V, W.BF16, "rollout", 17)
    ids = W.greedy_ids(d["draft"], W.BF16)
    tgt, _ = device_inputs(d)
    big = torch.zeros((B, K + 2, V + 3), dtype=tgt.dtype, device="cuda")
    big[:, 1:K + 2, 1:V + 1] = tgt
    view = big[:, 1:K + 2, 1:V + 1]
    idt = torch.from_numpy(ids).cuda()
    a = binding.verify_target_only(view, idt, 0.9, 4, 1, want_debug=True)
    b = binding.verify_target_only(tgt, idt, 0.9, 4, 1, want_debug=True)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k].nan_to_num(), b[k].nan_to_num()), k
    ref = verify_target_only_ref(W.to_float64(d["target"], W.BF16), ids, float(np.float32(0.9)), 4, 1)
    compare_target_only(a, ref, W.BF16)


def test_target_only_benchmark_batch_sampled_rows():
    cfg = W.CONFIGS["verify_bf16_b256_k3_v151936"]
    d = W.verify_inputs_torch(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"])
    ids = torch.argmax(d["draft"].float(), dim=-1).to(torch.int32).contiguous()
    out = binding.verify_target_only(d["target"], ids, d["temperature"], 5, 0, want_debug=True)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(1).choice(cfg["B"], size=24, replace=False))
    ri = torch.as_tensor(rows, device="cuda")
    ref = verify_target_only_ref(host_logits(d["target"][ri], W.BF16), ids[ri].cpu().numpy(),
                                 d["temperature"][ri].cpu().numpy().astype(np.float64), 5, 0, rows=rows)
    rep = compare_target_only(out, ref, W.BF16, rows=rows)
    acc = out["accept_len"].cpu().numpy()
    assert acc.min() >= 0
    print(rep, "mean accept_len", acc.mean())


# ----------------------------------------------------------------------------
# draft-stage sampler

def run_sample(z, T, dtype, seed=0, offset=0, rows_view=None):
    zd = _to_device(_store(z, dtype), dtype) if rows_view is None else rows_view
    out = binding.sample(zd, torch.from_numpy(T).cuda(), seed, offset, want_logz=True)
    torch.cuda.synchronize()
    ref = sample_ref(W.to_float64(_store(z, dtype), dtype), T.astype(np.float64), seed, offset)
    return out, ref


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_target_only_masked_vocabularies(dtype):
    d = W.masked_verify_inputs_numpy(15, 3, 20000, dtype, 43)
    out, ref = run_to(d, W.greedy_ids(d["draft"], dtype), seed=5, offset=2)
    compare_target_only(out, ref, dtype)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_sample_masked_vocabularies(dtype):
    d = W.masked_verify_inputs_numpy(15, 2, 20000, dtype, 44)
    z = W.to_float64(d["draft"], dtype).astype(np.float32).reshape(-1, 20000)
    T = np.repeat(d["temperature"], 2).astype(np.float32)
    T[::7] = 0.0  # greedy rows
    out, ref = run_sample(z, T, dtype, seed=6, offset=3)
    compare_sample(out, ref, dtype)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("R,V", [(40, 1024), (9, 20000), (17, 2049), (5, 7), (4, 1), (6, 65536 + 24),
                                 (2, 256 * 8192 + 8195), (9, 4096), (9, 8192), (9, 8193)])
def test_sample_ragged(dtype, R, V):
    rng = np.random.default_rng(R + V)
    z = (rng.standard_normal((R, V)) * rng.uniform(1, 8, size=(R, 1))).astype(np.float32)
    T = rng.uniform(0.6, 1.2, size=R).astype(np.float32)
    T[::4] = 0.0  # greedy rows
    out, ref = run_sample(z, T, dtype, seed=21, offset=5)
    rep = compare_sample(out, ref, dtype)
    print(dtype, R, V, rep)


def test_sample_greedy_ties_and_errors():
    V = 40000
    z = np.zeros((7, V), np.float32)
    z[0, [5, 20000, 39999]] = 3.0          # ties across chunks: first index
    z[1, [30000, 17000]] = 2.0             # ties, later chunk listed first
    z[2, :] = -np.inf; z[2, 39999] = -1.0  # only the last element has mass
    z[3, 100] = np.nan
    z[4, :] = -np.inf
    z[5, 3] = np.inf
    T = np.array([0, 0, 0, 0, 0, 0, -1], np.float32)
    out, ref = run_sample(z, T, W.F32)
    assert list(out["tokens"].cpu().numpy()) == [5, 17000, 39999, -1, -1, -1, -1]
    compare_sample(out, ref, W.F32)


def test_sample_chi_square_and_strided_rows():
    B, V = 65536, 8
    z = np.broadcast_to(np.linspace(-2, 1.5, V).astype(np.float32), (B, V)).copy()
    z[:, 4] = -np.inf
    T = np.full(B, 0.8, np.float32)
    out, ref = run_sample(z, T, W.F32, seed=31)
    compare_sample(out, ref, W.F32)
    counts = np.bincount(out["tokens"].cpu().numpy(), minlength=V)
    p = np.exp(z[0].astype(np.float64) / np.float64(np.float32(0.8)))
    pval = stats.chisquare(counts[p > 0], (p / p.sum() * B)[p > 0]).pvalue
    print("chi-square p-value", pval)
    assert pval > 1e-3 and counts[4] == 0
    # rows of a larger tensor (odd row stride, unaligned start)
    R, V2 = 11, 3001
    rng = np.random.default_rng(4)
    zz = (rng.standard_normal((R, V2)) * 3).astype(np.float32)
    big = torch.zeros((R, V2 + 5), dtype=torch.float32, device="cuda")
    big[:, 1:V2 + 1] = torch.from_numpy(zz).cuda()
    TT = np.full(R, 1.1, np.float32)
    out, ref = run_sample(zz, TT, W.F32, seed=6, rows_view=big[:, 1:V2 + 1])
    compare_sample(out, ref, W.F32)


def test_sample_benchmark_draft_rows():
    """The draft rows of the benchmark batch as B*K = 768 sampler rows."""
    cfg = W.CONFIGS["verify_bf16_b256_k3_v151936"]
    d = W.verify_inputs_torch(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"])
    flat = d["draft"].reshape(-1, cfg["V"])
    T = d["temperature"].repeat_interleave(cfg["K"]).contiguous()
    out = binding.sample(flat, T, 9, 4, want_logz=True)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(3).choice(flat.shape[0], size=32, replace=False))
    ri = torch.as_tensor(rows, device="cuda")
    ref = sample_ref(host_logits(flat[ri], W.BF16), T[ri].cpu().numpy().astype(np.float64), 9, 4, rows=rows)
    print(compare_sample(out, ref, W.BF16, rows=rows))


# ----------------------------------------------------------------------------
# diagnostics

def run_diag(d):
    tgt, drf = device_inputs(d)
    out = binding.diagnostics(tgt, drf, torch.from_numpy(d["temperature"]).cuda())
    torch.cuda.synchronize()
    ref = diagnostics_ref(W.to_float64(d["target"], d["dtype"]), W.to_float64(d["draft"], d["dtype"]),
                          d["temperature"].astype(np.float64))
    return out, ref


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("B,K,V", [(4, 1, 1024), (6, 3, 20000), (3, 2, 2049), (4, 4, 7), (3, 1, 1), (2, 8, 9000),
                                   (3, 3, 65536 + 24), (2, 1, 256 * 8192 + 8195),
                                   (3, 2, 4096), (3, 2, 8191), (3, 2, 8192), (3, 2, 8193)])
def test_diagnostics_ragged(dtype, B, K, V):
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", 300 + B + K + V)
    out, ref = run_diag(d)
    rep = compare_diagnostics(out, ref, dtype)
    print(dtype, B, K, V, rep)


def test_diagnostics_controls_and_errors():
    d = W.verify_inputs_numpy(6, 2, 30000, W.F32, "rollout", 12, q_equals_p=True)
    out, ref = run_diag(d)
    compare_diagnostics(out, ref, W.F32)
    np.testing.assert_allclose(out["alpha_rs"].cpu().numpy(), 1.0, rtol=1e-5)
    assert bool((out["alpha_p_gt_q"] == 0).all())
    # peaked and flat targets, ties in the draft's maximum, row errors
    z = np.zeros((5, 2, 20000), np.float32)
    zd = np.zeros((5, 1, 20000), np.float32)
    z[0, 0, 123] = 30.0; zd[0, 0, 123] = 5.0             # p almost one-hot on the greedy token
    zd[1, 0, [19000, 700]] = 4.0                         # draft ties: first index
    z[2, 0, 9] = np.nan
    zd[3, 0, :] = -np.inf
    T = np.array([1, 1, 1, 1, 0], np.float32)            # T = 0 is an error here
    d = dict(target=z, draft=zd, temperature=T, dtype=W.F32)
    out, ref = run_diag(d)
    compare_diagnostics(out, ref, W.F32)
    g = out["greedy_draft"].cpu().numpy()
    assert g[0, 0] == 123 and g[1, 0] == 700
    assert list(out["rs_preferred"].cpu().numpy()[2:, 0]) == [-1, -1, -1]


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_diagnostics_greedy_ties_inside_a_subchunk(dtype):
    """Ties of the draft's largest logit inside one 8192-element (bf16) or
    4096-element (fp32) sub-chunk: in one lane at two load steps, in several
    lanes and vectors of one step, at the last element of a sub-chunk against
    the next sub-chunk, and at every 37th element.  The greedy token is the
    first index among the ties."""
    V = 20000
    ties = [[4100, 1030, 517, 3000], [9000, 8191], [6000, 4096, 4097], [2055, 2047, 5000], list(range(0, V, 37))]
    z = np.random.default_rng(5).normal(0.0, 1.0, (len(ties), 1, V)).astype(np.float32)
    zd = np.random.default_rng(6).normal(0.0, 1.0, (len(ties), 1, V)).astype(np.float32)
    for r, pos in enumerate(ties):
        zd[r, 0, pos] = 8.0
    d = dict(target=W.f32_to_bf16_bits(z) if dtype == W.BF16 else z,
             draft=W.f32_to_bf16_bits(zd) if dtype == W.BF16 else zd,
             temperature=np.ones(len(ties), np.float32), dtype=dtype)
    out, ref = run_diag(d)
    compare_diagnostics(out, ref, dtype)
    assert list(out["greedy_draft"].cpu().numpy()[:, 0]) == [min(p) for p in ties]


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_diagnostics_masked_vocabularies(dtype):
    d = W.masked_verify_inputs_numpy(15, 3, 20000, dtype, 45)
    d["target"] = np.ascontiguousarray(d["target"][:, :3])  # rows i < K
    out, ref = run_diag(d)
    compare_diagnostics(out, ref, dtype)


def test_diagnostics_benchmark_batch_sampled_rows():
    cfg = W.CONFIGS["verify_bf16_b256_k3_v151936"]
    d = W.verify_inputs_torch(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"])
    out = binding.diagnostics(d["target"], d["draft"], d["temperature"])  # target [B, K+1, V]: rows i < K
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(2).choice(cfg["B"], size=16, replace=False))
    ri = torch.as_tensor(rows, device="cuda")
    ref = diagnostics_ref(host_logits(d["target"][ri], W.BF16), host_logits(d["draft"][ri], W.BF16),
                          d["temperature"][ri].cpu().numpy().astype(np.float64))
    rep = compare_diagnostics(out, ref, W.BF16, rows=rows)
    print(rep, "mean alpha_rs", float(out["alpha_rs"].mean()), "mean alpha_to", float(out["alpha_to"].mean()))
