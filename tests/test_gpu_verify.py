"""GPU parity of spec_verify against the float64 oracle (through the C ABI).

Small cases are compared on every row; the full-size workloads (rollout
B=64, the B=256 benchmark batch, the B=1024 / V=262144 batch) on every row or
on a sample of rows, which the oracle can check one by one because every
draw depends only on (seed, row, step, offset)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2606_12370_amd import binding
from paper_2606_12370_amd import workloads as W
from tests.parity import compare_verify, device_inputs, host_logits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    binding.load_library()
    yield
    torch.cuda.synchronize()


def run_numpy_case(d, seed=0, offset=0, scalar_t=None, debug=True):
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    if scalar_t is None:
        T = torch.from_numpy(d["temperature"]).cuda()
        T_ref = d["temperature"].astype(np.float64)
    else:
        T, T_ref = float(scalar_t), float(np.float32(scalar_t))
    out = binding.verify(tgt, drf, ids, T, seed, offset, want_debug=debug)
    torch.cuda.synchronize()
    ref = oracle.verify_ref(W.to_float64(d["target"], d["dtype"]), W.to_float64(d["draft"], d["dtype"]),
                            d["ids"], T_ref, seed, offset)
    return out, ref


def test_tiny_f32():
    d = W.verify_inputs_numpy(**{k: v for k, v in W.CONFIGS["tiny_f32_b4_k1_v1024"].items()})
    out, ref = run_numpy_case(d)
    rep = compare_verify(out, ref, W.F32)
    print("tiny", rep)
    assert rep["boundary_rows"] == 0


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("B,K,V", [(6, 3, 20000), (3, 2, 2049), (5, 1, 1023), (4, 4, 7), (3, 1, 1),
                                   (2, 8, 9000), (3, 3, 65536 + 24),
                                   # sub-chunk edges: one wave streams 8192 bf16 / 4096 fp32 elements
                                   (3, 2, 4095), (3, 2, 4096), (3, 2, 4097), (3, 2, 8191), (3, 2, 8192),
                                   (3, 2, 8193), (2, 3, 16384)])
def test_ragged_multi_chunk(dtype, B, K, V):
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", 7 + B + K + V)
    out, ref = run_numpy_case(d, seed=11, offset=3)
    rep = compare_verify(out, ref, dtype)
    print(dtype, B, K, V, rep)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_large_ragged_vocabulary(dtype):
    """A vocabulary of about two million entries, not a multiple of any tile:
    129 chunks per row, ragged last chunk and vector."""
    V = 256 * 8192 + 8195
    d = W.verify_inputs_numpy(2, 2, V, dtype, "rollout_t", 31)
    out, ref = run_numpy_case(d, seed=2, offset=1)
    rep = compare_verify(out, ref, dtype)
    print(dtype, V, rep)


def test_scalar_temperature():
    d = W.verify_inputs_numpy(5, 3, 5000, W.BF16, "rollout", 21)
    out, ref = run_numpy_case(d, seed=5, scalar_t=0.8)
    compare_verify(out, ref, W.BF16)


def test_exactness_batch_and_chi_square():
    """65536 rows, K=1, V=8: row-by-row parity, then the emitted-token
    histogram of a shared target against softmax(z) (chi-square)."""
    from scipy import stats
    cfg = W.CONFIGS["exact_f32_b65536_k1_v8"]
    d = W.verify_inputs_numpy(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"])
    out, ref = run_numpy_case(d, debug=False)
    rep = compare_verify(out, ref, W.F32)
    print("exact per-row", rep)
    d = W.verify_inputs_numpy(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"], shared_target=True)
    out, ref = run_numpy_case(d, seed=123, debug=False)
    compare_verify(out, ref, W.F32)
    p, _ = oracle.softmax_t(d["target"][0, 0].astype(np.float64), 1.0)
    counts = np.bincount(out["emitted"][:, 0].cpu().numpy(), minlength=8)
    pval = stats.chisquare(counts, p * counts.sum()).pvalue
    print("chi-square p-value", pval)
    assert pval > 1e-3


def test_q_equals_p_control_accepts_all():
    cfg = W.CONFIGS["exact_f32_b65536_k1_v8"]
    d = W.verify_inputs_numpy(cfg["B"], 1, 8, W.F32, "exact", cfg["seed"], q_equals_p=True)
    out, ref = run_numpy_case(d, debug=False)
    assert bool((out["accept_len"] == 1).all())
    compare_verify(out, ref, W.F32)
    d = W.verify_inputs_numpy(8, 3, 151936, W.BF16, "rollout", 44, q_equals_p=True)
    out, ref = run_numpy_case(d, debug=False)
    assert bool((out["accept_len"] == 3).all())
    compare_verify(out, ref, W.BF16)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_row_data_errors(dtype):
    d = W.verify_inputs_numpy(8, 2, 3000, dtype, "rollout", 9)
    tgt = W.to_float64(d["target"], dtype).astype(np.float32)
    drf = W.to_float64(d["draft"], dtype).astype(np.float32)
    tgt[0, 1, 3] = np.nan
    drf[1, 0, 0] = np.inf
    tgt[2, 2, :] = -np.inf
    d["ids"][3, 1] = 3000
    d["temperature"][4] = 0.0
    tgt[5, 0, :100] = -np.inf  # legal
    d["ids"][6, 0] = -1
    d["target"] = W.f32_to_bf16_bits(tgt) if dtype == W.BF16 else tgt
    d["draft"] = W.f32_to_bf16_bits(drf) if dtype == W.BF16 else drf
    out, ref = run_numpy_case(d)
    assert list(ref["row_error"]) == [True, True, True, True, True, False, True, False]
    compare_verify(out, ref, dtype)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_masked_vocabularies(dtype):
    """-inf masks (masked tokens, p = 0) that empty whole load steps and
    sub-chunks, sparse supports shared or half-shared by target and draft,
    and block masks: every row is valid and must match the oracle."""
    d = W.masked_verify_inputs_numpy(15, 3, 20000, dtype, 41)
    out, ref = run_numpy_case(d, seed=3, offset=1)
    assert not ref["row_error"].any()
    compare_verify(out, ref, dtype)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("seed", [51, 52])
def test_wide_draft_noise(dtype, seed):
    """Draft noise log-uniform over 0.001-100 per row: from nearly equal rows
    to drafts whose logits reach the hundreds (one-hot drafts, overlaps down
    to 1e-30).  Tokens must match; overlaps within the tolerance, or, for rows
    whose logits span more than tol 2^23 T, within the float32 temperature
    scale's 2^-23 span / T."""
    d = W.verify_inputs_numpy(40, 4, 8193, dtype, "wide", seed)
    out, ref = run_numpy_case(d, seed=seed, offset=5)
    assert not ref["row_error"].any()
    print(dtype, compare_verify(out, ref, dtype), "largest span / T", float(ref["logit_range"].max()))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_unaligned_strided_views(dtype):
    """Rows that are not 16-byte aligned and non-contiguous batch strides take
    the element-wise load path; results must not change."""
    B, K, V = 3, 2, 4099
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout", 17)
    tgt, drf = device_inputs(d)
    big_t = torch.zeros((B, K + 2, V + 3), dtype=tgt.dtype, device="cuda")
    big_d = torch.zeros((B, K + 1, V + 5), dtype=drf.dtype, device="cuda")
    big_t[:, 1:K + 2, 1:V + 1] = tgt
    big_d[:, :K, 3:V + 3] = drf
    vt, vd = big_t[:, 1:K + 2, 1:V + 1], big_d[:, :K, 3:V + 3]
    ids = torch.from_numpy(d["ids"]).cuda()
    T = torch.from_numpy(d["temperature"]).cuda()
    out_v = binding.verify(vt, vd, ids, T, 4, 0, want_debug=True)
    out_c = binding.verify(tgt, drf, ids, T, 4, 0, want_debug=True)
    torch.cuda.synchronize()
    for k in out_c:
        assert torch.equal(out_v[k].nan_to_num(), out_c[k].nan_to_num()), k
    ref = oracle.verify_ref(W.to_float64(d["target"], dtype), W.to_float64(d["draft"], dtype), d["ids"],
                            d["temperature"].astype(np.float64), 4, 0)
    compare_verify(out_v, ref, dtype)


def test_determinism_and_seed():
    d = W.verify_inputs_numpy(16, 3, 40000, W.BF16, "rollout_t", 5)
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    T = torch.from_numpy(d["temperature"]).cuda()
    a = binding.verify(tgt, drf, ids, T, 99, 1, want_debug=True)
    b = binding.verify(tgt, drf, ids, T, 99, 1, want_debug=True)
    c = binding.verify(tgt, drf, ids, T, 100, 1)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k
    assert not torch.equal(a["emitted"], c["emitted"])


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_without_overlap_output(dtype):
    """With no overlap requested only the first rejected pair is read again;
    accept lengths, tokens and the debug outputs must not change."""
    d = W.verify_inputs_numpy(24, 3, 50000, dtype, "rollout_t", 77)
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    T = torch.from_numpy(d["temperature"]).cuda()
    full = binding.verify(tgt, drf, ids, T, 5, 2, want_debug=True)
    lean = binding.verify(tgt, drf, ids, T, 5, 2, want_debug=True, want_overlap=False)
    torch.cuda.synchronize()
    assert "overlap" not in lean
    for k in lean:
        assert torch.equal(full[k], lean[k]), k
    ref = oracle.verify_ref(W.to_float64(d["target"], dtype), W.to_float64(d["draft"], dtype), d["ids"],
                            d["temperature"].astype(np.float64), 5, 2)
    compare_verify(lean, ref, dtype)


def _sampled(cfg_name, nsample, seed=0, gen=None):
    cfg = W.CONFIGS[cfg_name]
    d = W.verify_inputs_torch(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], gen or cfg["gen"], cfg["seed"])
    out = binding.verify(d["target"], d["draft"], d["ids"], d["temperature"], seed, 0, want_debug=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(cfg["seed"])
    rows = np.sort(rng.choice(cfg["B"], size=min(nsample, cfg["B"]), replace=False))
    ri = torch.as_tensor(rows, device="cuda")
    ref = oracle.verify_ref(host_logits(d["target"][ri], cfg["dtype"]), host_logits(d["draft"][ri], cfg["dtype"]),
                            d["ids"][ri].cpu().numpy(), d["temperature"][ri].cpu().numpy().astype(np.float64),
                            seed, 0, rows=rows)
    rep = compare_verify(out, ref, cfg["dtype"], rows=rows)
    acc = out["accept_len"].cpu().numpy()
    assert acc.min() >= 0 and acc.max() <= cfg["K"]
    print(cfg_name, rep, "mean accept_len", acc.mean())
    return rep


def test_rollout_full_batch():
    cfg = W.CONFIGS["rollout_bf16_b64_k3_v151936"]
    d = W.verify_inputs_numpy(cfg["B"], cfg["K"], cfg["V"], cfg["dtype"], cfg["gen"], cfg["seed"])
    out, ref = run_numpy_case(d, seed=0)
    rep = compare_verify(out, ref, W.BF16)
    print("rollout B=64", rep)


def test_benchmark_batch_sampled_rows():
    _sampled("verify_bf16_b256_k3_v151936", 24)


def test_large_batch_sampled_rows():
    _sampled("large_bf16_b1024_k3_v262144", 8, seed=7)


def test_benchmark_shape_near_equal_sampled_rows():
    """The B=256, K=3, V=151936 bf16 shape with the near-equal draft recipe
    (draft noise 0.01-0.1, acceptance about 0.9-0.99): 32 sampled rows exact
    or boundary draws."""
    rep = _sampled("verify_bf16_b256_k3_v151936", 32, seed=11, gen="near")
    print("near-equal boundary rows", rep["boundary_rows"])


def test_one_workspace_across_shapes_and_kernels():
    """Calls of different shapes and of both entry points share one scratch
    workspace filled with garbage: results must not depend on its contents."""
    ws = torch.full((64 << 20,), 0xA5, dtype=torch.uint8, device="cuda")
    td = W.tv_inputs_numpy(40, 3, 30000, W.BF16, 8)
    tt, tq = device_inputs(td)
    binding.tv_loss_fwd_bwd(tt, tq, 1.0, "prod", 1.0, ws=ws)
    for (B, K, V, dt) in [(700, 1, 8, W.F32), (9, 3, 70000, W.BF16), (4000, 2, 100, W.F32)]:
        d = W.verify_inputs_numpy(B, K, V, dt, "rollout_t", B + V)
        tgt, drf = device_inputs(d)
        ids = torch.from_numpy(d["ids"]).cuda()
        T = torch.from_numpy(d["temperature"]).cuda()
        out = binding.verify(tgt, drf, ids, T, 3, 0, ws=ws)
        torch.cuda.synchronize()
        ref = oracle.verify_ref(W.to_float64(d["target"], dt), W.to_float64(d["draft"], dt), d["ids"],
                                d["temperature"].astype(np.float64), 3, 0)
        compare_verify(out, ref, dt)


@pytest.mark.parametrize("dtype,B,K,V", [(W.BF16, 37, 3, 151936), (W.F32, 9, 2, 50000), (W.BF16, 5, 4, 20000),
                                         (W.BF16, 13, 1, 8200)])
def test_launch_shape_independence(dtype, B, K, V):
    """Every draw depends only on (seed, row, step, offset): the single-read
    path gives bit-identical accept lengths, tokens and overlaps for any
    number of workgroup groups, and both paths (single read, chain) match the
    oracle row by row."""
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", 90 + B)
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    T = torch.from_numpy(d["temperature"]).cuda()
    ref = oracle.verify_ref(W.to_float64(d["target"], dtype), W.to_float64(d["draft"], dtype), d["ids"],
                            d["temperature"].astype(np.float64), 3, 5)
    base = binding.verify(tgt, drf, ids, T, 3, 5, want_debug=True, path="single_read")
    torch.cuda.synchronize()
    compare_verify(base, ref, dtype)
    for groups in (1, 2, 3, 7):
        if groups > B:
            continue
        out = binding.verify(tgt, drf, ids, T, 3, 5, want_debug=True, path="single_read", groups=groups)
        torch.cuda.synchronize()
        for key in base:
            assert torch.equal(out[key], base[key]), (groups, key)
    chain = binding.verify(tgt, drf, ids, T, 3, 5, want_debug=True, path="chain")
    torch.cuda.synchronize()
    rep = compare_verify(chain, ref, dtype)
    same = bool(torch.equal(chain["accept_len"], base["accept_len"]) and torch.equal(chain["emitted"], base["emitted"]))
    print(dtype, B, K, V, "chain and single read give the same tokens:", same, rep)


@pytest.mark.parametrize("dtype,B,K,V,recipe", [(W.BF16, 64, 3, 151936, "rollout_t"), (W.F32, 7, 2, 50000, "near"),
                                                (W.BF16, 300, 3, 20000, "near"), (W.BF16, 5, 1, 8200, "rollout_t"),
                                                (W.F32, 33, 4, 16385, "rollout_t")])
def test_residual_shapes_give_identical_bits(dtype, B, K, V, recipe):
    """The chain's pair pass reads each row's residual step with one wave or
    one workgroup per sub-chunk (the small-batch shape), or as the library
    chooses: every output is bit-identical across the three, with and
    without overlaps, and the rows match the oracle."""
    d = W.verify_inputs_numpy(B, K, V, dtype, recipe, 300 + B)
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    T = torch.from_numpy(d["temperature"]).cuda()
    for want_ov in (True, False):
        outs = {}
        for shape in ("wave", "workgroup", "auto"):
            outs[shape] = binding.verify(tgt, drf, ids, T, 11, 4, want_debug=True, want_overlap=want_ov,
                                         path="chain", residual_shape=shape)
        torch.cuda.synchronize()
        for shape in ("workgroup", "auto"):
            for key in outs["wave"]:
                assert torch.equal(outs[shape][key], outs["wave"][key]), (shape, key, want_ov)
    ref = oracle.verify_ref(W.to_float64(d["target"], dtype), W.to_float64(d["draft"], dtype), d["ids"],
                            d["temperature"].astype(np.float64), 11, 4)
    out = binding.verify(tgt, drf, ids, T, 11, 4, want_debug=True, residual_shape="workgroup")
    torch.cuda.synchronize()
    print(dtype, B, K, V, recipe, compare_verify(out, ref, dtype))


@pytest.mark.parametrize("dtype,B,K,V", [(W.BF16, 11, 2, 20000), (W.F32, 6, 3, 16384)])
def test_single_read_scalar_temperature(dtype, B, K, V):
    """One temperature for every row (no per-row array): both paths match
    the oracle at that temperature (a boundary draw may differ between them,
    so their tokens are compared through the oracle)."""
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", 40 + B)
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    T = 0.8
    ref = oracle.verify_ref(W.to_float64(d["target"], dtype), W.to_float64(d["draft"], dtype), d["ids"],
                            np.full(B, np.float32(T), dtype=np.float64), 7, 1)
    outs = {}
    for path in ("single_read", "chain"):
        outs[path] = binding.verify(tgt, drf, ids, T, 7, 1, want_debug=True, path=path)
        torch.cuda.synchronize()
        compare_verify(outs[path], ref, dtype)
    same = torch.equal(outs["single_read"]["emitted"], outs["chain"]["emitted"])
    print(dtype, B, K, V, "chain and single read give the same tokens:", same)


@pytest.mark.parametrize("dtype,V", [(W.BF16, 8201), (W.F32, 8202)])
def test_single_read_refuses_rows_not_a_whole_number_of_vectors(dtype, V):
    """A row length that is not a multiple of the 16-byte vector (8 bf16 or 4
    fp32 elements), in rows padded to 16-byte aligned strides: the
    single-read path refuses it, the automatic launch takes the chain and
    matches the oracle."""
    B, K = 5, 2
    d = W.verify_inputs_numpy(B, K, V, dtype, "rollout_t", 23)
    tgt0, drf0 = device_inputs(d)
    epv = 8 if dtype == W.BF16 else 4
    vpad = -(-V // epv) * epv
    tgt = torch.zeros((B, K + 1, vpad), dtype=tgt0.dtype, device="cuda")[..., :V]
    drf = torch.zeros((B, K, vpad), dtype=drf0.dtype, device="cuda")[..., :V]
    tgt.copy_(tgt0)
    drf.copy_(drf0)
    assert tgt.stride(1) * tgt.element_size() % 16 == 0 and tgt.data_ptr() % 16 == 0
    ids = torch.from_numpy(d["ids"]).cuda()
    T = torch.from_numpy(d["temperature"]).cuda()
    with pytest.raises(binding.SpecError):
        binding.verify(tgt, drf, ids, T, 3, 1, path="single_read")
    out = binding.verify(tgt, drf, ids, T, 3, 1, want_debug=True)
    torch.cuda.synchronize()
    ref = oracle.verify_ref(W.to_float64(d["target"], dtype), W.to_float64(d["draft"], dtype), d["ids"],
                            d["temperature"].astype(np.float64), 3, 1)
    compare_verify(out, ref, dtype)


def test_single_read_unsupported_shapes_fall_back_or_refuse():
    """K = 8 (beyond the single-read path): the automatic launch takes the
    chain and matches the oracle; asking for the single-read path refuses."""
    d = W.verify_inputs_numpy(3, 8, 3000, W.BF16, "rollout_t", 17)
    tgt, drf = device_inputs(d)
    ids = torch.from_numpy(d["ids"]).cuda()
    T = torch.from_numpy(d["temperature"]).cuda()
    out = binding.verify(tgt, drf, ids, T, 1, 2)
    torch.cuda.synchronize()
    ref = oracle.verify_ref(W.to_float64(d["target"], W.BF16), W.to_float64(d["draft"], W.BF16), d["ids"],
                            d["temperature"].astype(np.float64), 1, 2)
    compare_verify(out, ref, W.BF16)
    with pytest.raises(binding.SpecError):
        binding.verify(tgt, drf, ids, T, 1, 2, path="single_read")
