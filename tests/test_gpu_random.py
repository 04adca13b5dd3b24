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


# TV cases that failed in randomized stress runs (dtype, N, K, V, mode, T,
# scale, generator seed, noise, q = p): bfloat16 rows with near-zero loss,
# while the pair pass folded each row's reference and log normaliser into
# one float, and fp32 rows where one token holds all but ~1e-7 of q and its
# p = q tie fell on the other side (the comparison then allowed each
# element's q error relative to the reference side's much smaller gradient)
TV_PINNED = [
    (W.F32, 17, 7, 17, 'per_step', 0.5353214849382344, 1.0, 636618818, 1.6280073720075454, False),
    (W.F32, 11, 3, 827, 'prod', 0.5985419008002765, 0.09090909090909091, 1923686899, 0.9318186958090015, False),
    (W.F32, 15, 3, 1024, 'per_step', 0.6399893742912574, 1.0, 1175399059, 0.6498682023615101, False),
    (W.F32, 11, 2, 1024, 'per_step', 0.614571305994735, 1.0, 294151511, 1.5900077923807518, False),
    # bfloat16 rows whose loss is near zero
    (W.BF16, 2, 1, 16383, 'e2e', 0.5877370358756856, 0.25, 1653754116, 0.751039508264932, True),
    (W.BF16, 1, 1, 16383, 'per_step', 0.6186013660245805, 1.0, 1042489572, 1.4123678573769916, True),
    (W.BF16, 3, 1, 16385, 'e2e', 0.6499377445544088, 0.3333333333333333, 1208717596, 1.3566071828856683, True),
    (W.BF16, 1, 2, 16384, 'e2e', 0.5758949762727816, 0.25, 1902288605, 0.31587158591191594, True),
    (W.BF16, 2, 1, 16385, 'per_step', 0.6046346804459134, 0.5, 1211503907, 1.9666147812916421, True),
    (W.BF16, 9, 1, 16385, 'per_step', 0.5068135506584948, 1.0, 1375254717, 1.2314571047451253, True),
    (W.BF16, 1, 1, 16383, 'per_step', 0.8709754052063011, 0.25, 1952137118, 1.7246157496063186, True),
    (W.BF16, 1, 1, 16384, 'e2e', 0.767167800756143, 0.25, 1460852105, 0.7678491894880181, True),
    (W.BF16, 1, 1, 16383, 'per_step', 0.6014531949959884, 1.0, 1412154745, 0.08421718972298331, False),
    (W.BF16, 1, 1, 18987, 'e2e', 0.5906463100345116, 0.25, 717875406, 0.8520056415615747, False),
    (W.BF16, 1, 1, 16384, 'e2e', 0.9257776668088197, 1.0, 896317902, 1.204378151527916, True),
    (W.BF16, 1, 1, 16383, 'per_step', 0.912704378732363, 1.0, 641862368, 0.39371383558581613, True),
    (W.BF16, 5, 1, 16384, 'per_step', 0.5414575110207168, 0.2, 1311359329, 0.2932597081905951, True),
    (W.BF16, 2, 1, 16384, 'per_step', 0.5349859701205368, 0.25, 1664052861, 1.399472496691149, True),
    (W.BF16, 1, 1, 16384, 'per_step', 1.1983738458833348, 1.0, 932581209, 1.9321023546053684, True),
    (W.BF16, 1, 1, 16383, 'per_step', 0.8987362545180111, 1.0, 1693577719, 1.7072305140983055, True),
    (W.BF16, 6, 1, 29267, 'per_step', 0.5925547810098444, 1.0, 125867505, 0.9281341164427155, True),
    (W.BF16, 3, 1, 16383, 'per_step', 0.785600122257349, 1.0, 1095618033, 1.2208713649347236, True),
    (W.BF16, 1, 1, 6471, 'e2e', 0.8545928886685633, 0.25, 1531813447, 0.46515509063923144, True),
    (W.BF16, 1, 1, 16385, 'e2e', 0.5130557432825963, 1.0, 1762346916, 0.5716181136422819, False),
    (W.BF16, 1, 3, 22356, 'e2e', 0.598449550488403, 1.0, 1580701396, 1.534411649376996, True),
    (W.BF16, 2, 1, 16385, 'per_step', 0.5183057385141903, 0.25, 2050962110, 1.8358958432146375, True),
    (W.BF16, 3, 1, 1024, 'e2e', 0.50592089890605, 1.0, 370203199, 0.5553004830737357, True),
    (W.BF16, 1, 1, 24401, 'per_step', 0.5894536973637956, 0.25, 1271492971, 0.34621057971260943, False),
    (W.BF16, 1, 1, 16383, 'e2e', 1.0555792752193194, 0.25, 660464438, 1.912859216052098, True),
]


def _tv_id(c):
    c = c.values[0] if hasattr(c, "values") else c
    return "%s-%s-V%d-gen%d" % (c[0], c[4], c[3], c[7])


@pytest.mark.parametrize("case", TV_PINNED, ids=_tv_id)
def test_tv_previously_failing_cases(case):
    dt, N, K, V, mode, T, scale, gen_seed, noise, qp = case
    d = W.tv_inputs_numpy(N, K, V, dt, gen_seed, noise=noise, q_equals_p=qp)
    tgt, drf = device_inputs(d)
    loss, ov, grad = binding.tv_loss_fwd_bwd(tgt, drf, T, mode, scale, want_grad=True)
    torch.cuda.synchronize()
    ref = oracle.tv_ref(W.to_float64(d["target"], dt), W.to_float64(d["draft"], dt),
                        float(np.float32(T)), MODES[mode], float(np.float32(scale)), want_grad=True)
    print(compare_tv(loss, ov, grad, ref, dt))


# CE / KL cases that failed the gradient comparison in randomized stress runs
# (dtype, N, K, V, kind, T, scale, generator seed, noise): before the kernels
# formed q - p and log q - log p from the exact logit difference, before the
# log ratio of the two partition functions came from a pairwise sum, and one
# (p = 1 - 1e-14) where the oracle itself lacked the precision
KL_PINNED = [
    (W.F32, 1, 8, 16384, "ce", 0.6142656209495022, 1.0, 972971823, 0.6013167328216604),
    (W.F32, 12, 6, 1024, "forward", 0.6594872303890863, 1.0 / 12, 1863491364, 1.7870415269416062),
    (W.BF16, 3, 8, 7127, "forward", 0.512600391689029, 1.0, 2003678062, 0.9935898934096685),
    (W.BF16, 18, 8, 1024, "ce", 0.5121693881247089, 1.0 / 18, 1721427363, 0.5153431730050316),
    (W.BF16, 21, 6, 1024, "forward", 0.5474361362359242, 1.0 / 21, 972473126, 1.713698312056721),
    (W.F32, 12, 1, 16383, "ce", 0.8530768906914661, 1.0, 1635841073, 0.11479992343740825),
    (W.BF16, 14, 8, 3, "reverse", 0.6647809515092243, 1.0, 1633114726, 0.8159640099163816),
    (W.F32, 11, 5, 1024, "reverse", 0.5962657758118375, 1.0 / 11, 1568780994, 1.2949953247572092),
    (W.F32, 13, 3, 1024, "reverse", 0.5356229022213345, 1.0 / 13, 2124375422, 0.682026940167951),
    (W.BF16, 12, 7, 1024, "reverse", 0.5186915158172206, 1.0 / 12, 1904719211, 0.3153271407658461),
    # the element holding both rows' largest logit at p = 0.57-0.98
    (W.F32, 21, 8, 1024, "forward", 1.475596639665728, 1.0, 770393847, 0.10252011838269154),
    (W.F32, 8, 6, 1024, "ce", 0.5467098178304036, 1.0, 227129657, 0.5021796655738667),
    (W.F32, 22, 8, 1024, "forward", 0.7322401060693238, 1.0 / 22, 351533975, 0.13656003589084276),
    # two tokens sharing nearly all the mass (p = 0.57 / 0.43, 0.62 / 0.38, 0.72 / 0.28):
    # q - p of the second one needs the pairwise ratio of the partition functions
    (W.F32, 18, 7, 1024, "ce", 0.8062491954075379, 0.25, 856847184, 0.34104919671853684),
    (W.BF16, 23, 4, 1024, "ce", 0.5342029822933412, 0.25, 133561473, 1.8033742587645176),
    (W.F32, 23, 7, 4, "ce", 1.1026908684545669, 1.0, 411418841, 0.2399019811457977),
    (W.F32, 21, 3, 1024, "forward", 0.7164230454170811, 0.25, 518468016, 0.08514644897277253),
    (W.BF16, 21, 4, 1024, "ce", 0.5368787480304352, 1.0 / 21, 1952651588, 0.06469459190593548),
    # one token holding all but 1e-14 of both distributions
    (W.F32, 15, 3, 1024, "forward", 0.5975192604769664, 1.0, 831808222, 1.319960033772397),
    # draft noise per position up to 18-92 (draft logits in the hundreds): rows whose exact
    # gradient lies below float32's range, and reverse KL where the draft's leading tokens
    # have nearly equal log ratios
    (W.BF16, 4, 3, 16383, "reverse", 1.46381765942616, 0.25, 1732116239,
     [0.08311337671380507, 0.827313912110449, 8.235116129721746, 81.97267890371153]),
    (W.BF16, 12, 2, 1024, "reverse", 0.6184885680468026, 1.0 / 12, 763233859,
     list(np.logspace(np.log10(0.0672955349239528), np.log10(41.74713811512776), 12))),
    (W.F32, 16, 8, 1024, "reverse", 0.7918173928408779, 0.25, 302259778,
     list(np.logspace(np.log10(0.09885397484826319), np.log10(91.54849261054336), 16))),
    (W.F32, 7, 7, 1024, "reverse", 0.5040757477292378, 0.25, 165275283,
     list(np.logspace(np.log10(0.09873318975182539), np.log10(18.93387516804222), 7))),
    (W.F32, 8, 1, 16385, "reverse", 0.9818716294638743, 0.25, 416231049,
     list(np.logspace(np.log10(0.053817650185256485), np.log10(48.11081547835813), 8))),
    (W.BF16, 14, 6, 1024, "reverse", 0.5128602475661578, 1.0 / 14, 156701734,
     list(np.logspace(np.log10(0.09527860944217414), np.log10(32.25606597973363), 14))),
]


def _kl_case(dt, N, K, V, kind, T, scale, gen_seed, noise, qp=False):
    from oracle.kl import kl_ref
    from tests.parity import compare_kl
    from tests.test_gpu_kl import KINDS
    d = W.tv_inputs_numpy(N, K, V, dt, gen_seed, noise=noise, q_equals_p=qp)
    tgt, drf = device_inputs(d)
    loss, ps, grad = binding.kl_loss_fwd_bwd(tgt, drf, T, kind, scale, want_grad=True)
    torch.cuda.synchronize()
    ref = kl_ref(W.to_float64(d["target"], dt), W.to_float64(d["draft"], dt), float(np.float32(T)), KINDS[kind],
                 float(np.float32(scale)))
    return compare_kl(loss, ps, grad, ref, dt)


def _kl_id(c):
    c = c.values[0] if hasattr(c, "values") else c
    return "%s-%s-V%d-gen%d" % (c[0], c[4], c[3], c[7])


@pytest.mark.parametrize("case", KL_PINNED, ids=_kl_id)
def test_kl_previously_failing_cases(case):
    print(_kl_case(*case))


def test_random_shapes_kl_gradients():
    """300 CE / forward-KL / reverse-KL cases from the recipe whose gradients
    used to fail (float32 and bf16, T 0.5-1.5, draft noise 0.05-2, rows where
    one token holds nearly all the mass), at the unchanged tolerance."""
    rng = np.random.default_rng(20261204)
    worst = 0.0
    for _ in range(300):
        dt = W.BF16 if rng.random() < 0.5 else W.F32
        K = int(rng.integers(1, 9))
        V = int(rng.choice([int(rng.integers(1, 30000)), 16383, 16384, 16385, 1024]))
        N = int(rng.integers(1, max(2, min(24, 600_000 // (V * 2 * K)))))
        kind = str(rng.choice(["forward", "ce", "reverse"]))
        T = float(rng.uniform(0.5, 1.5))
        scale = float(rng.choice([1.0, 1.0 / N, 0.25]))
        gen_seed = int(rng.integers(0, 2**31))
        noise = float(rng.uniform(0.05, 2.0))
        qp = bool(rng.random() < 0.05)
        rep = _kl_case(dt, N, K, V, kind, T, scale, gen_seed, noise, qp)
        worst = max(worst, rep.get("max_normwise_grad", 0.0) / (1e-5 if dt == W.F32 else 2e-3))
    print("largest gradient error as a fraction of the tolerance", worst)


def test_random_shapes_near_equal_verify():
    """Verification in the paper's operating regime: draft noise 0.01-0.1,
    per-step acceptance about 0.9-0.99, residual masses down to about 1e-3.
    Every row exact or a boundary draw; the boundary count is reported."""
    rng = np.random.default_rng(20261205)
    boundary = rows = 0
    alphas = []
    for _ in range(120):
        dt = W.BF16 if rng.random() < 0.6 else W.F32
        K = int(rng.integers(1, 5))
        V = int(rng.choice([int(rng.integers(1000, 40000)), 8192, 16385, 151936]))
        B = int(rng.integers(1, max(2, min(32, 3_000_000 // (V * (2 * K + 1))))))
        seed_, offset = int(rng.integers(0, 2**63)), int(rng.integers(0, 2**40))
        d = W.verify_inputs_numpy(B, K, V, dt, "near", int(rng.integers(0, 2**31)))
        tgt, drf = device_inputs(d)
        T = torch.from_numpy(d["temperature"]).cuda()
        out = binding.verify(tgt, drf, torch.from_numpy(d["ids"]).cuda(), T, seed_, offset, want_debug=True)
        torch.cuda.synchronize()
        ref = oracle.verify_ref(W.to_float64(d["target"], dt), W.to_float64(d["draft"], dt), d["ids"],
                                d["temperature"].astype(np.float64), seed_, offset)
        rep = compare_verify(out, ref, dt)
        boundary += rep["boundary_rows"]
        rows += rep["rows"]
        alphas.append(ref["overlap"].ravel())
    al = np.concatenate(alphas)
    print("rows", rows, "boundary rows", boundary, "acceptance quartiles", np.percentile(al, [25, 50, 75]))
