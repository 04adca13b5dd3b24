"""Seeded synthetic inputs shaped like the paper's rollout and MTP-training
workloads.

This module holds input generation only: random draws, rounding to the
storage dtype and the draft-token sampler that stands in for the draft
stage.  It contains none of the verification or TV-loss arithmetic, and both
the HIP path (through the tests and the benchmark) and the CPU oracle read
the same arrays it produces.

The paper's data (Qwen rollouts on reasoning, coding, SWE and agent tasks;
SFT corpora) is not available, so every workload is synthetic with the
paper's shapes: Qwen-scale vocabularies, gamma = 3 draft steps verified
against 4 target positions, K = 1..3.  Recipes (all per batch row b):

  rollout-like verify: s_b ~ U[1, 8], sigma_b ~ U[0.2, 1.5],
      target[b, i, :] ~ N(0, s_b^2) i.i.d. per (b, i),
      draft[b, i, :]  = target[b, i, :] + N(0, sigma_b^2),
      both rounded to the storage dtype (round-to-nearest-even),
      temperature T_b = 1, or T_b ~ U[0.6, 1.2] for the large batch;
  draft ids: x[b, i] ~ softmax(stored draft[b, i, :] / T_b), drawn with the
      Gumbel-max trick from the stored (rounded) logits; for target-only
      verification the greedy ids argmax_v draft[b, i, v] instead;
  near-equal verify ("near"): the rollout recipe with draft noise
      sigma_b ~ U[0.01, 0.1] and T_b ~ U[0.6, 1.2], so that the per-step
      acceptance sum_v min(p, q) lies near 0.9-0.99 and the residual mass
      1 - alpha near 1e-2 - 1e-3 (the paper's operating regime, Sec. 6
      Tables 1-2: acceptance 0.75-0.99);
  TV loss: s_n ~ U[1, 8], target ~ N(0, s_n^2), draft = target + N(0, 1).

Two backends: ``numpy`` (host, ``numpy.random.default_rng``) for the small
cases, ``torch`` (device generator) for the large ones.  Each is
deterministic for a given seed; the two backends draw different numbers.
"""

import numpy as np

F32 = "f32"
BF16 = "bf16"

# name -> parameters.  "gen" is the generation recipe.
CONFIGS = {
    "tiny_f32_b4_k1_v1024": dict(B=4, K=1, V=1024, dtype=F32, gen="tiny", seed=1001),
    "exact_f32_b65536_k1_v8": dict(B=65536, K=1, V=8, dtype=F32, gen="exact", seed=1002),
    "rollout_bf16_b64_k3_v151936": dict(B=64, K=3, V=151936, dtype=BF16, gen="rollout", seed=1003),
    "verify_bf16_b256_k3_v151936": dict(B=256, K=3, V=151936, dtype=BF16, gen="rollout", seed=1006),
    "large_bf16_b1024_k3_v262144": dict(B=1024, K=3, V=262144, dtype=BF16, gen="rollout_t", seed=1004),
    "tv_bf16_n16384_k3_v151936": dict(N=16384, K=3, V=151936, dtype=BF16, gen="tv", seed=1005),
}


# ----------------------------------------------------------------------------
# storage-dtype helpers (bit manipulation only)

def f32_to_bf16_bits(x):
    """Round float32 values to bfloat16 (nearest-even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits):
    """Exact widening of bfloat16 bit patterns to float32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_float64(arr, dtype):
    """Exact float64 values of stored logits (uint16 bits for bf16)."""
    if dtype == BF16:
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def _store(x32, dtype):
    return f32_to_bf16_bits(x32) if dtype == BF16 else np.ascontiguousarray(x32, np.float32)


# ----------------------------------------------------------------------------
# numpy backend

def _gumbel_ids(rng, draft64, T):
    """x ~ softmax(draft / T) per row via argmax(draft / T + Gumbel)."""
    u = rng.random(draft64.shape)
    with np.errstate(divide="ignore"):
        g = -np.log(-np.log(u))
    return np.argmax(draft64 / T + g, axis=-1).astype(np.int32)


def verify_inputs_numpy(B, K, V, dtype, gen, seed, shared_target=False, q_equals_p=False):
    """Host-side verify inputs.

    Returns dict(target [B, K+1, V], draft [B, K, V] in storage form,
    ids [B, K] int32, temperature [B] float32, dtype, B, K, V).
    shared_target: replicate one target/draft pair over all rows (so a
    histogram over rows estimates one distribution).  q_equals_p: draft rows
    are copies of target rows 0..K-1 (every draft must be accepted).
    """
    rng = np.random.default_rng(seed)
    Bg = 1 if shared_target else B
    if gen == "tiny":
        s = rng.uniform(1.0, 4.0, size=Bg).astype(np.float32)
        sig = np.full(Bg, 0.5, np.float32)
    elif gen == "exact":
        s = np.ones(Bg, np.float32)
        sig = np.ones(Bg, np.float32)
    elif gen in ("rollout", "rollout_t"):
        s = rng.uniform(1.0, 8.0, size=Bg).astype(np.float32)
        sig = rng.uniform(0.2, 1.5, size=Bg).astype(np.float32)
    elif gen == "near":
        s = rng.uniform(1.0, 8.0, size=Bg).astype(np.float32)
        sig = rng.uniform(0.01, 0.1, size=Bg).astype(np.float32)
    elif gen == "wide":
        # draft noise log-uniform over 0.001-100 per row: from nearly equal
        # rows to drafts whose logits reach the hundreds
        s = rng.uniform(1.0, 8.0, size=Bg).astype(np.float32)
        sig = (10.0 ** rng.uniform(-3.0, 2.0, size=Bg)).astype(np.float32)
    else:
        raise ValueError(gen)
    tgt32 = rng.standard_normal((Bg, K + 1, V), dtype=np.float32) * s[:, None, None]
    tgt = _store(tgt32, dtype)
    tgt64 = to_float64(tgt, dtype)
    if q_equals_p:
        drf = tgt[:, :K].copy()
    else:
        noise = rng.standard_normal((Bg, K, V), dtype=np.float32) * sig[:, None, None]
        drf = _store(to_float64(tgt[:, :K], dtype).astype(np.float32) + noise, dtype)
    if gen in ("rollout_t", "near", "wide"):
        T = rng.uniform(0.6, 1.2, size=Bg).astype(np.float32)
    else:
        T = np.ones(Bg, np.float32)
    if shared_target:
        tgt = np.repeat(tgt, B, axis=0)
        drf = np.repeat(drf, B, axis=0)
        T = np.repeat(T, B)
    id_rng = np.random.default_rng(seed + 7)
    ids = _gumbel_ids(id_rng, to_float64(drf, dtype), T.astype(np.float64)[:, None, None])
    del tgt64
    return dict(target=tgt, draft=drf, ids=ids, temperature=T, dtype=dtype, B=B, K=K, V=V)


def masked_verify_inputs_numpy(B, K, V, dtype, seed):
    """Rollout-shaped verify inputs with -inf masks (masked tokens, p = 0),
    one of five patterns per batch row (b % 5):
      0  target rows masked on [0, 5000), draft rows on [8192, 16384);
      1  the same random support of 50 tokens in target and draft;
      2  random supports of 200 tokens, target and draft sharing half;
      3  draft rows masked beyond the first 3000 tokens;
      4  target rows masked on every other 512-token block.
    Draft ids are drawn from the masked draft distribution.  V >= 16384."""
    d = verify_inputs_numpy(B, K, V, dtype, "rollout_t", seed)
    tgt = to_float64(d["target"], dtype).astype(np.float32)
    drf = to_float64(d["draft"], dtype).astype(np.float32)
    rng = np.random.default_rng(seed + 11)
    for b in range(B):
        pat = b % 5
        if pat == 0:
            tgt[b, :, :5000] = -np.inf
            drf[b, :, 8192:16384] = -np.inf
        elif pat == 1:
            keep = rng.choice(V, size=50, replace=False)
            m = np.ones(V, bool); m[keep] = False
            tgt[b, :, m] = -np.inf
            drf[b, :, m] = -np.inf
        elif pat == 2:
            both = rng.choice(V, size=300, replace=False)
            mt = np.ones(V, bool); mt[both[:200]] = False
            md = np.ones(V, bool); md[both[100:]] = False
            tgt[b, :, mt] = -np.inf
            drf[b, :, md] = -np.inf
        elif pat == 3:
            drf[b, :, 3000:] = -np.inf
        else:
            blocks = (np.arange(V) // 512) % 2 == 1
            tgt[b, :, blocks] = -np.inf
    d["target"] = _store(tgt, dtype)
    d["draft"] = _store(drf, dtype)
    id_rng = np.random.default_rng(seed + 13)
    d["ids"] = _gumbel_ids(id_rng, to_float64(d["draft"], dtype), d["temperature"].astype(np.float64)[:, None, None])
    return d


def greedy_ids(draft, dtype):
    """The draft's greedy tokens (first index of each row's largest stored
    logit), the draft choice target-only verification assumes."""
    return np.argmax(to_float64(draft, dtype), axis=-1).astype(np.int32)


def tv_inputs_numpy(N, K, V, dtype, seed, noise=1.0, q_equals_p=False):
    """Host-side TV-loss inputs: target [N, K, V], draft [N, K, V].

    noise: the standard deviation of the draft's perturbation, one value or
    one per position (a length-N sequence).
    """
    rng = np.random.default_rng(seed)
    s = rng.uniform(1.0, 8.0, size=N).astype(np.float32)
    tgt = _store(rng.standard_normal((N, K, V), dtype=np.float32) * s[:, None, None], dtype)
    if q_equals_p:
        drf = tgt.copy()
    else:
        sd = np.float32(noise) if np.ndim(noise) == 0 else np.asarray(noise, dtype=np.float32).reshape(N, 1, 1)
        nz = rng.standard_normal((N, K, V), dtype=np.float32) * sd
        drf = _store(to_float64(tgt, dtype).astype(np.float32) + nz, dtype)
    return dict(target=tgt, draft=drf, dtype=dtype, N=N, K=K, V=V, temperature=1.0)


# ----------------------------------------------------------------------------
# torch (device) backend for the large cases

def _torch_dtype(dtype):
    import torch
    return torch.bfloat16 if dtype == BF16 else torch.float32


def verify_inputs_torch(B, K, V, dtype, gen, seed, device="cuda"):
    """Device-side verify inputs with the rollout recipe (torch generator).

    Returns dict(target [B, K+1, V], draft [B, K, V] torch tensors of the
    storage dtype, ids [B, K] int32, temperature [B] float32 (device), ...).
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    td = _torch_dtype(dtype)
    s = torch.empty(B, device=device).uniform_(1.0, 8.0, generator=g)
    lo, hi = (0.01, 0.1) if gen == "near" else (0.2, 1.5)
    sig = torch.empty(B, device=device).uniform_(lo, hi, generator=g)
    if gen in ("rollout_t", "near"):
        T = torch.empty(B, device=device).uniform_(0.6, 1.2, generator=g)
    else:
        T = torch.ones(B, device=device)
    tgt = torch.empty((B, K + 1, V), dtype=td, device=device)
    drf = torch.empty((B, K, V), dtype=td, device=device)
    ids = torch.empty((B, K), dtype=torch.int32, device=device)
    for b in range(B):  # one row at a time keeps the float32 temporaries small
        zt = torch.randn((K + 1, V), device=device, generator=g) * s[b]
        tgt[b] = zt.to(td)
        zd = tgt[b, :K].float() + torch.randn((K, V), device=device, generator=g) * sig[b]
        drf[b] = zd.to(td)
        u = torch.rand((K, V), device=device, generator=g, dtype=torch.float64)
        gum = -torch.log(-torch.log(u))
        ids[b] = torch.argmax(drf[b].double() / T[b].double() + gum, dim=-1).to(torch.int32)
    return dict(target=tgt, draft=drf, ids=ids, temperature=T.float(), dtype=dtype, B=B, K=K, V=V)


def tv_inputs_torch(N, K, V, dtype, seed, device="cuda", noise=1.0, chunk=256):
    """Device-side TV-loss inputs (torch generator): target, draft [N, K, V]."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    td = _torch_dtype(dtype)
    s = torch.empty(N, device=device).uniform_(1.0, 8.0, generator=g)
    tgt = torch.empty((N, K, V), dtype=td, device=device)
    drf = torch.empty((N, K, V), dtype=td, device=device)
    for n0 in range(0, N, chunk):
        n1 = min(N, n0 + chunk)
        zt = torch.randn((n1 - n0, K, V), device=device, generator=g) * s[n0:n1, None, None]
        tgt[n0:n1] = zt.to(td)
        zd = tgt[n0:n1].float() + noise * torch.randn((n1 - n0, K, V), device=device, generator=g)
        drf[n0:n1] = zd.to(td)
    return dict(target=tgt, draft=drf, dtype=dtype, N=N, K=K, V=V, temperature=1.0)
