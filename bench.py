"""Benchmark of the verification hot path on one MI355X.

One step = one spec_verify call over a batch of B=256 rows, K=3 draft steps,
V=151936 (bf16 logits): temperature softmax of 4 target and 3 draft rows per
batch row, accept tests, accept length, residual / bonus resampling and the
per-step overlap sum_v min(p, q).  Inputs are synthetic (rollout-shaped
recipe, see paper_2606_12370_amd/workloads.py) and already resident in HBM;
two input copies alternate so the 256 MB last-level cache cannot serve a
step from the previous one.

Prints ONE JSON line.  `value` = verified draft tokens/s = B*K / step time.
`roofline` relates the algorithmic bytes of one call (the logits it must
read once, ids and outputs) to the call time measured with HIP events on the
launch stream; `ms_per_call_distribution` gives p10 / median / p90 of single
calls from a separate pass with an event between calls.  `cpu_baseline` times the float64 CPU oracle on a bounded
sample of rows of the same workload (`cpu_baseline_all_cores`: the same on
every host core the box grants, rows split over worker processes), and
`parity` compares the oracle's
pass over every row of that batch with the library's outputs for it.  The fused TV-loss forward+backward on the training
workload (N=16384 positions x 3 steps) is timed too and reported under
`tv_loss`; target-only verification, the draft-stage sampler (the B*K draft
rows) and the per-step diagnostics on the same batch under `target_only`,
`sample` and `diagnostics`, the Gumbel-max variants of verification and
sampling under `verify_gumbel` and `sample_gumbel`, the forward- and
reverse-KL losses with gradients on the training workload under `kl_loss`,
and spec_verify without overlaps (`verify_serving`) and on the B=64 and
B=1024 / V=262144 batches (none of them part of `value`).
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak, GB/s
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_12370_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(key, launches_bytes):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel sources; else None."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            rec = json.load(f).get(key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(d_host, K, budget_s=10.0, gpu_out=None):
    """The float64 oracle over the rows of the benchmark batch, repeated until
    about budget_s of CPU time is spent (one thread: NumPy's element-wise
    kernels do not multithread).  With gpu_out (the library's outputs for the
    same batch, seed 0, offset 0) the oracle's first pass over the batch is
    also compared with them: see parity_summary."""
    import oracle
    from paper_2606_12370_amd import workloads as W
    tgt, drf, ids, T = d_host
    B = tgt.shape[0]
    zt_all = W.to_float64(tgt, W.BF16)
    zd_all = W.to_float64(drf, W.BF16)
    rows_done, t_used = 0, 0.0
    first = []
    while t_used < budget_s or len(first) * 4 < B:
        for s0 in range(0, B, 4):
            sl = slice(s0, min(B, s0 + 4))
            t0 = time.perf_counter()
            r = oracle.verify_ref(zt_all[sl], zd_all[sl], ids[sl], T[sl], 0, 0, rows=np.arange(sl.start, sl.stop))
            t_used += time.perf_counter() - t0
            rows_done += sl.stop - sl.start
            if len(first) * 4 < B:
                first.append(r)
            if t_used >= budget_s and len(first) * 4 >= B:
                break
    parity = parity_summary(gpu_out, first, K) if gpu_out is not None else None
    return parity, {
        "value": rows_done * K / t_used,
        "unit": "verified draft tokens/s",
        "cores": 1,
        "kind": "oracle",
        "sample": "%d rows (passes over all %d rows of the B=256 K=3 V=151936 bf16 batch) through the "
                  "float64 NumPy oracle on one thread, %.1f s of CPU time" % (rows_done, B, t_used),
    }


def _oracle_rows_worker(args):
    """One worker of the all-cores CPU baseline (a spawned process: NumPy and
    the oracle only, no GPU): the oracle over its rows of the batch, repeated
    for about budget_s of wall time.  Returns (rows verified, seconds)."""
    tgt, drf, ids, T, row0, budget_s = args
    import oracle

    def f64(bits):  # bfloat16 bit patterns -> float64, exactly
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)

    zt, zd = f64(tgt), f64(drf)
    B = tgt.shape[0]
    rows, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        for s0 in range(0, B, 4):
            sl = slice(s0, min(B, s0 + 4))
            oracle.verify_ref(zt[sl], zd[sl], ids[sl], T[sl], 0, 0, rows=np.arange(row0 + sl.start, row0 + sl.stop))
            rows += sl.stop - sl.start
            if time.perf_counter() - t0 >= budget_s:
                break
    return rows, time.perf_counter() - t0


def cpu_baseline_all_cores(d_host, K, budget_s=10.0, workers=None):
    """The same oracle on up to 16 worker processes (fewer where the host
    reports fewer CPUs): the batch's rows split over spawned workers, each
    timing its own loop; throughput = all rows verified / the longest
    worker's time.  `cores` is the number of workers, `host_cpus` what the
    host reports (os.cpu_count(), which may exceed what the job is granted)."""
    import multiprocessing as mp
    n = workers or max(1, min(16, os.cpu_count() or 1))
    tgt, drf, ids, T = d_host
    parts = [c for c in np.array_split(np.arange(tgt.shape[0]), n) if len(c)]
    with mp.get_context("spawn").Pool(len(parts)) as pool:
        res = pool.map(_oracle_rows_worker,
                       [(tgt[c], drf[c], ids[c], T[c], int(c[0]), budget_s) for c in parts])
    rows = sum(r for r, _ in res)
    span = max(t for _, t in res)
    return {
        "value": rows * K / span,
        "unit": "verified draft tokens/s",
        "cores": len(parts),
        "host_cpus": os.cpu_count(),
        "kind": "oracle",
        "sample": "%d rows of the B=256 K=3 V=151936 bf16 batch through the float64 NumPy oracle, its rows split "
                  "over %d worker processes (the host reports %s CPUs), %.1f s of wall time each"
                  % (rows, len(parts), os.cpu_count(), span),
    }


def parity_summary(gpu_out, ref_chunks, K, boundary=1e-6):
    """The benchmark batch's spec_verify outputs (seed 0, offset 0) against
    the oracle, every row: accept lengths and emitted ids equal, or the first
    divergence is a boundary draw (the uniform within `boundary` of p/q for
    an accept test, or of a CDF step for the resample; the oracle's float64
    values decide), and the overlaps' largest relative error."""
    acc_r = np.concatenate([c["accept_len"] for c in ref_chunks])
    em_r = np.concatenate([c["emitted"] for c in ref_chunks])
    ov_r = np.concatenate([c["overlap"] for c in ref_chunks])
    u_r = np.concatenate([c["u_accept"] for c in ref_chunks])
    ratio_r = np.concatenate([c["ratio"] for c in ref_chunks])
    margin_r = np.concatenate([c["resample_margin"] for c in ref_chunks])
    acc_g, em_g, ov_g = gpu_out
    exact = boundary_rows = mismatch = 0
    for r in range(len(acc_r)):
        if acc_g[r] == acc_r[r] and np.array_equal(em_g[r], em_r[r]):
            exact += 1
            continue
        ng, nr = int(acc_g[r]), int(acc_r[r])
        if 0 <= ng <= K and 0 <= nr <= K:
            if ng != nr and abs(u_r[r, min(ng, nr)] - ratio_r[r, min(ng, nr)]) <= boundary:
                boundary_rows += 1
                continue
            if ng == nr and np.array_equal(em_g[r, :ng], em_r[r, :nr]) and margin_r[r] <= boundary:
                boundary_rows += 1
                continue
        mismatch += 1
    ok = np.isfinite(ov_r)
    rel = np.abs(ov_g[ok].astype(np.float64) - ov_r[ok]) / np.abs(ov_r[ok])
    return {"rows": int(len(acc_r)), "exact": exact, "boundary_draws": boundary_rows, "mismatches": mismatch,
            "max_rel_overlap": float(rel.max()) if rel.size else 0.0,
            "against": "float64 CPU oracle, seed 0, offset 0, every row of the batch"}


def quantile(sorted_vals, q):
    """Linear-interpolation quantile of an ascending list."""
    if not sorted_vals:
        return None
    x = q * (len(sorted_vals) - 1)
    i = int(x)
    j = min(i + 1, len(sorted_vals) - 1)
    return sorted_vals[i] + (sorted_vals[j] - sorted_vals[i]) * (x - i)


def timed(torch, stream, fn, steps, warmup=1):
    """Mean milliseconds of fn(it) over `steps` calls, HIP events on `stream`,
    after `warmup` untimed calls (the clocks rise over tens of milliseconds of
    sustained load)."""
    for it in range(max(1, warmup)):
        fn(it)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for it in range(steps):
        fn(it)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def verify_sweep(torch, binding, W, stream, warmup, steps):
    """spec_verify over B x K x V x dtype (rollout recipe, per-row temperatures,
    overlaps requested, two input copies of at least 1 GiB in all so that the
    Infinity Cache cannot hold them), one JSON line each: context for the
    headline, not part of it."""
    for dt in (W.BF16, W.F32):
        for V in (151936, 262144):
            for B in (64, 256, 1024):
                for K in (1, 2, 3):
                    esz = 2 if dt == W.BF16 else 4
                    batch = B * (2 * K + 1) * V * esz
                    ncp = max(2, min(8, -(-(1 << 30) // batch)))
                    cps = [W.verify_inputs_torch(B, K, V, dt, "rollout_t", 7000 + 97 * i + B + K) for i in range(ncp)]
                    o = {"accept_len": torch.empty(B, dtype=torch.int32, device="cuda"),
                         "emitted": torch.empty((B, K + 1), dtype=torch.int32, device="cuda"),
                         "overlap": torch.empty((B, K), dtype=torch.float32, device="cuda")}

                    def step(it):
                        c = cps[it % ncp]
                        binding.verify(c["target"], c["draft"], c["ids"], c["temperature"], seed=it, out=o)

                    for it in range(warmup):
                        step(it)
                    ms = timed(torch, stream, step, steps)
                    nbytes = verify_bytes(B, K, V, esz)
                    print(json.dumps({"sweep": "spec_verify", "B": B, "K": K, "V": V,
                                      "logits": "bf16" if dt == W.BF16 else "f32", "input_copies": ncp,
                                      "ms_per_call": ms, "verified_draft_tokens_per_s": B * K / (ms * 1e-3),
                                      "frac_of_8TBps": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}), flush=True)
                    del cps
                    torch.cuda.empty_cache()


# Ceilings measured on MI355X: a streaming read of this library's statistics
# passes with non-temporal loads and a resident grid, and a device-to-device
# copy (read + write traffic together).
STREAM_READ_GBS = 6650.0
COPY_GBS = 5050.0


def tv_three_pass_floor_ms(N, K, V):
    """The TV loss's three passes at those ceilings, for bf16 logits: both
    logit tensors read (statistics), read again with one 64-bit indicator
    word per thread and 16384-element chunk written (pair pass), the draft
    and the indicator words read and the float32 gradient written (gradient
    pass)."""
    logits = N * K * V * 2
    words = N * K * (-(-V // 16384)) * 256 * 8
    reads = 2 * logits / STREAM_READ_GBS + (2 * logits + words) / STREAM_READ_GBS
    grad = (logits + words + N * K * V * 4) / COPY_GBS
    return (reads + grad) / 1e6


def hbm_roofline(nbytes, ms, key):
    achieved = nbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(key, nbytes) if key else None}


def bench_variants(torch, binding, copies, stream, steps, B, K, V):
    """Target-only verification, the draft-stage sampler and the per-step
    diagnostics on the same batch (reported beside `value`, not in it)."""
    out = {}
    greedy = [torch.argmax(c["draft"].float(), dim=-1).to(torch.int32).contiguous() for c in copies]
    to_out = {"accept_len": torch.empty(B, dtype=torch.int32, device="cuda"),
              "emitted": torch.empty((B, K + 1), dtype=torch.int32, device="cuda")}

    def to_step(it):
        c = copies[it % len(copies)]
        binding.verify_target_only(c["target"], greedy[it % len(copies)], c["temperature"], seed=it, out=to_out)

    ms = timed(torch, stream, to_step, steps, warmup=100)
    nbytes = B * (K + 1) * V * 2 + B * K * 4 + B * 4 + B * 4 + B * (K + 1) * 4
    out["target_only"] = {"ms_per_call": ms, "verified_draft_tokens_per_s": B * K / (ms * 1e-3),
                          "mean_accept_len": float(to_out["accept_len"].float().mean()),
                          "roofline": hbm_roofline(nbytes, ms, "target_only_bf16_b256_k3_v151936")}
    R = B * K
    flats = [c["draft"].reshape(R, V) for c in copies]
    temps = [c["temperature"].repeat_interleave(K).contiguous() for c in copies]
    s_out = {"tokens": torch.empty(R, dtype=torch.int32, device="cuda")}

    def sample_step(it):
        binding.sample(flats[it % len(copies)], temps[it % len(copies)], seed=it, out=s_out)

    ms = timed(torch, stream, sample_step, steps, warmup=100)
    nbytes = R * V * 2 + R * 4 + R * 4
    out["sample"] = {"ms_per_call": ms, "rows": R, "rows_per_s": R / (ms * 1e-3),
                     "roofline": hbm_roofline(nbytes, ms, "sample_bf16_r768_v151936")}
    g_out = {"accept_len": torch.empty(B, dtype=torch.int32, device="cuda"),
             "emitted": torch.empty((B, K + 1), dtype=torch.int32, device="cuda"),
             "overlap": torch.empty((B, K), dtype=torch.float32, device="cuda")}

    def gumbel_step(it):
        c = copies[it % len(copies)]
        binding.verify(c["target"], c["draft"], c["ids"], c["temperature"], seed=it, out=g_out, gumbel=True)

    ms = timed(torch, stream, gumbel_step, steps, warmup=100)
    nbytes = B * (2 * K + 1) * V * 2 + B * K * 4 + B * 4 + B * 4 + B * (K + 1) * 4 + B * K * 4
    out["verify_gumbel"] = {"ms_per_call": ms, "verified_draft_tokens_per_s": B * K / (ms * 1e-3),
                            "roofline": hbm_roofline(nbytes, ms, "verify_gumbel_bf16_b256_k3_v151936")}
    sg_out = {"tokens": torch.empty(R, dtype=torch.int32, device="cuda")}

    def sample_gumbel_step(it):
        binding.sample_gumbel(flats[it % len(copies)], temps[it % len(copies)], seed=it, out=sg_out)

    ms = timed(torch, stream, sample_gumbel_step, steps, warmup=100)
    nbytes = R * V * 2 + R * 4 + R * 4
    out["sample_gumbel"] = {"ms_per_call": ms, "rows": R, "rows_per_s": R / (ms * 1e-3),
                            "roofline": hbm_roofline(nbytes, ms, "sample_gumbel_bf16_r768_v151936")}
    diag = {}

    def diag_step(it):
        c = copies[it % len(copies)]
        diag["d"] = binding.diagnostics(c["target"], c["draft"], c["temperature"])

    ms = timed(torch, stream, diag_step, steps, warmup=100)
    nbytes = B * 2 * K * V * 2 + B * 4 + B * K * (7 * 4 + 4 + 4)
    d = diag["d"]
    out["diagnostics"] = {"ms_per_call": ms, "roofline": hbm_roofline(nbytes, ms, "diagnostics_bf16_b256_k3_v151936"),
                          "mean_alpha_rs": float(d["alpha_rs"].mean()), "mean_alpha_to": float(d["alpha_to"].mean()),
                          "mean_entropy_target": float(d["entropy_target"].mean()),
                          "rs_preferred_fraction": float(d["rs_preferred"].float().mean())}
    return out


def verify_bytes(B, K, V, esize=2):
    """Algorithmic bytes of one spec_verify call: logits read once, ids and
    per-row temperatures in, accept lengths, emitted ids and overlaps out."""
    return B * (2 * K + 1) * V * esize + B * K * 4 + B * 4 + B * (K + 1) * 4 + B * 4 + B * K * 4


def bench_verify_context(torch, binding, W, copies, stream, steps):
    """spec_verify beside the headline: the same batch without overlaps
    (serving: only the first rejected step's pair is read again), and the
    rollout (B=64) and large (B=1024, V=262144, per-row temperature) batches.
    Reported next to `value`, not in it."""
    out = {}
    cfg = W.CONFIGS["verify_bf16_b256_k3_v151936"]
    B, K, V = cfg["B"], cfg["K"], cfg["V"]
    o = {"accept_len": torch.empty(B, dtype=torch.int32, device="cuda"),
         "emitted": torch.empty((B, K + 1), dtype=torch.int32, device="cuda")}

    def serving(it):
        c = copies[it % len(copies)]
        binding.verify(c["target"], c["draft"], c["ids"], c["temperature"], seed=it, want_overlap=False, out=o)

    ms = timed(torch, stream, serving, steps, warmup=100)
    nbytes = verify_bytes(B, K, V) - B * K * 4
    out["verify_serving"] = {"workload": "verify_bf16_b256_k3_v151936 without overlaps", "ms_per_call": ms,
                             "verified_draft_tokens_per_s": B * K / (ms * 1e-3),
                             "roofline": hbm_roofline(nbytes, ms, None)}
    for key in ("rollout_bf16_b64_k3_v151936", "large_bf16_b1024_k3_v262144"):
        c2 = W.CONFIGS[key]
        B2, K2, V2 = c2["B"], c2["K"], c2["V"]
        # enough copies that the 256 MB Infinity Cache cannot hold the inputs of
        # the previous calls (4 x 136 MB for B=64; 2 x 3.8 GB for B=1024)
        ncp = 4 if B2 * (2 * K2 + 1) * V2 * 2 < (512 << 20) else 2
        cps = [W.verify_inputs_torch(B2, K2, V2, W.BF16, c2["gen"], c2["seed"] + 100 * i) for i in range(ncp)]
        o2 = {"accept_len": torch.empty(B2, dtype=torch.int32, device="cuda"),
              "emitted": torch.empty((B2, K2 + 1), dtype=torch.int32, device="cuda"),
              "overlap": torch.empty((B2, K2), dtype=torch.float32, device="cuda")}

        def step2(it):
            c = cps[it % len(cps)]
            binding.verify(c["target"], c["draft"], c["ids"], c["temperature"], seed=it, out=o2)

        ms = timed(torch, stream, step2, steps, warmup=100)
        out["verify_" + key] = {"ms_per_call": ms, "input_copies": ncp,
                                "verified_draft_tokens_per_s": B2 * K2 / (ms * 1e-3),
                                "roofline": hbm_roofline(verify_bytes(B2, K2, V2), ms, None)}
        if ncp > 2:  # a batch the 256 MB Infinity Cache can hold: also warm (one copy, every call)
            def step_warm(it):
                c = cps[0]
                binding.verify(c["target"], c["draft"], c["ids"], c["temperature"], seed=it, out=o2)

            msw = timed(torch, stream, step_warm, steps, warmup=100)
            out["verify_" + key]["warm"] = {"ms_per_call": msw, "input_copies": 1,
                                            "roofline": hbm_roofline(verify_bytes(B2, K2, V2), msw, None)}
        del cps
    torch.cuda.empty_cache()
    return out


def copy_calibration(torch, dev, gib=1, reps=3):
    """A plain device-to-device copy of known size, for scaling the FETCH_SIZE
    and WRITE_SIZE counters of the other kernels in the same profile."""
    n = gib << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    log("copy calibration: %d x %d bytes" % (reps, n))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the GPU takes some tens of milliseconds of sustained load to reach its
    # clocks: 300 untimed calls (about 55 ms) put the timed ones at steady state
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=300)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-tv", action="store_true")
    ap.add_argument("--tv-steps", type=int, default=3)
    ap.add_argument("--no-verify", action="store_true", help="skip the verify benchmark (profiling runs)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip target-only verification, the sampler and the diagnostics")
    ap.add_argument("--variant-steps", type=int, default=100)
    ap.add_argument("--no-context", action="store_true",
                    help="skip spec_verify without overlaps and on the B=64 / B=1024 batches")
    ap.add_argument("--no-kl", action="store_true", help="skip the CE / KL loss legs")
    ap.add_argument("--no-tv-loss", action="store_true", help="skip the TV loss leg (keeps the KL legs)")
    ap.add_argument("--sweep", action="store_true",
                    help="only the context sweep of spec_verify: B in {64, 256, 1024} x K in {1, 2, 3} x "
                         "V in {151936, 262144} x {bf16, fp32}, one JSON line per configuration")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device copy (scales the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (the verification "
              "rows are independent and would shard over GPUs with no exchange)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_12370_amd import binding
    from paper_2606_12370_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    binding.load_library()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    if args.sweep:
        verify_sweep(torch, binding, W, stream, args.warmup, args.steps)
        return
    cfg = W.CONFIGS["verify_bf16_b256_k3_v151936"]
    B, K, V = cfg["B"], cfg["K"], cfg["V"]
    result = {
        "metric": "verified draft tokens/sec at B=256,K=3,V=151936 bf16; % of HBM peak BW",
        "value": None,
        "unit": "verified draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": None,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded rollout-shaped logits generated on the GPU)",
        "config": {"workload": "verify_bf16_b256_k3_v151936", "B": B, "K": K, "V": V, "logits": "bf16",
                   "arithmetic": "float32 per element, float64 sums", "temperature": "per row, 1.0",
                   "input_copies": 2},
    }

    if not args.no_verify or not args.no_variants:
        log("generating inputs B=%d K=%d V=%d bf16" % (B, K, V))
        copies = [W.verify_inputs_torch(B, K, V, W.BF16, cfg["gen"], cfg["seed"] + 100 * c) for c in range(2)]
    if not args.no_verify:
        outs = [{
            "accept_len": torch.empty(B, dtype=torch.int32, device=dev),
            "emitted": torch.empty((B, K + 1), dtype=torch.int32, device=dev),
            "overlap": torch.empty((B, K), dtype=torch.float32, device=dev),
        } for _ in copies]
        ws = binding.workspace(binding.verify_workspace_size(B, K, V, torch.bfloat16), dev)

        def step(it):
            c = copies[it % len(copies)]
            binding.verify(c["target"], c["draft"], c["ids"], c["temperature"], seed=it, offset=0, ws=ws,
                           out=outs[it % len(copies)])

        for it in range(args.warmup):
            step(it)
        torch.cuda.synchronize()
        log("timing %d steps" % args.steps)
        t0 = time.perf_counter()
        ev0.record(stream)
        for it in range(args.steps):
            step(it)
        ev1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms_per_step = ev0.elapsed_time(ev1) / args.steps
        acc = outs[0]["accept_len"].float()
        assert float(acc.min()) >= 0
        # logits read once, plus ids and per-row temperatures in, all outputs out
        algo_bytes = verify_bytes(B, K, V)
        achieved = algo_bytes / (ms_per_step * 1e-3) / 1e9
        result.update({
            "value": B * K / (ms_per_step * 1e-3),
            "ms_per_step": ms_per_step,
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBS,
                         "traffic": measured_traffic("verify_bf16_b256_k3_v151936", algo_bytes)},
            "emitted_tokens_per_s": float((acc + 1).sum()) / (ms_per_step * 1e-3),
            "mean_accept_len": float(acc.mean()),
            "wall_s_timed_region": wall,
        })
        # per-call distribution, from a separate pass with an event between calls
        n_dist = min(args.steps, 100)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_dist + 1)]
        evs[0].record(stream)
        for it in range(n_dist):
            step(it)
            evs[it + 1].record(stream)
        torch.cuda.synchronize()
        per_call = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(n_dist))
        result["ms_per_call_distribution"] = {"calls": n_dist, "p10": quantile(per_call, 0.10),
                                              "median": quantile(per_call, 0.50), "p90": quantile(per_call, 0.90)}
        del outs
        if not args.no_context:
            log("timing spec_verify without overlaps and on the B=64 and B=1024 batches")
            result.update(bench_verify_context(torch, binding, W, copies, stream, args.variant_steps))
    if not args.no_variants:
        log("timing target-only verification, the sampler and the diagnostics")
        result.update(bench_variants(torch, binding, copies, stream, args.variant_steps, B, K, V))
    if not args.no_verify or not args.no_variants:
        del copies
        torch.cuda.empty_cache()

    if not args.no_tv:
        tcfg = W.CONFIGS["tv_bf16_n16384_k3_v151936"]
        N, KT, VT = tcfg["N"], tcfg["K"], tcfg["V"]
        log("generating TV inputs N=%d K=%d V=%d bf16" % (N, KT, VT))
        td = W.tv_inputs_torch(N, KT, VT, W.BF16, tcfg["seed"])
        grad = torch.empty((N, KT, VT), dtype=torch.float32, device=dev)
        tws = binding.workspace(max(binding.tv_workspace_size(N, KT, VT, torch.bfloat16),
                                    binding.kl_workspace_size(N, KT, VT, torch.bfloat16)), dev)
        # both logit tensors read once, the float32 gradient written once
        tv_bytes = N * KT * VT * (2 + 2 + 4) + N * KT * 4 + 4
        if not args.no_tv_loss:
            binding.tv_loss_fwd_bwd(td["target"], td["draft"], 1.0, "prod", 1.0, ws=tws, grad_out=grad)
            torch.cuda.synchronize()
            ev0.record(stream)
            for _ in range(args.tv_steps):
                binding.tv_loss_fwd_bwd(td["target"], td["draft"], 1.0, "prod", 1.0, ws=tws, grad_out=grad)
            ev1.record(stream)
            torch.cuda.synchronize()
            tv_ms = ev0.elapsed_time(ev1) / args.tv_steps
            tv_ach = tv_bytes / (tv_ms * 1e-3) / 1e9
            result["tv_loss"] = {
                "workload": "tv_bf16_n16384_k3_v151936", "mode": "prod", "ms_per_call": tv_ms,
                "positions_per_s": N / (tv_ms * 1e-3),
                "algorithmic_bytes": tv_bytes,
                "three_pass_floor_ms": tv_three_pass_floor_ms(N, KT, VT),
                "roofline": {"bound": "hbm", "achieved": tv_ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": tv_ach / HBM_PEAK_GBS,
                             "traffic": measured_traffic("tv_bf16_n16384_k3_v151936", tv_bytes)},
            }
        if not args.no_kl:
            # the baselines the TV loss is compared against, on the same workload
            result["kl_loss"] = {}
            for kind in ("forward", "reverse"):
                binding.kl_loss_fwd_bwd(td["target"], td["draft"], 1.0, kind, 1.0, ws=tws, grad_out=grad)
                torch.cuda.synchronize()
                ev0.record(stream)
                for _ in range(args.tv_steps):
                    binding.kl_loss_fwd_bwd(td["target"], td["draft"], 1.0, kind, 1.0, ws=tws, grad_out=grad)
                ev1.record(stream)
                torch.cuda.synchronize()
                kl_ms = ev0.elapsed_time(ev1) / args.tv_steps
                result["kl_loss"][kind] = {
                    "workload": "tv_bf16_n16384_k3_v151936", "ms_per_call": kl_ms,
                    "positions_per_s": N / (kl_ms * 1e-3),
                    "roofline": hbm_roofline(tv_bytes, kl_ms, "kl_%s_bf16_n16384_k3_v151936" % kind)}
        del td, grad
        torch.cuda.empty_cache()

    if args.copy_calibration:
        copy_calibration(torch, dev)

    if not args.no_cpu_baseline and not args.no_verify:
        log("timing the CPU oracle on a sample")
        c0 = W.verify_inputs_torch(B, K, V, W.BF16, cfg["gen"], cfg["seed"])
        g = binding.verify(c0["target"], c0["draft"], c0["ids"], c0["temperature"], seed=0, offset=0)
        torch.cuda.synchronize()
        gpu_out = (g["accept_len"].cpu().numpy(), g["emitted"].cpu().numpy(), g["overlap"].cpu().numpy())
        tgt = c0["target"].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        drf = c0["draft"].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        ids = c0["ids"].cpu().numpy()
        T = c0["temperature"].cpu().numpy().astype(np.float64)
        del c0, g
        parity, result["cpu_baseline"] = cpu_baseline((tgt, drf, ids, T), K, gpu_out=gpu_out)
        result["parity"] = parity
        log("timing the CPU oracle on every host core")
        result["cpu_baseline_all_cores"] = cpu_baseline_all_cores((tgt, drf, ids, T), K)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
