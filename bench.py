#!/usr/bin/env python3
"""Benchmark of one speculative verify step on one MI355X: block-verify attention
(sd_block_attn, one layer) followed by vocabulary-wide acceptance (sd_accept).

Workload: the instance-adaptive ragged-block batch in the Qwen3-4B shape -- 8 sequences,
32 query / 8 kv heads, head_dim 128, bf16 KV cache with 4096 committed tokens each,
per-sequence block sizes from {8,10,...,20,24} around the training size 16, causal-in-block
mask, acceptance over the 151936-token vocabulary at T = 1 (seeded synthetic inputs).

One step = one attention call + one acceptance call over one batch.  Inputs are resident
in HBM before the timed region; the step cycles through copies of every input whose total
exceeds 1 GB so the 256 MB Infinity Cache cannot serve them.  Prints one JSON line.

The line's `roofline` is the step's: algorithmic bytes of both calls over the step time,
against the 8 TB/s HBM3E peak and against this GPU's streaming-read ceiling measured in the
same run (`read_ceiling`); `roofline.per_call` splits it into sd_block_attn and sd_accept,
each with its counter-measured HBM traffic from profiles/ (null once the kernel sources
differ from the profiled ones).  Per-call and step times are also given per batch
(`*_us_batches`).  `cpu_baseline` is the fp64 oracle on the host: median of three runs at
every OpenMP thread and single-threaded, with the CPU model.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--temperature T] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
METRIC = "verified draft tokens/s + KV/logit HBM GB/s (% of peak), Qwen3-4B shape"


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--temperature", type=float, default=1.0)
    ap.add_argument("--copies", type=int, default=0, help="input copies to rotate (0: enough for >= 1 GB)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="bound on the oracle timing")
    ap.add_argument("--verify-layers", type=int, default=36,
                    help="layers of the whole verify step timed after the main measurement (0: skip)")
    ap.add_argument("--verify-steps", type=int, default=20)
    ap.add_argument("--policy-prompts", type=int, default=1,
                    help="prompts of the block-size policy timed after the main measurement (0: skip)")
    ap.add_argument("--survival-samples", type=int, default=1 << 20,
                    help="samples of the prefix-survival model timed after the main measurement (0: skip)")
    ap.add_argument("--survival-trials", type=int, default=1024)
    ap.add_argument("--no-other-configs", dest="other_configs", action="store_false",
                    help="skip the drafter and long-context timings after the main measurement")
    return ap.parse_args()


def cpu_model() -> str:
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(work, T, seconds, gpu=None):
    """The fp64 oracle on the host cores, on the same step: attention for every block row and
    head, then acceptance.  Timed three times single-threaded and three times with every
    thread the oracle's OpenMP runtime uses (OMP_NUM_THREADS, else the core count); each
    leg reports the median (a leg stops early once `seconds` have elapsed).

    With ``gpu`` = (attention output, accept_len, next_token) of the timed step on the same
    inputs, the oracle's last results also check them under the parity rule: attention
    max-abs within 2e-2 (bf16) or 1e-5 (fp32); accept_len and next_token equal, except that a
    sequence whose accept test lies within 1e-5 of its threshold is counted and skipped, and a
    final draw within 1e-5 of a CDF edge only has to fall inside the band's tokens."""
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import oracle
    a = work.attn
    acc = work.accept[T]
    q = a.q.float().numpy()
    k = a.k_cache.float().numpy()
    v = a.v_cache.float().numpy()
    tl = acc.target.float().numpy()
    dl = acc.draft.float().numpy() if acc.draft is not None else None
    nthreads = oracle.num_threads()

    def leg(threads):
        oracle.set_threads(threads)
        times, t_start = [], time.perf_counter()
        for _ in range(3):
            t0 = time.perf_counter()
            o_ref = oracle.block_attn(q, k, v, a.ctx_lens, a.block_lens, a.q_offsets, a.mask_mode)
            r = oracle.accept(tl, dl, acc.draft_tokens, acc.uniforms, acc.block_lens, acc.q_offsets, T)
            times.append(time.perf_counter() - t0)
            if time.perf_counter() - t_start >= seconds:
                break
        return float(np.median(times)), times, o_ref, r

    t1, times1, _, _ = leg(1)
    tn, timesn, o_ref, r = leg(nthreads)
    oracle.set_threads(nthreads)
    ntok = work.verified_draft_tokens()
    res = {"value": round(ntok / tn, 1), "unit": "verified draft tokens/s", "cores": nthreads, "kind": "oracle",
           "sample": f"the full step (attention for all {a.total_q} block rows x {a.Hq} heads + acceptance of "
                     f"{a.S} sequences at T={T:g}), median of {len(timesn)} runs at {nthreads} threads: "
                     f"{tn * 1e3:.1f} ms per step",
           "ms_per_step": round(tn * 1e3, 2), "runs_ms": [round(x * 1e3, 2) for x in timesn],
           "single_thread": {"value": round(ntok / t1, 1), "cores": 1, "ms_per_step": round(t1 * 1e3, 2),
                             "runs_ms": [round(x * 1e3, 2) for x in times1]},
           "cpu_model": cpu_model(), "host_cores": os.cpu_count()}
    if gpu is not None:
        attn_gpu, al_g, nt_g = gpu
        err = float(np.abs(attn_gpu.astype(np.float64) - o_ref).max()) if o_ref.size else 0.0
        tol = 2e-2 if a.dtype == "bf16" else 1e-5
        band = 1e-5
        compared = ties_a = ties_s = mism = 0
        for s in range(acc.S):
            if T > 0 and r.accept_margin[s] < band:
                ties_a += 1
                continue
            compared += 1
            ok = al_g[s] == r.accept_len[s]
            if T == 0 or r.sample_margin[s] >= band:
                ok = ok and nt_g[s] == r.next_token[s]
            else:
                ties_s += 1
                ok = ok and r.sample_lo[s] <= nt_g[s] <= r.sample_hi[s]
            mism += int(not ok)
        res["parity"] = {"attn_max_abs": err, "attn_tol": tol, "attn_ok": bool(err <= tol),
                         "accept_compared": compared, "accept_near_ties": ties_a, "sample_near_ties": ties_s,
                         "accept_mismatches": mism,
                         "what": "the timed step's own outputs against the oracle's on the same inputs"}
        if err > tol or mism:
            print(f"bench.py: parity FAILED on the timed step: attention max-abs {err:.3g} (tol {tol}), "
                  f"{mism} acceptance mismatches", file=sys.stderr)
    return res


ROOT = os.path.dirname(os.path.abspath(__file__))
COUNTERS = os.path.join(ROOT, "profiles", "counters_qwen3_4b_ragged_S8_ctx4096_T1.txt")


def kernel_source_hash() -> str:
    """sha256 over the kernel sources and the public header (file names and contents)."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2606_31315_amd", "csrc", "*")))
    files.append(os.path.join(ROOT, "include", "sd_block.h"))
    for f in files:
        h.update(os.path.relpath(f, ROOT).encode())
        h.update(b"\0")
        with open(f, "rb") as fh:
            h.update(fh.read())
        h.update(b"\0")
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per sd_block_attn and per sd_accept call from the committed counter runs
    (FETCH_SIZE and WRITE_SIZE scaled by a plain copy): {"sd_block_attn": n, "sd_accept": n},
    with None for each once the kernel sources have changed since those counters were taken."""
    out = {"sd_block_attn": None, "sd_accept": None}
    try:
        with open(COUNTERS) as fh:
            text = fh.read()
    except OSError:
        return out
    m_h = re.search(r"^source-sha256: ([0-9a-f]{64})$", text, re.M)
    if not m_h or m_h.group(1) != kernel_source_hash():
        return out
    for key in out:
        m_b = re.search(r"^traffic-bytes-per-call %s: (\d+)$" % key, text, re.M)
        out[key] = int(m_b.group(1)) if m_b else None
    return out


def copy_calibration(torch, dev, nbytes=1 << 29, reps=3):
    """A plain device-to-device copy of known size, run before the timed steps.  Its
    FETCH_SIZE / WRITE_SIZE counters in a profiling run scale the counters of the step's
    kernels to bytes; its event-timed rate is reported as the copy rate of this GPU."""
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=dev).normal_()
    dst = torch.empty_like(src)
    dst.copy_(src)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(reps):
        dst.copy_(src)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    del src, dst
    return {"bytes_read": nbytes, "bytes_written": nbytes, "us": round(ms * 1e3, 2),
            "gbps_read_plus_write": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}


def read_ceiling(torch, dev, nbuf=4, nbytes=1 << 28, grids=(256, 512, 1024, 2048, 4096), reps=20):
    """Streaming-read ceiling of this GPU: 16-byte non-temporal loads (libsdbench.so, a
    measurement kernel outside the library) over nbuf rotating buffers of nbytes each (1 GiB
    in all, so the 256 MB Infinity Cache cannot serve them), at several grid sizes.  GB/s of
    bytes read per second of event-timed kernel time; the best grid is the ceiling."""
    import ctypes
    from paper_2606_31315_amd import build_lib
    lib = ctypes.CDLL(build_lib.BENCH_LIB)
    lib.sdbench_stream_read.restype = ctypes.c_int
    lib.sdbench_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_ulonglong, ctypes.c_int, ctypes.c_void_p,
                                        ctypes.c_void_p]
    bufs = [torch.empty(nbytes, dtype=torch.uint8, device=dev).random_() for _ in range(nbuf)]
    sink = torch.zeros(max(grids), dtype=torch.int32, device=dev)
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    res = {}
    for grid in grids:
        def call(i):
            rc = lib.sdbench_stream_read(ctypes.c_void_p(bufs[i % nbuf].data_ptr()), nbytes, grid,
                                         ctypes.c_void_p(sink.data_ptr()), st)
            if rc != 0:
                raise RuntimeError(f"sdbench_stream_read failed ({rc})")
        for i in range(4):
            call(i)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record()
        for i in range(reps):
            call(i)
        t1.record()
        torch.cuda.synchronize()
        res[grid] = nbytes / (t0.elapsed_time(t1) / reps * 1e-3) / 1e9
    del bufs
    torch.cuda.empty_cache()
    best = max(res, key=res.get)
    return {"gbps": round(res[best], 1), "grid": best, "by_grid": {str(g): round(v, 1) for g, v in res.items()},
            "bytes_per_call": nbytes, "buffers": nbuf,
            "what": "16-byte non-temporal loads, 512-thread workgroups each reading one contiguous share, "
                    "rotating over 1 GiB"}


def verify_step_run(torch, sd, work, T, layers, steps, warmup=3):
    """The whole verify step through sd_verify_step: for every layer the block attends over that
    layer's cache and its own keys and values, which the same launch writes into the cache; then
    acceptance and the commit.  Consecutive decode steps: ctx starts at the workload's 4096 and advances by
    accept_len + 1 each step.  Caches and block inputs are random bf16 on the device."""
    a, acc = work.attn, work.accept[T]
    dev = torch.device("cuda:0")
    S, Hq, Hkv, D = a.S, a.Hq, a.Hkv, a.D
    mb = int(a.max_block)
    Lmax = int(a.max_ctx) + mb * (steps + warmup + 1)
    g = torch.Generator(device=dev).manual_seed(7)
    tq = a.total_q
    L = []
    for _ in range(layers):
        L.append(dict(q=torch.randn(tq, Hq, D, device=dev, generator=g).to(torch.bfloat16),
                      k_new=torch.randn(tq, Hkv, D, device=dev, generator=g).to(torch.bfloat16),
                      v_new=torch.randn(tq, Hkv, D, device=dev, generator=g).to(torch.bfloat16),
                      k_cache=torch.randn(S, Hkv, Lmax, D, device=dev, generator=g).to(torch.bfloat16),
                      v_cache=torch.randn(S, Hkv, Lmax, D, device=dev, generator=g).to(torch.bfloat16),
                      out=torch.empty(tq, Hq, D, device=dev, dtype=torch.bfloat16)))
    ctx = torch.from_numpy(a.ctx_lens).to(dev)
    bl, off = torch.from_numpy(a.block_lens).to(dev), torch.from_numpy(a.q_offsets).to(dev)
    t_ = acc.target.to(dev)
    d_ = acc.draft.to(dev) if acc.draft is not None else None
    tok = torch.from_numpy(acc.draft_tokens).to(dev)
    u = torch.from_numpy(acc.uniforms).to(dev)
    al = torch.empty(S, dtype=torch.int32, device=dev)
    nt = torch.empty(S, dtype=torch.int32, device=dev)
    max_ctx = int(a.max_ctx)

    def one(max_ctx):
        sd.verify_step(L, ctx, bl, off, a.mask_mode, t_, d_, tok, u, T, max_ctx=max_ctx, max_block=mb,
                       accept_len=al, next_token=nt)

    for _ in range(warmup):
        one(max_ctx)
        max_ctx += mb
    torch.cuda.synchronize()
    ctx0 = int(ctx.max().item())
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        one(max_ctx)
        max_ctx += mb
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) / steps * 1e3
    return {"layers": layers, "steps": steps, "us_per_step": round(us, 1),
            "verified_draft_tokens_per_s": round(work.verified_draft_tokens() / (us * 1e-6), 1),
            "ctx_start": ctx0, "ctx_end": int(ctx.max().item()),
            "what": "sd_verify_step: per layer sd_block_attn_append (the block's keys and values written into "
                    "the cache by the attention launch), then sd_accept (T=%g) and sd_commit; consecutive decode "
                    "steps" % T}


def policy_run(torch, sd, prompts, reps=20, V=151936, H=2048, radius=2, base_block=16):
    """The block-size policy (softmax of the last-token logits, then the two-hidden-layer MLP
    and the argmax over 2k+1 candidates) on random bf16 weights generated on the device.  The
    weights (622 MB at V=151936, H=2048) exceed the 256 MB Infinity Cache, so every call reads
    them from HBM."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(11)
    C = 2 * radius + 1
    logits = (torch.randn(prompts, V, device=dev, generator=g) * 3).to(torch.bfloat16)
    w1 = torch.randn(H, V, device=dev, generator=g).to(torch.bfloat16)
    w2 = (torch.randn(H, H, device=dev, generator=g) / H ** 0.5).to(torch.bfloat16)
    w3 = (torch.randn(C, H, device=dev, generator=g) / H ** 0.5).to(torch.bfloat16)
    b1, b2 = torch.randn(H, device=dev, generator=g) * 0.05, torch.randn(H, device=dev, generator=g) * 0.05
    b3 = torch.randn(C, device=dev, generator=g) * 0.05
    for _ in range(3):
        sd.block_size_policy(logits, w1, b1, w2, b2, w3, b3, base_block)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        sd.block_size_policy(logits, w1, b1, w2, b2, w3, b3, base_block)
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) / reps * 1e3
    nbytes = 2 * (w1.numel() + w2.numel() + w3.numel()) + logits.numel() * 2
    return {"prompts": prompts, "vocab": V, "hidden": H, "candidates": C, "us_per_call": round(us, 1),
            "bytes": nbytes, "gbps": round(nbytes / (us * 1e-6) / 1e9, 1),
            "hbm_frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "what": "sd_block_size_policy: softmax of the last-token logits, W1 (H x V), W2 (H x H), W3 (2k+1 x H), "
                    "argmax; random bf16 weights"}


def survival_run(torch, sd, N, trials, reps=20):
    """The prefix-survival model over a synthetic population: tau(b; x) for the candidates
    {14, ..., 18} around the training size 16 (alpha = 0.001), B*(x), the regret of a uniformly drawn
    prediction and L_tau (sd_survival_tau), then the Monte-Carlo lengths of 2^16 samples
    (sd_survival_sample)."""
    from paper_2606_31315_amd import workloads as W
    dev = torch.device("cuda:0")
    p = W.make_survival(1006, N=N, P=32, train_block=16, radius=2, alpha=0.001)
    g = torch.from_numpy(p.gamma).to(dev)
    bh = torch.from_numpy(p.b_hat).to(dev)

    def tau_call():
        return sd.survival_tau(g, p.cands, p.train_block, p.alpha, bh)

    for _ in range(3):
        tau_call()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        out = tau_call()
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) / reps * 1e3
    tau, b_star, regret, lip = out
    C = len(p.cands)
    nbytes = N * (p.P * 4 + 4 + C * 8 + 4 + 8 + 8)
    bs = b_star.cpu().numpy()
    reg = regret.cpu().numpy()
    bound = (lip * (b_star - bh).abs().double()).cpu().numpy()
    Nmc = min(N, 1 << 16)
    gmc = g[:Nmc].contiguous()
    sd.survival_sample(gmc, p.cands, p.train_block, p.alpha, 1, trials, hist=False)
    torch.cuda.synchronize()
    t0.record()
    mean, _ = sd.survival_sample(gmc, p.cands, p.train_block, p.alpha, 2, trials, hist=False)
    t1.record()
    torch.cuda.synchronize()
    mc_us = t0.elapsed_time(t1) * 1e3
    gap = (mean - tau[:Nmc]).abs().mean().item()
    return {"samples": N, "candidates": [int(b) for b in p.cands], "tau_us_per_call": round(us, 1),
            "tau_bytes": nbytes, "tau_gbps": round(nbytes / (us * 1e-6) / 1e9, 1),
            "b_star_hist": {int(b): int((bs == b).sum()) for b in p.cands},
            "mean_regret_uniform_prediction": round(float(reg.mean()), 4),
            "regret_bound_holds": bool((reg <= bound + 1e-12).all()),
            "mc_samples": Nmc, "mc_trials": trials, "mc_us": round(mc_us, 1),
            "mc_trials_per_s": round(Nmc * C * trials / (mc_us * 1e-6), 1),
            "mc_mean_abs_mean_minus_tau": round(gap, 4),
            "what": "sd_survival_tau over 2^20 synthetic samples (gamma_x ~ U(0.6, 0.97), 32 positions); "
                    "sd_survival_sample over the first 2^16, Philox4x64-10 draws"}


def c2_run(torch, sd, reps=200):
    """The Qwen3-4B verify step at batch 1 (ctx 2048, B = 16, causal, acceptance at T = 1 over
    V = 151936) on its seeded inputs, rotated over copies totalling >= 1 GB: attention and
    acceptance per call (median of 5 batches), the step, and algorithmic GB/s."""
    from paper_2606_31315_amd import workloads as W
    dev = torch.device("cuda:0")
    w = W.c2_qwen3_4b_verify(temperatures=(1.0,))
    a, acc = w.attn, w.accept[1.0]
    attn_bytes, acc_bytes = a.kv_bytes() + a.qo_bytes(), acc.logit_bytes()
    copies = max(2, int(np.ceil(1.0e9 / (attn_bytes + acc_bytes))))
    bufs = [dict(q=a.q.to(dev), k=a.k_cache.to(dev), v=a.v_cache.to(dev), t=acc.target.to(dev),
                 d=acc.draft.to(dev)) for _ in range(copies)]
    ctx, bl, off = (torch.from_numpy(x).to(dev) for x in (a.ctx_lens, a.block_lens, a.q_offsets))
    tok, u = torch.from_numpy(acc.draft_tokens).to(dev), torch.from_numpy(acc.uniforms).to(dev)
    o = torch.empty_like(bufs[0]["q"])
    al = torch.empty(a.S, dtype=torch.int32, device=dev)
    nt = torch.empty(a.S, dtype=torch.int32, device=dev)

    def attn(i):
        b = bufs[i % copies]
        sd.block_attn(b["q"], b["k"], b["v"], ctx, bl, off, a.mask_mode, max_ctx=a.max_ctx, max_block=a.max_block,
                      out=o)

    def accept(i):
        b = bufs[i % copies]
        sd.accept(b["t"], b["d"], tok, u, bl, off, 1.0, max_block=a.max_block, accept_len=al, next_token=nt)

    def step(i):
        attn(i)
        accept(i)

    for i in range(20):
        step(i)
    a_us, c_us, s_us = (batched_us(torch, fn, reps) for fn in (attn, accept, step))
    del bufs
    torch.cuda.empty_cache()
    med = lambda x: float(np.median(x))
    return {"num_seqs": a.S, "ctx": int(a.ctx_lens[0]), "block_len": int(a.block_lens[0]), "temperature": 1.0,
            "attn_us": round(med(a_us), 2), "attn_bytes": attn_bytes,
            "attn_gbps": round(attn_bytes / (med(a_us) * 1e-6) / 1e9, 1),
            "accept_us": round(med(c_us), 2), "accept_bytes": acc_bytes,
            "accept_gbps": round(acc_bytes / (med(c_us) * 1e-6) / 1e9, 1),
            "step_us": round(med(s_us), 2),
            "step_gbps": round((attn_bytes + acc_bytes) / (med(s_us) * 1e-6) / 1e9, 1),
            "step_hbm_frac": round((attn_bytes + acc_bytes) / (med(s_us) * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "verified_draft_tokens_per_s": round(w.verified_draft_tokens() / (med(s_us) * 1e-6), 1),
            "input_copies": copies,
            "what": "Qwen3-4B verify step, batch 1 (seeded inputs): latency-bound at 18 MB per step"}


def batched_us(torch, fn, n, nb=5):
    """Mean us per call of each of nb batches of n // nb back-to-back calls (events on the
    launch stream)."""
    per = max(1, n // nb)
    out = []
    for b in range(nb):
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record()
        for i in range(per):
            fn(b * per + i)
        t1.record()
        torch.cuda.synchronize()
        out.append(t0.elapsed_time(t1) / per * 1e3)
    return out


def other_configs_run(torch, sd, reps=200):
    """The drafter pass (16 sequences, ctx U{1024..8192}, B U{8..32}, bidirectional) and the
    long-context serving step (32 sequences, ctx U{8192..32768}, B U{4..32}, causal attention,
    then acceptance at T = 1 over V = 151936), with the seeded lengths of those workloads and
    random bf16 values generated on the device.  Per-call times and algorithmic GB/s."""
    from paper_2606_31315_amd import workloads as W
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(17)
    Hq, Hkv, D, V = 32, 8, 128, 151936
    out = {"qwen3_4b_verify_S1_ctx2048_B16": c2_run(torch, sd)}

    def timed(fn, n):
        # 20 untimed calls first: a GPU that has idled runs its first few milliseconds of work
        # several percent slower while its clocks come back up
        for i in range(20):
            fn(i)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for i in range(n):
            fn(i)
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / n * 1e3

    for name, (ctx, B), mask, Lmax, copies in (
            ("drafter_bidir_S16_ctx1k-8k_B8-32", W.c4_lens(), 1, 8192 + 32, 3),
            ("qwen3_8b_long_S32_ctx8k-32k_B4-32", W.c5_lens(), 0, 32768 + 32, 1)):
        S = len(ctx)
        off = np.concatenate([[0], np.cumsum(B)]).astype(np.int32)
        tq = int(off[-1])
        bufs = [dict(q=torch.randn(tq, Hq, D, device=dev, generator=g).to(torch.bfloat16),
                     k=torch.randn(S, Hkv, Lmax, D, device=dev, generator=g).to(torch.bfloat16),
                     v=torch.randn(S, Hkv, Lmax, D, device=dev, generator=g).to(torch.bfloat16)) for _ in range(copies)]
        o = torch.empty_like(bufs[0]["q"])
        dc, db, do = (torch.from_numpy(x).to(dev) for x in (ctx, B, off))
        mc, mb = int(ctx.max()), int(B.max())

        def attn(i=0):
            b = bufs[i % copies]
            sd.block_attn(b["q"], b["k"], b["v"], dc, db, do, mask, max_ctx=mc, max_block=mb, out=o)

        us = timed(attn, reps)
        nbytes = int(((ctx + B).astype(np.int64) * Hkv * D * 2 * 2).sum() + 2 * tq * Hq * D * 2)
        rec = {"num_seqs": S, "mask": "bidirectional_in_block" if mask else "causal_in_block",
               "attn_us": round(us, 1), "attn_bytes": nbytes, "attn_gbps": round(nbytes / (us * 1e-6) / 1e9, 1)}
        del bufs
        if mask == 0:
            t_ = (torch.randn(tq, V, device=dev, generator=g) * 3).to(torch.bfloat16)
            d_ = (t_[:tq - S].float() + torch.randn(tq - S, V, device=dev, generator=g)).to(torch.bfloat16)
            tok = torch.randint(0, V, (tq - S,), device=dev, generator=g, dtype=torch.int32)
            u = torch.rand(tq, device=dev, generator=g)
            al = torch.empty(S, dtype=torch.int32, device=dev)
            nt = torch.empty(S, dtype=torch.int32, device=dev)

            def acc(i=0):
                sd.accept(t_, d_, tok, u, db, do, 1.0, max_block=mb, accept_len=al, next_token=nt)

            aus = timed(acc, reps)
            abytes = (2 * tq - S) * V * 2
            rec.update({"accept_us": round(aus, 1), "accept_bytes": abytes,
                        "accept_gbps": round(abytes / (aus * 1e-6) / 1e9, 1)})
            del t_, d_
        out[name] = rec
        torch.cuda.empty_cache()
    return out


def paged_run(torch, sd, a, bufs, page_size, reps, shuffle=True):
    """sd_block_attn_paged on the same keys and values as the timed step, scattered over a pool
    of page_size-key pages in a shuffled (or in-order) page order, one pool per input copy."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(13)
    S, Hkv, Lmax, D = bufs[0]["k"].shape
    mp = (Lmax + page_size - 1) // page_size
    pools = []
    for b in bufs:
        perm = (torch.randperm(S * mp, device=dev, generator=g) if shuffle
                else torch.arange(S * mp, device=dev))
        pk = []
        for name in ("k", "v"):
            x = torch.nn.functional.pad(b[name], (0, 0, 0, mp * page_size - Lmax))
            x = x.reshape(S, Hkv, mp, page_size, D).permute(0, 2, 1, 3, 4).reshape(S * mp, Hkv, page_size, D)
            pool = torch.empty_like(x)
            pool[perm] = x
            pk.append(pool)
        pools.append((pk[0], pk[1], perm.to(torch.int32).reshape(S, mp).contiguous()))
    ctx = torch.from_numpy(a.ctx_lens).to(dev)
    bl, off = torch.from_numpy(a.block_lens).to(dev), torch.from_numpy(a.q_offsets).to(dev)
    out = torch.empty_like(bufs[0]["q"])

    def call(i):
        kp, vp, tab = pools[i % len(pools)]
        sd.block_attn_paged(bufs[i % len(bufs)]["q"], kp, vp, tab, ctx, bl, off, a.mask_mode, max_ctx=a.max_ctx,
                            max_block=a.max_block, out=out)

    for i in range(10):
        call(i)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(reps):
        call(i)
    t1.record()
    torch.cuda.synchronize()
    return round(t0.elapsed_time(t1) / reps * 1e3, 2)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        return 2
    import torch
    import paper_2606_31315_amd as sd
    from paper_2606_31315_amd import workloads as W

    T = float(args.temperature)
    copy_cal = copy_calibration(torch, torch.device("cuda:0"))
    ceiling = read_ceiling(torch, torch.device("cuda:0"))
    temps = tuple(sorted({T}))
    work = W.c3_ragged(temperatures=temps)
    a = work.attn
    acc = work.accept[T]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    attn_bytes = a.kv_bytes() + a.qo_bytes()
    acc_bytes = acc.logit_bytes()
    step_bytes = attn_bytes + acc_bytes
    copies = args.copies or max(2, int(np.ceil(1.0e9 / step_bytes)))

    def upload():
        d = dict(q=a.q.to(dev), k=a.k_cache.to(dev), v=a.v_cache.to(dev), t=acc.target.to(dev))
        d["d"] = acc.draft.to(dev) if acc.draft is not None else None
        return d

    small = dict(ctx=torch.from_numpy(a.ctx_lens).to(dev), bl=torch.from_numpy(a.block_lens).to(dev),
                 off=torch.from_numpy(a.q_offsets).to(dev),
                 tok=torch.from_numpy(acc.draft_tokens).to(dev), u=torch.from_numpy(acc.uniforms).to(dev))
    bufs = [upload() for _ in range(copies)]
    outs = [torch.empty_like(bufs[0]["q"]) for _ in range(copies)]
    al = torch.empty(a.S, dtype=torch.int32, device=dev)
    nt = torch.empty(a.S, dtype=torch.int32, device=dev)
    ws_attn = torch.zeros(sd.attn_workspace_size(sd.attn_shape(bufs[0]["q"], bufs[0]["k"], a.max_ctx, a.max_block)),
                          dtype=torch.uint8, device=dev)
    ws_acc = torch.zeros(sd.accept_workspace_size(sd.accept_shape(bufs[0]["t"], a.S, a.max_block), T),
                         dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def attn_call(i):
        b = bufs[i % copies]
        sd.block_attn(b["q"], b["k"], b["v"], small["ctx"], small["bl"], small["off"], a.mask_mode,
                      max_ctx=a.max_ctx, max_block=a.max_block, out=outs[i % copies], workspace=ws_attn)

    def accept_call(i):
        b = bufs[i % copies]
        sd.accept(b["t"], b["d"], small["tok"], small["u"], small["bl"], small["off"], T, max_block=a.max_block,
                  accept_len=al, next_token=nt, workspace=ws_acc)

    def step(i):
        attn_call(i)
        accept_call(i)

    def timed(fn, n):
        """Mean ms per call of n back-to-back calls on the launch stream (torch's current
        stream, which the binding launches on), between two events."""
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record()
        for i in range(n):
            fn(i)
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / n

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # timed region: exactly K whole steps, nothing else on the stream
    K = args.steps
    ms_per_step = timed(step, K)
    # Legs after the timed region (never part of value) run at least 200 calls: each batch
    # starts from an idle stream, so a short batch would mostly measure the host's enqueue
    # latency of its first call (about 13 us), not the kernels.
    KI = max(K, 200)
    # spread: the same steps again in 5 batches; per-call durations: KI calls of each operation
    # back to back in 5 batches (an event between every call would add a few microseconds of
    # its own to each); each reported as the median batch mean with the batch range
    step_b = batched_us(torch, step, KI)
    attn_b = batched_us(torch, attn_call, KI)
    acc_b = batched_us(torch, accept_call, KI)
    attn_us, acc_us = float(np.median(attn_b)), float(np.median(acc_b))

    ntok = work.verified_draft_tokens()
    value = ntok / (ms_per_step * 1e-3)
    attn_gbps = attn_bytes / (attn_us * 1e-6) / 1e9
    acc_gbps = acc_bytes / (acc_us * 1e-6) / 1e9
    step_gbps = step_bytes / (ms_per_step * 1e-3) / 1e9
    al_h, nt_h = al.cpu().numpy(), nt.cpu().numpy()
    attn_h = outs[0].float().cpu().numpy()

    traffic = measured_traffic()
    rc_gbps = ceiling["gbps"]

    def call_entry(us, nbytes, kernels, tr):
        gbps = nbytes / (us * 1e-6) / 1e9
        return {"kernels": kernels, "us": round(us, 2), "algorithmic_bytes": int(nbytes), "achieved": round(gbps, 1),
                "frac": round(gbps / HBM_PEAK_GBPS, 4), "frac_of_read_ceiling": round(gbps / rc_gbps, 4),
                "traffic": tr}

    step_traffic = (traffic["sd_block_attn"] + traffic["sd_accept"]
                    if traffic["sd_block_attn"] is not None and traffic["sd_accept"] is not None else None)
    res = {
        "metric": METRIC, "value": round(value, 1), "unit": "verified draft tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 6), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": work.name, "num_seqs": a.S, "q_heads": a.Hq, "kv_heads": a.Hkv, "head_dim": a.D,
                   "ctx": int(a.ctx_lens[0]), "block_lens": [int(b) for b in a.block_lens], "vocab": acc.V,
                   "temperature": T, "mask": "causal_in_block", "layers_timed": 1, "input_copies": copies},
        "step_gbps": round(step_gbps, 1), "step_hbm_frac": round(step_gbps / HBM_PEAK_GBPS, 4),
        "step_us_batches": [round(x, 2) for x in step_b],
        "attn_us": round(attn_us, 2), "attn_gbps": round(attn_gbps, 1),
        "attn_us_batches": [round(x, 2) for x in attn_b],
        "accept_us": round(acc_us, 2), "accept_gbps": round(acc_gbps, 1),
        "accept_us_batches": [round(x, 2) for x in acc_b],
        "bytes": {"attn": attn_bytes, "accept": acc_bytes, "step": step_bytes},
        "verify_rows_per_s": round(a.total_q / (ms_per_step * 1e-3), 1),
        "committed_tokens_per_s": round(float((al_h + 1).sum()) / (ms_per_step * 1e-3), 1),
        "mean_accept_len": float(al_h.mean()),
        "copy_calibration": copy_cal,
        "read_ceiling": ceiling,
        # the metric's unit is the step: algorithmic bytes of one attention call and one
        # acceptance call over the step's event-timed duration; per call below, each with its
        # counter-measured HBM traffic
        "roofline": {"bound": "hbm", "scope": "step = sd_block_attn (one layer) + sd_accept",
                     "achieved": round(step_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(step_gbps / HBM_PEAK_GBPS, 4), "traffic": step_traffic,
                     "read_ceiling_gbps": rc_gbps, "frac_of_read_ceiling": round(step_gbps / rc_gbps, 4),
                     "per_call": {
                         "sd_block_attn": call_entry(attn_us, attn_bytes,
                                                     "block_attn_bf16_kernel + block_attn_merge_kernel",
                                                     traffic["sd_block_attn"]),
                         "sd_accept": call_entry(acc_us, acc_bytes,
                                                 "accept_stats_kernel + accept_draw_kernel",
                                                 traffic["sd_accept"])}},
    }
    # rows a sequential acceptance would have read: target rows 0..accept_len and the drafts
    # tested up to the first rejection (the data-parallel pass reads every row)
    B_h = a.block_lens.astype(np.int64)
    useful_rows = int((al_h + 1).sum() + (np.minimum(al_h + 1, B_h - 1) if T > 0 else 0 * B_h).sum())
    res["accept_useful_bytes"] = useful_rows * acc.V * 2
    # the same step with greedy acceptance (T = 0): same target logits, drafts = the drafter's argmax
    acc0 = W.c3_ragged(temperatures=(0.0,), with_attn=False, dtype="bf16").accept[0.0]
    tok0 = torch.from_numpy(acc0.draft_tokens).to(dev)
    al0 = torch.empty_like(al)
    nt0 = torch.empty_like(nt)

    def step0(i):
        attn_call(i)
        sd.accept(bufs[i % copies]["t"], None, tok0, None, small["bl"], small["off"], 0.0, max_block=a.max_block,
                  accept_len=al0, next_token=nt0, workspace=ws_acc)

    for i in range(args.warmup):
        step0(i)
    ms0 = timed(step0, KI)
    acc0_bytes = acc0.logit_bytes()
    al0_h = al0.cpu().numpy()
    gbps0 = (attn_bytes + acc0_bytes) / (ms0 * 1e-3) / 1e9
    res["t0"] = {"ms_per_step": round(ms0, 6), "verified_draft_tokens_per_s": round(ntok / (ms0 * 1e-3), 1),
                 "accept_bytes": acc0_bytes, "accept_useful_bytes": int((al0_h + 1).sum()) * acc0.V * 2,
                 "step_gbps": round(gbps0, 1), "step_hbm_frac": round(gbps0 / HBM_PEAK_GBPS, 4),
                 "frac_of_read_ceiling": round(gbps0 / rc_gbps, 4),
                 "what": "the same step with greedy acceptance (T = 0): every target row read once"}
    res["paged_attn_us"] = {f"page_{ps}_shuffled": paged_run(torch, sd, a, bufs, ps, KI) for ps in (16, 64, 256)}
    res["paged_attn_us"]["page_64_in_order"] = paged_run(torch, sd, a, bufs, 64, KI, shuffle=False)
    if args.policy_prompts > 0:
        res["policy"] = policy_run(torch, sd, args.policy_prompts)
    if args.other_configs:
        res["other_configs"] = other_configs_run(torch, sd)
    if args.survival_samples > 0:
        res["survival"] = survival_run(torch, sd, args.survival_samples, args.survival_trials)
    if args.verify_layers > 0:
        res["verify_step"] = verify_step_run(torch, sd, work, T, args.verify_layers, args.verify_steps)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(work, T, args.cpu_seconds, gpu=(attn_h, al_h, nt_h))
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
