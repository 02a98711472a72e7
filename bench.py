#!/usr/bin/env python3
"""Paged-attention benchmark on one MI355X.

A step is one pa_forward_hinted call over one batch (every kernel of the
path: decode split-KV + log-sum-exp merge for single-token rows, the Q-block
kernel for the rest; the hint is what the host knows of the batch, the
number of single-token rows and the longest query, and only drops launches
that would find no work), inputs resident in HBM.  The plain pa_forward
time is reported next to it.  The headline workload is the
Llama-3-8B-shaped decode batch (64 sequences, context U[512, 8192], Hq 32 /
Hkv 8, d 128, bf16, block size 16); the other four benchmark batches are
measured in the same run and reported under "configs".

Algorithmic work per batch (what the method must move / compute):
  bytes = sum_i L_i*Hkv*d*2*b_kv + 2*T*Hq*d*2 + sum_i ceil(L_i/bs)*4 + (2S+1)*4
  flops = 4*d*Hq*sum_i sum_j (c_i + j + 1)
Roofline peaks: HBM 8.0 TB/s, dense bf16 MFMA 2516.6 TFLOP/s.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config k]
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2516.6
METRIC = "paged-attn decode HBM GB/s & prefill TFLOP/s (% of MI355X roofline), µs/batch"
# Parity tolerances against the fp64 oracle (max / mean abs error of the
# bf16 output): bf16 caches, fp8 e4m3 caches.
TOL_BF16 = (2e-2, 2e-3)
TOL_FP8 = (5e-2, 5e-3)


def alg_bytes(w):
    b_kv = 1 if w.kv_fp8 else 2
    L = w.seq_len_list
    T = sum(w.q_lens)
    return (sum(L) * w.num_kv_heads * w.head_dim * 2 * b_kv + 2 * T * w.num_q_heads * w.head_dim * 2
            + sum(-(-x // w.block_size) for x in L) * 4 + (2 * w.num_seqs + 1) * 4)


def alg_flops(w):
    pairs = sum(q * c + q * (q + 1) // 2 for c, q in zip(w.ctx_lens, w.q_lens))
    return 4 * w.head_dim * w.num_q_heads * pairs


def decode_bytes(w):
    """Bytes of the single-token (decode) rows only."""
    b_kv = 1 if w.kv_fp8 else 2
    L = [c + q for c, q in zip(w.ctx_lens, w.q_lens) if q == 1]
    return (sum(L) * w.num_kv_heads * w.head_dim * 2 * b_kv + 2 * len(L) * w.num_q_heads * w.head_dim * 2
            + sum(-(-x // w.block_size) for x in L) * 4)


def prefill_flops(w):
    pairs = sum(q * c + q * (q + 1) // 2 for c, q in zip(w.ctx_lens, w.q_lens) if q >= 2)
    return 4 * w.head_dim * w.num_q_heads * pairs


KERNEL_SOURCES = {
    "decode_kernel": ("decode.hip", "common.hpp", "kernels.h"),
    "qblock_kernel": ("qblock.hip", "common.hpp", "kernels.h"),
}


def kernel_source_hash(kernel):
    """sha256 over the source files a kernel is built from."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2511_11581_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def rocprof_record(key, workload):
    """The rocprofv3 record of kernel `key` ("decode_kernel", "qblock_kernel",
    "@fp8" for fp8 caches) on `workload` in profiles/traffic.json: HBM bytes
    per launch from the FETCH_SIZE / WRITE_SIZE runs (each counter scaled by
    what it reads for a plain device copy of known size), the trace's
    average duration and, for the Q-block kernel, the matrix-core busy
    fraction.  None when no record exists or the kernel's sources have
    changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
        k = rec["kernels"][key]
    except (OSError, KeyError, ValueError):
        return None
    if k.get("workload") != workload or k.get("source_sha256") != kernel_source_hash(key.split("@")[0]):
        return None
    cal = rec["calibration"]
    out = {"kernel": key.split("@")[0],
           "dram_bytes": k["fetch_kib"] * 1024 * cal["fetch_scale"] + k["write_kib"] * 1024 * cal["write_scale"],
           "avg_us_trace": k.get("avg_us_trace")}
    if "mfma_busy_frac" in k:
        out["mfma_busy"] = k["mfma_busy_frac"]
    return out


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` (rocprof_record), or None."""
    r = rocprof_record(kernel, workload)
    return r["dram_bytes"] if r else None


def make_attention(w, profile=False, no_split_kv=False):
    from paper_2511_11581_amd import pa
    return pa.PagedAttention(w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size,
                             w.k_cache.dtype, w.k_scale, w.v_scale, max_tokens=w.num_tokens,
                             max_seqs=w.num_seqs, max_blocks_per_seq=int(w.block_table.shape[1]),
                             profile=profile, no_split_kv=no_split_kv)


def hint_of(w):
    """What the host knows of the batch (pa_forward_hinted): the number of
    single-token rows and the longest query."""
    return (sum(1 for q in w.q_lens if q == 1), max(w.q_lens + [0]))


def time_steps(w, att, out, steps, warmup, hint=None):
    """Mean ms per step over `steps` back-to-back calls, events on the launch
    stream around all of them."""
    import torch
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc)
    for _ in range(warmup):
        att.forward(*args, w.scale, out=out, hint=hint)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        att.forward(*args, w.scale, out=out, hint=hint)
    ev1.record()
    torch.cuda.synchronize()
    return ev0.elapsed_time(ev1) / steps


def per_call_ms(w, att, out, steps, hint=None):
    """Per-call durations (an event pair around each call): median, min, max."""
    import torch
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record()
        att.forward(*args, w.scale, out=out, hint=hint)
        e1.record()
    torch.cuda.synchronize()
    t = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    return {"median": t[len(t) // 2], "min": t[0], "max": t[-1]}


def time_graph(w, att, out, steps, warmup, hint=None, calls_per_graph=16):
    """Mean ms per pa_forward call replayed from a HIP graph that holds
    `calls_per_graph` calls (as a model's forward graph holds one attention
    call per layer): the host's per-call work is gone and the graph launch
    is shared by the calls; the same kernels and work."""
    import torch
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        att.forward(*args, w.scale, out=out, hint=hint)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(calls_per_graph):
            att.forward(*args, w.scale, out=out, hint=hint)
    for _ in range(max(1, warmup // calls_per_graph)):
        g.replay()
    torch.cuda.synchronize()
    reps = max(2, steps // calls_per_graph)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(reps):
        g.replay()
    ev1.record()
    torch.cuda.synchronize()
    del g
    return ev0.elapsed_time(ev1) / (reps * calls_per_graph)


def per_kernel_ms(w, out, steps, warmup, hint=None):
    """Average duration of each kernel (HIP events recorded by the library
    around every launch on the same stream)."""
    import torch
    att = make_attention(w, profile=True)
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc)
    for _ in range(warmup):
        att.forward(*args, w.scale, out=out, hint=hint)
    torch.cuda.synchronize()
    att.profile(reset=True)
    for _ in range(steps):
        att.forward(*args, w.scale, out=out, hint=hint)
    prof = att.profile(reset=True)
    att.close()
    return {k: (tot / n if n else 0.0) for k, (n, tot) in prof.items()}


def sampled_error(w, out, nrows=256, seed=0):
    """Max / mean abs error of `out` against the fp64 oracle on sampled rows
    (first and last token of every sequence plus random ones; every row of
    every batch is compared in the GPU tests)."""
    import numpy as np
    import oracle
    wc = w.to("cpu")
    qsl = wc.query_start_loc.tolist()
    rng = np.random.default_rng(seed)
    rows = set()
    for i in range(len(qsl) - 1):
        if qsl[i + 1] > qsl[i]:
            rows.add((qsl[i], int(rng.integers(w.num_q_heads))))
            rows.add((qsl[i + 1] - 1, int(rng.integers(w.num_q_heads))))
    nrows = min(nrows, qsl[-1] * w.num_q_heads)   # a batch may hold fewer rows
    while len(rows) < nrows:
        rows.add((int(rng.integers(qsl[-1])), int(rng.integers(w.num_q_heads))))
    rows = sorted(rows)
    import concurrent.futures as cf
    nt = oracle.default_threads()
    chunks = np.array_split(np.asarray(rows, dtype=np.int64), min(nt, len(rows)))

    def one(ch):
        return oracle.rows(wc.q, wc.k_cache, wc.v_cache, wc.block_table, wc.seq_lens,
                           wc.query_start_loc, wc.scale, ch, k_scale=wc.k_scale, v_scale=wc.v_scale)

    t_or = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=len(chunks)) as ex:
        ref = np.concatenate(list(ex.map(one, chunks)), 0)
    t_or = time.perf_counter() - t_or
    got = out.cpu()
    g = np.stack([got[t, h].double().numpy() for t, h in rows])
    err = np.abs(g - ref)
    tol = TOL_FP8 if w.kv_fp8 else TOL_BF16
    mx, mn = float(err.max()), float(err.mean())
    return {"rows": len(rows), "max_abs_err": mx, "mean_abs_err": mn,
            "tolerance": {"max": tol[0], "mean": tol[1]}, "pass": bool(mx <= tol[0] and mn <= tol[1]),
            "oracle_s": t_or, "oracle_threads": len(chunks)}


def measure(k, steps, warmup, block_size=None, with_error=True, kv_dtype=None):
    import torch
    from paper_2511_11581_amd import workloads as W
    if block_size is None and kv_dtype is None:
        w = W.make_config(k, device="cuda", poison=False)
    else:   # the same batch on pages of another size, or in a cache of another dtype
        seqs, kw, gen, seed = W.config_seqs(k)
        kw = dict(kw)
        if kv_dtype is not None:
            kw["kv_dtype"] = kv_dtype
        bs = block_size if block_size is not None else 16
        w = W.make_batch(seqs, seed=seed, device="cuda", poison=False, block_size=bs,
                         name=f"config{k}-bs{bs}-{kw.get('kv_dtype', 'bf16')}", _gen=gen, **kw)
    att = make_attention(w)
    out = torch.empty_like(w.q)
    hint = hint_of(w)
    ms = time_steps(w, att, out, steps, warmup)
    ms_h = time_steps(w, att, out, steps, warmup, hint)
    calls = per_call_ms(w, att, out, steps, hint)
    gms = time_graph(w, att, out, steps, warmup)
    gms_h = time_graph(w, att, out, steps, warmup, hint)
    kms = per_kernel_ms(w, out, steps, warmup, hint)
    plan = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]))
    err = sampled_error(w, out, seed=k) if with_error else None
    att.close()
    B, F = alg_bytes(w), alg_flops(w)
    res = {
        "config": k, "name": W.CONFIG_NAMES[k], "seed": w.seed, "sum_L": sum(w.seq_len_list),
        "block_size": w.block_size,
        "us_per_batch": ms_h * 1e3, "us_per_batch_unhinted": ms * 1e3,
        "us_median": calls["median"] * 1e3, "us_min": calls["min"] * 1e3, "us_max": calls["max"] * 1e3,
        "graph_us_per_batch": gms_h * 1e3, "graph_us_per_batch_unhinted": gms * 1e3,
        "graph_calls_per_replay": 16,
        "hint": {"num_decode_seqs": hint[0], "max_query_len": hint[1]},
        "alg_bytes": B, "alg_flops": F,
        "GBps": B / (ms_h * 1e-3) / 1e9, "TFLOPs": F / (ms_h * 1e-3) / 1e12,
        "per_kernel_us": {kk: v * 1e3 for kk, v in kms.items() if v > 0},
        "plan": {kk: plan[kk] for kk in ("decode_step", "decode_workers", "decode_min_steps",
                                         "block_m", "block_q", "decode_grid", "prefill_grid")},
    }
    if err:
        res["error_vs_oracle"] = err
    # the rocprofv3 record of the batch's dominant kernel, where one was taken
    rkey = {2: "decode_kernel", 3: "qblock_kernel", 5: "decode_kernel"}.get(k) if block_size is None else None
    if rkey is not None:
        wname = W.CONFIG_NAMES[k] + (" (fp8 e4m3 caches)" if kv_dtype is not None and k == 3 else "")
        rp = rocprof_record(rkey + ("@fp8" if w.kv_fp8 else ""), wname)
        if rp is not None:
            res["rocprof"] = rp
    res["frac_hbm"] = res["GBps"] / HBM_PEAK_GBS
    res["frac_mfma"] = res["TFLOPs"] / BF16_PEAK_TFLOPS
    db, pf = decode_bytes(w), prefill_flops(w)
    if kms.get("decode", 0) > 0 and db > 0:
        res["decode_kernel_GBps"] = db / (kms["decode"] * 1e-3) / 1e9
    if kms.get("prefill", 0) > 0 and pf > 0:
        res["prefill_kernel_TFLOPs"] = pf / (kms["prefill"] * 1e-3) / 1e12
    return w, res


def measure_cache_write(kv, steps, warmup, T=4216, Hkv=8, d=128, bs=16):
    """pa_cache_write of the mixed batch's 4216 new tokens (Hkv 8, d 128) into a
    pool of random slots: us per call and GB/s over the bytes it must move
    (K and V read as bf16, written as bf16 or fp8)."""
    import torch
    from paper_2511_11581_amd import pa
    FP8 = torch.float8_e4m3fn
    g = torch.Generator(device="cuda").manual_seed(4216)
    NB = (T + bs - 1) // bs * 4
    key = torch.randn(T, Hkv, d, device="cuda", generator=g).bfloat16()
    value = torch.randn(T, Hkv, d, device="cuda", generator=g).bfloat16()
    slots = torch.randperm(NB * bs, device="cuda", generator=g)[:T].to(torch.int32)
    cdt = FP8 if kv == "fp8" else torch.bfloat16
    kc = torch.zeros(NB, bs, Hkv, d, device="cuda", dtype=torch.bfloat16).to(cdt)
    vc = torch.zeros_like(kc)
    att = pa.PagedAttention(4 * Hkv, Hkv, d, bs, kv_dtype=cdt, k_scale=0.03, v_scale=0.03,
                            max_tokens=T, max_seqs=1, max_blocks_per_seq=1)
    for _ in range(warmup):
        att.cache_write(key, value, slots, kc, vc)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        att.cache_write(key, value, slots, kc, vc)
    e1.record()
    torch.cuda.synchronize()
    us_eager = e0.elapsed_time(e1) * 1e3 / steps
    # the same call replayed from a HIP graph: the GPU time without the
    # per-call host work (argument checks, marshalling) between launches
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        att.cache_write(key, value, slots, kc, vc, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    reps = 20
    with torch.cuda.graph(graph):
        for _ in range(reps):
            att.cache_write(key, value, slots, kc, vc, stream=torch.cuda.current_stream())
    graph.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(max(1, steps // reps)):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (max(1, steps // reps) * reps)
    nbytes = T * Hkv * d * 2 * (2 + (1 if kv == "fp8" else 2)) + T * 4
    return {"tokens": T, "kv_heads": Hkv, "head_dim": d, "kv": kv, "us": us, "us_eager": us_eager,
            "GBps": nbytes / (us * 1e-6) / 1e9, "frac_hbm": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS}


def measure_ladder(steps=20, warmup=3):
    """The paper's optimisation ladder (Sec. 7) on this GPU, three rungs: the
    baseline decomposition (one wave per (token, q head), one page per tile),
    Q-blocks without the split-KV decode kernel (single-token rows as
    Q-blocks of one token, no split, no merge), and the full path (the hinted
    call: the launcher picks split-KV decode + merge + Q-blocks, or, for a
    mixed batch whose Q-blocks fit one round of workgroups, every row as
    Q-blocks); for 16 sequences (ctx U[512, 4096], Hq 32 / Hkv 8, d 128,
    bf16) whose decode share is 0, 50 or 100 % (decode rows q = 1, the
    others chunked prefill q = 128).  Relative numbers only."""
    import torch
    from paper_2511_11581_amd import workloads as W
    g = torch.Generator().manual_seed(805)
    ctxs = torch.randint(512, 4097, (16,), generator=g).tolist()
    res = {}
    for share in (0, 50, 100):
        nd = 16 * share // 100
        seqs = [(c, 1) for c in ctxs[:nd]] + [(c, 128) for c in ctxs[nd:]]
        w = W.make_batch(seqs, 32, 8, 128, seed=805 + share, name=f"ladder{share}", device="cuda",
                         poison=False)
        att = make_attention(w)
        att_nosplit = make_attention(w, no_split_kv=True)
        out = torch.empty_like(w.q)
        timings = {}
        hint = hint_of(w)
        full = lambda *a, **kw: att.forward(*a, hint=hint, **kw)
        for rung, fn in (("baseline", att.forward_baseline), ("qblock", att_nosplit.forward),
                         ("full", full)):
            for _ in range(warmup):
                fn(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc,
                   w.scale, out=out)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(steps):
                fn(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc,
                   w.scale, out=out)
            e1.record()
            torch.cuda.synchronize()
            timings[rung + "_us"] = e0.elapsed_time(e1) * 1e3 / steps
        timings["baseline_over_qblock"] = timings["baseline_us"] / timings["qblock_us"]
        timings["qblock_over_full"] = timings["qblock_us"] / timings["full_us"]
        timings["speedup"] = timings["baseline_us"] / timings["full_us"]
        route = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]), hint)
        if route["prefill_qmin"] == 1:
            timings["full_route"] = "every row as Q-blocks, one launch"
        elif hint[0] == 0:
            timings["full_route"] = "Q-blocks"
        elif hint[1] < 2:
            timings["full_route"] = "split-KV decode"
        else:
            timings["full_route"] = "split-KV decode, then Q-blocks"
        res[str(share)] = timings
        att.close()
        att_nosplit.close()
        del w, att, att_nosplit, out
        torch.cuda.empty_cache()
    return res


def cpu_baseline(w, budget_s=15.0, flops=False):
    """The fp64 oracle on the host cores over the first m sequences of the
    batch (m chosen so the run takes about budget_s), in the headline's unit
    (GB/s of algorithmic bytes, or TFLOP/s of algorithmic flops)."""
    import oracle
    import dataclasses
    wc = w.to("cpu")
    threads = oracle.default_threads()

    def sub(m):
        t_end = int(wc.query_start_loc[m])
        return dataclasses.replace(
            wc, q=wc.q[:t_end].contiguous(), block_table=wc.block_table[:m].contiguous(),
            seq_lens=wc.seq_lens[:m].contiguous(), query_start_loc=wc.query_start_loc[:m + 1].contiguous(),
            ctx_lens=wc.ctx_lens[:m], q_lens=wc.q_lens[:m])

    def run(s):
        t = time.perf_counter()
        oracle.forward(s.q, s.k_cache, s.v_cache, s.block_table, s.seq_lens, s.query_start_loc,
                       s.scale, k_scale=s.k_scale, v_scale=s.v_scale, threads=threads)
        return time.perf_counter() - t

    probe = sub(min(threads, w.num_seqs))
    tp = run(probe)
    per_seq = tp / probe.num_seqs
    m = max(1, min(w.num_seqs, int(budget_s / max(per_seq, 1e-6))))
    s = sub(m)
    t = run(s) if m != probe.num_seqs else tp
    # a whole batch that takes well under the budget is run repeatedly
    passes = 1
    if m == w.num_seqs and t < budget_s / 2:
        passes = max(1, min(100, int(budget_s / max(t, 1e-6))))
        t = sum(run(s) for _ in range(passes))
    work = alg_flops(s) if flops else alg_bytes(s)
    value, unit = (work * passes / t / 1e12, "TFLOP/s") if flops else (work * passes / t / 1e9, "GB/s")
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            model = next(l.split(":", 1)[1].strip() for l in fh if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    return {"value": value, "unit": unit, "cores": threads, "kind": "oracle", "cpu_model": model,
            "nproc": os.cpu_count(),
            "sample": f"first {m} of {w.num_seqs} sequences (sum_L={sum(s.seq_len_list)})"
                      + (f", {passes} passes" if passes > 1 else "") + f", fp64 C oracle, {t:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="headline batch (1..5)")
    ap.add_argument("--only", action="store_true", help="measure the headline batch only")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cache-write", action="store_true",
                    help="only measure pa_cache_write (mixed batch's 4216 tokens, bf16 and fp8 caches)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MiB",
                    help="only run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--trace", action="store_true",
                    help="only run the headline batch's timed steps (warm-up + steps, hinted calls): "
                         "what a profiler attached to this command records")
    ap.add_argument("--kv", choices=("bf16", "fp8"), default=None,
                    help="with --trace: the batch with caches of this dtype")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: this path has no multi-GPU mode (asked for {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2511_11581_amd import pa
    if not os.path.exists(pa.LIB_PATH):
        from paper_2511_11581_amd import build as hip_build
        hip_build.build()
    pa.load_library()
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(max(1, args.steps)):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "copies": max(1, args.steps)}))
        return

    if args.trace:
        from paper_2511_11581_amd import workloads as W
        if args.kv is None:
            w = W.make_config(args.config, device="cuda", poison=False)
        else:
            seqs, kw, gen, seed = W.config_seqs(args.config)
            kw = dict(kw, kv_dtype=args.kv)
            w = W.make_batch(seqs, seed=seed, device="cuda", poison=False, name=f"config{args.config}-{args.kv}",
                             _gen=gen, **kw)
        att = make_attention(w)
        out = torch.empty_like(w.q)
        ms = time_steps(w, att, out, args.steps, args.warmup, hint_of(w))
        print(json.dumps({"trace_config": args.config, "kv": args.kv, "ms_per_step": ms, "steps": args.steps}))
        return

    if args.cache_write:
        print(json.dumps({kv: measure_cache_write(kv, args.steps, args.warmup) for kv in ("bf16", "fp8")}))
        return

    configs = {}

    def report(k, r):
        e = r.get("error_vs_oracle") or {}
        print(f"# config {k}: {r['us_per_batch']:.1f} us/batch (median {r['us_median']:.1f}, min "
              f"{r['us_min']:.1f}; {r['us_per_batch_unhinted']:.1f} without the hint; "
              f"{r['graph_us_per_batch']:.1f} per call replayed from a HIP graph of 16), {r['GBps']:.0f} GB/s "
              f"({100 * r['frac_hbm']:.1f}% HBM), {r['TFLOPs']:.1f} TFLOP/s "
              f"({100 * r['frac_mfma']:.1f}% MFMA), kernels {r['per_kernel_us']}, "
              f"error vs oracle max {e.get('max_abs_err', float('nan')):.2e} "
              f"mean {e.get('mean_abs_err', float('nan')):.2e} ({e.get('rows', 0)} rows, "
              f"{'pass' if e.get('pass') else 'FAIL'})", file=sys.stderr, flush=True)

    headline_w, headline = measure(args.config, args.steps, args.warmup)
    configs[args.config] = headline
    report(args.config, headline)
    if not args.only:
        for k in (1, 2, 3, 4, 5):
            if k != args.config:
                _, r = measure(k, args.steps, args.warmup)
                configs[k] = r
                report(k, r)
                torch.cuda.empty_cache()

    # the decode and prefill batches on non-power-of-two pages (hybrid models)
    block_sizes = {}
    if not args.only:
        for k, bs in ((2, 528), (3, 400)):
            _, r = measure(k, args.steps, args.warmup, block_size=bs, with_error=False)
            block_sizes[f"config{k}_bs{bs}"] = {kk: r[kk] for kk in (
                "block_size", "us_per_batch", "us_median", "GBps", "frac_hbm", "TFLOPs", "frac_mfma",
                "per_kernel_us")}
            print(f"# config {k} at block size {bs}: {r['us_per_batch']:.1f} us/batch, "
                  f"{r['GBps']:.0f} GB/s, {r['TFLOPs']:.1f} TFLOP/s, kernels {r['per_kernel_us']}",
                  file=sys.stderr, flush=True)
            torch.cuda.empty_cache()

    # the prefill and mixed batches with fp8 e4m3 caches
    kv_fp8 = {}
    if not args.only:
        for k in (3, 4):
            _, r = measure(k, args.steps, args.warmup, kv_dtype="fp8")
            kv_fp8[f"config{k}_fp8"] = {kk: r[kk] for kk in (
                "us_per_batch", "us_median", "GBps", "frac_hbm", "TFLOPs", "frac_mfma",
                "per_kernel_us", "error_vs_oracle", "rocprof") if kk in r}
            for kk in ("prefill_kernel_TFLOPs", "decode_kernel_GBps"):
                if kk in r:
                    kv_fp8[f"config{k}_fp8"][kk] = r[kk]
            e = r.get("error_vs_oracle") or {}
            print(f"# config {k} with fp8 caches: {r['us_per_batch']:.1f} us/batch, "
                  f"{r['GBps']:.0f} GB/s, {r['TFLOPs']:.1f} TFLOP/s, kernels {r['per_kernel_us']}, "
                  f"error vs oracle max {e.get('max_abs_err', float('nan')):.2e} "
                  f"mean {e.get('mean_abs_err', float('nan')):.2e}", file=sys.stderr, flush=True)
            torch.cuda.empty_cache()

    cache_write = {}
    if not args.only:
        for kv in ("bf16", "fp8"):
            cw = measure_cache_write(kv, args.steps, args.warmup)
            cache_write[kv] = cw
            print(f"# cache write ({cw['tokens']} tokens, Hkv {cw['kv_heads']}, d {cw['head_dim']}, "
                  f"{kv} cache): {cw['us']:.1f} us per call replayed from a HIP graph "
                  f"({cw['us_eager']:.1f} us eager), {cw['GBps']:.0f} GB/s "
                  f"({100 * cw['frac_hbm']:.1f}% HBM)", file=sys.stderr, flush=True)

    ladder = None
    if not args.only:
        ladder = measure_ladder()
        for share, r in ladder.items():
            print(f"# ladder, decode share {share}%: baseline decomposition {r['baseline_us']:.0f} us, "
                  f"Q-blocks without split {r['qblock_us']:.0f} us, full path {r['full_us']:.0f} us "
                  f"({r['speedup']:.1f}x; {r['full_route']})", file=sys.stderr, flush=True)

    decode_like = args.config != 3
    h = headline
    if decode_like:
        value, unit = h["GBps"], "GB/s"
        dom_ms = h["per_kernel_us"].get("decode", 0) / 1e3
        achieved = decode_bytes(headline_w) / (dom_ms * 1e-3) / 1e9 if dom_ms else None
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS if achieved else None,
                "traffic": measured_traffic("decode_kernel", h["name"]),
                "kernel": "decode_kernel", "kernel_us": dom_ms * 1e3}
    else:
        value, unit = h["TFLOPs"], "TFLOP/s"
        dom_ms = h["per_kernel_us"].get("prefill", 0) / 1e3
        achieved = prefill_flops(headline_w) / (dom_ms * 1e-3) / 1e12 if dom_ms else None
        roof = {"bound": "mfma", "achieved": achieved, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / BF16_PEAK_TFLOPS if achieved else None,
                "traffic": measured_traffic("qblock_kernel", h["name"]),
                "kernel": "qblock_kernel", "kernel_us": dom_ms * 1e3}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(headline_w, flops=not decode_like)
    line = {
        "metric": METRIC, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": h["us_per_batch"] / 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if not headline_w.kv_fp8 else "bf16/fp8-kv",
        "data": "synthetic (seeded N(0,1) bf16 Q/K/V, random block tables)",
        "config": {"workload": h["name"], "seq_lens_sum": h["sum_L"], "seed": h["seed"],
                   "block_size": h["block_size"], "us_per_batch": h["us_per_batch"],
                   "us_median": h["us_median"], "us_min": h["us_min"],
                   "us_per_batch_unhinted": h["us_per_batch_unhinted"],
                   "graph_us_per_batch": h["graph_us_per_batch"], "hint": h["hint"],
                   "parallelism": "single GPU"},
        "roofline": roof, "cpu_baseline": cpu,
        "configs": {str(k): {kk: v for kk, v in r.items() if kk != "name"} for k, r in configs.items()},
        "block_sizes": block_sizes,
        "kv_fp8": kv_fp8,
        "cache_write": cache_write,
        "ladder": ladder,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
