"""Helpers shared by the GPU tests: run the HIP path through the C ABI and
compare with the fp64 oracle."""
import concurrent.futures as cf
import os

import numpy as np
import torch

import oracle
from paper_2511_11581_amd import pa

SENTINEL = 7.0  # written into out before a call; rows the call must not touch keep it

TOL = {False: (2e-2, 2e-3), True: (5e-2, 5e-3)}  # (max abs, mean abs) for bf16 / fp8 KV


def attention_for(w, validate=False, max_tokens=None, max_seqs=None, max_blocks=None):
    return pa.PagedAttention(
        w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size, w.k_cache.dtype,
        w.k_scale, w.v_scale,
        max_tokens=max_tokens or max(1, w.num_tokens), max_seqs=max_seqs or max(1, w.num_seqs),
        max_blocks_per_seq=max_blocks or max(1, int(w.block_table.shape[1])), validate=validate)


def run_gpu(w, att=None, out=None):
    """Run pa_forward on a workload (moved to the GPU if needed); returns out on the CPU."""
    wd = w if w.q.is_cuda else w.to("cuda")
    att = att or attention_for(w)
    if out is None:
        out = torch.full(wd.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
    att.forward(wd.q, wd.k_cache, wd.v_cache, wd.block_table, wd.seq_lens,
                wd.query_start_loc, w.scale, out=out)
    torch.cuda.synchronize()
    return out.cpu()


def cpu_inputs(w):
    if w.q.is_cuda:
        return w.to("cpu")
    return w


def oracle_full(w):
    wc = cpu_inputs(w)
    return oracle.forward(wc.q, wc.k_cache, wc.v_cache, wc.block_table, wc.seq_lens,
                          wc.query_start_loc, wc.scale, k_scale=wc.k_scale, v_scale=wc.v_scale)


def oracle_rows(w, rows, threads=None):
    """fp64 rows (token, head) computed in parallel chunks."""
    wc = cpu_inputs(w)
    rows = np.asarray(rows, dtype=np.int64).reshape(-1, 2)
    nt = threads or oracle.default_threads()
    chunks = np.array_split(rows, max(1, min(nt, len(rows))))
    args = (wc.q, wc.k_cache, wc.v_cache, wc.block_table, wc.seq_lens, wc.query_start_loc,
            wc.scale)

    def one(ch):
        return oracle.rows(*args, ch, k_scale=wc.k_scale, v_scale=wc.v_scale)

    with cf.ThreadPoolExecutor(max_workers=len(chunks)) as ex:
        parts = list(ex.map(one, chunks))
    return np.concatenate(parts, 0)


def valid_token_count(w):
    return int(w.query_start_loc[-1])


def check_close(got, ref, fp8, what=""):
    """got: bf16 tensor/array rows; ref: fp64 rows of the same shape."""
    g = got.double().numpy() if isinstance(got, torch.Tensor) else np.asarray(got, np.float64)
    err = np.abs(g - ref)
    mx_tol, mean_tol = TOL[fp8]
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    mx, mean = float(err.max()), float(err.mean())
    assert mx <= mx_tol and mean <= mean_tol, f"{what}: max abs {mx:.3e}, mean abs {mean:.3e}"
    return mx, mean


def sample_rows(w, n, seed=0):
    """n (token, head) rows: first and last token of every sequence plus random ones."""
    rng = np.random.default_rng(seed)
    qsl = w.query_start_loc.cpu().numpy()
    rows = set()
    for i in range(len(qsl) - 1):
        a, b = int(qsl[i]), int(qsl[i + 1])
        if b > a:
            rows.add((a, int(rng.integers(w.num_q_heads))))
            rows.add((b - 1, int(rng.integers(w.num_q_heads))))
    T = int(qsl[-1])
    while len(rows) < n and T > 0:
        rows.add((int(rng.integers(T)), int(rng.integers(w.num_q_heads))))
    return sorted(rows)
