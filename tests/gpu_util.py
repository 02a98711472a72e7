"""Helpers shared by the GPU tests: run the HIP path through the C ABI and
compare with the fp64 oracle."""
import concurrent.futures as cf
import contextlib
import os
import zlib

import numpy as np
import torch

import oracle
from paper_2511_11581_amd import pa

SENTINEL = 7.0  # written into out before a call; rows the call must not touch keep it

TOL = {False: (2e-2, 2e-3), True: (5e-2, 5e-3)}  # (max abs, mean abs) for bf16 / fp8 KV
LOG2E = 1.4426950408889634


def seed_of(name: str) -> int:
    """A seed that is the same in every process (str hashes are not)."""
    return zlib.crc32(name.encode()) % 100000


@contextlib.contextmanager
def _env(name, value):
    old = os.environ.get(name)
    os.environ[name] = str(value)
    try:
        yield
    finally:
        if old is None:
            del os.environ[name]
        else:
            os.environ[name] = old


def qblock_rows(n):
    """Handles created inside use Q-blocks of n rows (PA_QBLOCK_ROWS, bf16
    caches: 128 or 256), whatever the tuned rule would pick."""
    return _env("PA_QBLOCK_ROWS", n)


@contextlib.contextmanager
def decode_min_steps(n):
    """Handles created inside take the decode minimum share n (the planner
    knob PA_DECODE_MIN_STEPS, read when a handle is created)."""
    old = os.environ.get("PA_DECODE_MIN_STEPS")
    os.environ["PA_DECODE_MIN_STEPS"] = str(n)
    try:
        yield
    finally:
        if old is None:
            del os.environ["PA_DECODE_MIN_STEPS"]
        else:
            os.environ["PA_DECODE_MIN_STEPS"] = old


def attention_for(w, validate=False, max_tokens=None, max_seqs=None, max_blocks=None,
                  no_split_kv=False):
    return pa.PagedAttention(
        w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size, w.k_cache.dtype,
        w.k_scale, w.v_scale,
        max_tokens=max_tokens or max(1, w.num_tokens), max_seqs=max_seqs or max(1, w.num_seqs),
        max_blocks_per_seq=max_blocks or max(1, int(w.block_table.shape[1])), validate=validate,
        no_split_kv=no_split_kv)


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


def row_scores_log2(w, rows):
    """Per-key scores of each (token, head) row in log2 units, from the
    oracle's normalised weights and log-sum-exp: s_p = (lse + ln w_p) log2(e).
    Returns a list of 1-D arrays (one per row, over the row's visible keys)."""
    wc = cpu_inputs(w)
    rows = np.asarray(rows, dtype=np.int64).reshape(-1, 2)
    qsl = wc.query_start_loc.numpy()
    sl = wc.seq_lens.numpy()
    maxk = int(sl.max()) if len(sl) else 1
    _, lse, wt = oracle.rows(wc.q, wc.k_cache, wc.v_cache, wc.block_table, wc.seq_lens,
                             wc.query_start_loc, wc.scale, rows, k_scale=wc.k_scale,
                             v_scale=wc.v_scale, with_lse=True, max_keys=maxk)
    out = []
    for k, (t, h) in enumerate(rows):
        i = int(np.searchsorted(qsl, t, side="right") - 1)
        n = int(sl[i] - (qsl[i + 1] - qsl[i]) + (t - qsl[i]) + 1)
        with np.errstate(divide="ignore"):
            out.append((lse[k] + np.log(wt[k, :n])) * LOG2E)
    return out


def tile_maxima(s, first, end, size):
    """Maxima of s over consecutive tiles of `size` keys of [first, end)."""
    return [float(np.max(s[a:min(a + size, end)])) for a in range(first, end, size)]


def jumps_over_running_max(tm):
    """Largest rise of a tile's maximum over the running maximum of the
    tiles before it (-inf for a single tile)."""
    best, run = float("-inf"), tm[0]
    for x in tm[1:]:
        best = max(best, x - run)
        run = max(run, x)
    return best
