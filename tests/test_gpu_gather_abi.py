"""Bit-exact block-table addressing of the attention kernels' own loaders
(gather-only debug mode, Sec. 4.3) and the ABI's error reporting on a GPU.

pa_debug_gather runs the plan kernel and the decode / Q-block kernels'
loads for a batch and stores the bytes each loader reads; every key a row
attends to must arrive exactly as the oracle's independent block-table walk
copies it.  Sequences with query length 1 go through the decode kernel's
loader (its block-id window, 16-key block addressing and head units),
those with query length >= 2 through the Q-block kernel's loader (bf16:
the copies straight into the LDS ring and its swizzles; fp8: the copies
into each wave's staging area, then the widening into the same ring);
sequences with no query rows are read by nothing.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2511_11581_amd import pa
from paper_2511_11581_amd import workloads as W
from gpu_util import attention_for, run_gpu, seed_of

pytestmark = pytest.mark.gpu


def gather_check(w, att=None):
    att = att or attention_for(w)
    wd = w.to("cuda")
    kd, vd = att.gather(wd.k_cache, wd.v_cache, wd.block_table, wd.seq_lens, wd.query_start_loc,
                        w.num_tokens)
    torch.cuda.synchronize()
    wc = w.to("cpu")
    rk, rv = oracle.gather(wc.k_cache, wc.v_cache, wc.block_table, wc.seq_lens)
    kb = kd.cpu().view(torch.uint8).numpy().reshape(rk.shape)
    vb = vd.cpu().view(torch.uint8).numpy().reshape(rv.shape)
    for i, (L, ql) in enumerate(zip(wc.seq_lens.tolist(), wc.q_lens)):
        n = L if ql >= 1 else 0
        assert np.array_equal(kb[i, :n], rk[i, :n]), f"K bytes differ in sequence {i} (q_len {ql})"
        assert np.array_equal(vb[i, :n], rv[i, :n]), f"V bytes differ in sequence {i} (q_len {ql})"
        assert not kb[i, n:].any() and not vb[i, n:].any(), f"sequence {i}: unread positions written"


@pytest.mark.parametrize("k", [1, 2, 3])
def test_gather_benchmark_batches(k):
    gather_check(W.make_config(k))


def test_gather_long_fp8_subset():
    # three of the long-context fp8 sequences (32K-128K keys), decode loader
    # with two-head units and windows of block ids far past the first
    w = W.make_config(5, device="cuda")
    sub = W.Workload(**{**w.__dict__})
    sub.block_table = w.block_table[:3].contiguous()
    sub.seq_lens = w.seq_lens[:3].contiguous()
    sub.query_start_loc = w.query_start_loc[:4].contiguous()
    sub.q = w.q[:3].contiguous()
    sub.ctx_lens, sub.q_lens = w.ctx_lens[:3], w.q_lens[:3]
    gather_check(sub)


GATHER_CASES = {
    # name: (seqs, Hq, Hkv, d, kv, block_size, extra)
    "bf16_d64_bs16": ([(37, 1), (0, 100), (250, 7), (1, 0), (5000, 1)], 8, 2, 64, "bf16", 16, {}),
    "fp8_d64_bs32": ([(37, 1), (0, 100), (250, 7), (1, 0), (3000, 1)], 8, 4, 64, "fp8", 32, {}),
    "bf16_d128_bs64": ([(37, 1), (0, 100), (250, 7), (1, 0), (4100, 1)], 8, 2, 128, "bf16", 64, {}),
    "fp8_d128_bs128": ([(600, 1), (0, 300), (190, 66), (8000, 1)], 16, 2, 128, "fp8", 128, {}),
    "bf16_d128_bs256_g1": ([(999, 1), (0, 257), (300, 2)], 4, 4, 128, "bf16", 256, {}),
    "fp8_d128_g8_hu1": ([(2000, 1), (70, 40), (5, 1)], 8, 1, 128, "fp8", 16, {}),
    "bf16_d64_hu1_odd_heads": ([(700, 1), (20, 90)], 3, 3, 64, "bf16", 16, {}),
    "fp8_d64_hu4": ([(1500, 1), (0, 77), (33, 1)], 16, 8, 64, "fp8", 16, {}),
    "wide_table_padded_rows": ([(70, 1), (0, 40), (0, 0)], 8, 2, 128, "bf16", 16,
                               dict(token_pad=5, table_width=20, pool_blocks=64)),
    "strided_window_moves": ([(70000, 1), (300, 1)], 8, 8, 128, "bf16", 16, {}),
    "bf16_d128_bs48": ([(37, 1), (0, 100), (250, 7), (1, 0), (4100, 1)], 8, 2, 128, "bf16", 48, {}),
    "fp8_d128_bs80": ([(600, 1), (0, 300), (190, 66), (8000, 1)], 16, 2, 128, "fp8", 80, {}),
    "bf16_d64_bs400": ([(999, 1), (0, 257), (300, 2), (20000, 1)], 8, 2, 64, "bf16", 400, {}),
    "fp8_d64_bs528_hu4": ([(1500, 1), (0, 77), (33, 1)], 16, 8, 64, "fp8", 528, {}),
}


@pytest.mark.parametrize("name", list(GATHER_CASES))
def test_gather_random_tables(name):
    seqs, Hq, Hkv, d, kv, bs, extra = GATHER_CASES[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of(name), name=name,
                     **extra)
    gather_check(w)


# ---- error reporting -----------------------------------------------------------

def _w():
    return W.make_batch([(30, 1), (0, 20)], 8, 2, 128, seed=3).to("cuda")


def _call(att, w, **over):
    args = dict(q=w.q, k_cache=w.k_cache, v_cache=w.v_cache, block_table=w.block_table,
                seq_lens=w.seq_lens, query_start_loc=w.query_start_loc, scale=w.scale,
                out=torch.empty_like(w.q))
    args.update(over)
    pa.pa_forward(att.handle, args["q"], args["k_cache"], args["v_cache"], args["block_table"],
                  args["seq_lens"], args["query_start_loc"], args["scale"], args["out"])


@pytest.mark.parametrize("bad", ["q_dtype", "out_shape", "q_misaligned", "table_rows", "qsl_len",
                                 "cache_heads", "scale", "kv_dtype"])
def test_invalid_arguments_are_reported_before_launch(bad):
    w = _w()
    att = attention_for(w)
    over = {}
    if bad == "q_dtype":
        over["q"] = w.q.float()
    elif bad == "out_shape":
        over["out"] = torch.empty(w.q.shape[0] + 1, *w.q.shape[1:], dtype=torch.bfloat16, device="cuda")
    elif bad == "q_misaligned":
        buf = torch.empty(w.q.numel() + 1, dtype=torch.bfloat16, device="cuda")
        over["q"] = buf[1:].view(w.q.shape)
    elif bad == "table_rows":
        over["block_table"] = w.block_table[:1]
    elif bad == "qsl_len":
        over["query_start_loc"] = w.query_start_loc[:-1]
    elif bad == "cache_heads":
        over["k_cache"] = w.k_cache[:, :, :1]
    elif bad == "scale":
        over["scale"] = float("nan")
    elif bad == "kv_dtype":
        over["k_cache"] = w.k_cache.view(torch.float8_e4m3fn)[..., :128]
    with pytest.raises(pa.PaError) as ei:
        _call(att, w, **over)
    assert ei.value.status == pa.PA_ERR_INVALID_ARG, str(ei.value)


def test_workspace_too_small():
    # a batch with 600 prefill rows on a workspace sized for decode only
    w = W.make_batch([(30, 600), (20, 1)], 8, 2, 128, seed=4).to("cuda")
    att = attention_for(w, max_tokens=1)
    with pytest.raises(pa.PaError) as ei:
        _call(att, w)
    assert ei.value.status == pa.PA_ERR_WORKSPACE


@pytest.mark.parametrize("bad", ["block_id", "q_gt_L", "qsl_order"])
def test_validate_flag_reports_bad_metadata(bad):
    w = _w()
    att = attention_for(w, validate=True)
    bt, sl, qsl = w.block_table.clone(), w.seq_lens.clone(), w.query_start_loc.clone()
    if bad == "block_id":
        bt[0, 0] = w.num_blocks + 5
    elif bad == "q_gt_L":
        sl[1] = 3
    elif bad == "qsl_order":
        qsl[1] = 25
        qsl[2] = 21
    with pytest.raises(pa.PaError) as ei:
        _call(att, w, block_table=bt, seq_lens=sl, query_start_loc=qsl)
    assert ei.value.status == pa.PA_ERR_DEVICE
    # the well-formed batch passes validation and runs
    _call(att, w)
    torch.cuda.synchronize()
