"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Tolerances: max abs 2e-2 / mean abs 2e-3 with bf16 K/V, 5e-2 / 5e-3 with
fp8 K/V.  Every batch, the five benchmark batches at full size included, is
compared element by element on every valid row, the benchmark batches in the
launch configuration the benchmark times.  Seeds are fixed per case.
"""
import numpy as np
import pytest
import torch

from paper_2511_11581_amd import workloads as W
from gpu_util import (SENTINEL, attention_for, check_close, oracle_full, oracle_rows, qblock_rows,
                      run_gpu, sample_rows, seed_of, valid_token_count)

pytestmark = pytest.mark.gpu


def full_check(w):
    out = run_gpu(w)
    ref = oracle_full(w)
    T = valid_token_count(w)
    check_close(out[:T], ref[:T], w.kv_fp8, w.name)
    assert (out[T:].float() == SENTINEL).all(), "rows past query_start_loc[S] were written"
    return out


SMALL = {
    # name: (seqs [(ctx, q)], Hq, Hkv, d, kv, block_size, extra kwargs)
    "decode_g4_d64": ([(17, 1), (64, 1), (100, 1), (255, 1)], 8, 2, 64, "bf16", 16, {}),
    "decode_g1": ([(40, 1), (700, 1), (1, 1)], 4, 4, 128, "bf16", 16, {}),
    "decode_g8_split": ([(3000, 1), (257, 1), (0, 1), (1500, 1)], 16, 2, 128, "bf16", 16, {}),
    "decode_g16_split": ([(2200, 1), (31, 1)], 16, 1, 128, "bf16", 16, {}),
    "decode_g2_d64_split": ([(1025, 1), (4096, 1), (15, 1)], 4, 2, 64, "bf16", 16, {}),
    "decode_bs32": ([(990, 1), (33, 1)], 8, 2, 128, "bf16", 32, {}),
    "decode_fp8": ([(1800, 1), (77, 1), (4000, 1)], 8, 1, 128, "fp8", 16, {}),
    "decode_fp8_d64": ([(600, 1), (9, 1)], 8, 2, 64, "fp8", 16, {}),
    "prefill_g4": ([(0, 100), (0, 33), (0, 2)], 8, 2, 128, "bf16", 16, {}),
    "prefill_g1": ([(0, 300), (0, 129)], 2, 2, 128, "bf16", 16, {}),
    "prefill_g8_d64": ([(0, 77), (0, 16), (0, 17)], 16, 2, 64, "bf16", 16, {}),
    "prefill_g16": ([(0, 45), (0, 9)], 16, 1, 128, "bf16", 16, {}),
    "chunked": ([(500, 64), (17, 130), (1000, 3)], 8, 2, 128, "bf16", 16, {}),
    "chunked_bs32": ([(45, 80), (300, 40)], 8, 2, 128, "bf16", 32, {}),
    "prefill_fp8": ([(0, 150), (200, 70)], 8, 2, 128, "fp8", 16, {}),
    "mixed": ([(1200, 1), (0, 90), (30, 1), (400, 65), (5000, 1), (0, 2)], 32, 8, 128, "bf16", 16, {}),
    "mixed_d64_g4": ([(0, 50), (130, 1), (60, 20)], 8, 2, 64, "bf16", 16, {}),
    "empty_queries": ([(50, 0), (30, 1), (0, 0), (20, 5)], 8, 2, 128, "bf16", 16, {}),
    "padded_rows_wide_table": ([(70, 1), (0, 40)], 8, 2, 128, "bf16", 16,
                               dict(token_pad=5, table_width=20, pool_blocks=64)),
    "ragged_tails": ([(15, 1), (16, 1), (17, 1), (31, 2), (33, 31), (0, 63), (0, 65)], 8, 2, 128,
                     "bf16", 16, {}),
    # block sizes past 32 on every kernel (decode, bf16 Q-block, fp8 Q-block)
    "decode_bs64": ([(990, 1), (33, 1), (4000, 1)], 8, 2, 128, "bf16", 64, {}),
    "decode_bs128_fp8": ([(1800, 1), (77, 1), (300, 1)], 8, 1, 128, "fp8", 128, {}),
    "decode_bs256_d64": ([(1025, 1), (15, 1), (600, 1)], 4, 2, 64, "bf16", 256, {}),
    "decode_bs256_fp8_d64": ([(3000, 1), (255, 1), (256, 1)], 16, 4, 64, "fp8", 256, {}),
    "prefill_bs64": ([(0, 150), (70, 64), (300, 9)], 8, 2, 128, "bf16", 64, {}),
    "prefill_bs128_d64": ([(0, 77), (100, 40)], 16, 2, 64, "bf16", 128, {}),
    "prefill_bs256": ([(0, 300), (500, 33), (255, 2)], 8, 2, 128, "bf16", 256, {}),
    # the fp8 Q-block kernel: head sizes, group sizes, block sizes (bs > 64
    # moves the tile start inside a block), chunks with long contexts
    "prefill_fp8_bs64": ([(0, 150), (200, 70)], 8, 2, 128, "fp8", 64, {}),
    "prefill_fp8_bs128": ([(0, 150), (130, 70), (1000, 5)], 8, 2, 128, "fp8", 128, {}),
    "prefill_fp8_bs256_d64": ([(0, 100), (300, 20)], 8, 2, 64, "fp8", 256, {}),
    "prefill_fp8_g1": ([(0, 200), (40, 33)], 4, 4, 128, "fp8", 16, {}),
    "prefill_fp8_g8_d64": ([(0, 77), (0, 16), (60, 17)], 16, 2, 64, "fp8", 16, {}),
    "prefill_fp8_g16": ([(0, 45), (100, 9)], 16, 1, 128, "fp8", 32, {}),
    "chunked_fp8_long": ([(2000, 200), (64, 64), (5000, 3)], 32, 8, 128, "fp8", 16, {}),
    "mixed_fp8": ([(1200, 1), (0, 90), (30, 1), (400, 65), (5000, 1), (0, 2)], 32, 8, 128, "fp8", 16, {}),
    # block sizes that are multiples of 16 but not powers of two (the large
    # pages of hybrid attention / state-space models, Sec. 4.6)
    "decode_bs48": ([(990, 1), (47, 1), (48, 1), (4000, 1)], 8, 2, 128, "bf16", 48, {}),
    "decode_bs80_fp8": ([(1800, 1), (79, 1), (300, 1)], 8, 1, 128, "fp8", 80, {}),
    "decode_bs400_d64": ([(1025, 1), (399, 1), (2600, 1)], 4, 2, 64, "bf16", 400, {}),
    "decode_bs528_fp8_d64": ([(3000, 1), (527, 1), (528, 1)], 16, 4, 64, "fp8", 528, {}),
    "prefill_bs48": ([(0, 150), (70, 64), (300, 9)], 8, 2, 128, "bf16", 48, {}),
    "prefill_bs80_d64": ([(0, 77), (100, 40), (0, 300)], 16, 2, 64, "bf16", 80, {}),
    "prefill_bs400": ([(0, 700), (500, 33), (399, 2)], 8, 2, 128, "bf16", 400, {}),
    "prefill_fp8_bs48": ([(0, 150), (200, 70)], 8, 2, 128, "fp8", 48, {}),
    "prefill_fp8_bs400_d64": ([(0, 500), (300, 20)], 8, 2, 64, "fp8", 400, {}),
    "mixed_bs528": ([(1200, 1), (0, 90), (30, 1), (400, 65), (5000, 1), (0, 2)], 32, 8, 128, "bf16", 528, {}),
    "mixed_fp8_bs80": ([(1200, 1), (0, 90), (30, 1), (400, 65), (5000, 1)], 32, 8, 128, "fp8", 80, {}),
    # short sequences only (table width <= 8 decode steps): whole (sequence,
    # unit) pairs per workgroup, merged inside it; more pairs than
    # workgroups, so a workgroup runs several pairs in turn
    "decode_many_short": ([((37 * i) % 207, 1) for i in range(300)], 32, 8, 128, "bf16", 16, {}),
    # whole pairs (table width <= 8 steps) with the largest pieces the
    # workgroup merges from LDS: 4 heads per unit, and 16 query heads per kv head
    "decode_whole_hu4_fp8_d64": ([(200, 1), (31, 1), (129, 1), (250, 1)], 16, 4, 64, "fp8", 16, {}),
    "decode_whole_g16": ([(255, 1), (100, 1), (17, 1)], 16, 1, 128, "bf16", 16, {}),
    "decode_whole_g16_d64_hu2": ([(240, 1), (64, 1), (1, 1)], 32, 2, 64, "bf16", 16, {}),
    "decode_many_short_fp8_g8": ([((53 * i) % 250 + 1, 1) for i in range(100)], 64, 8, 128, "fp8", 16, {}),
    "mixed_short_g16_d64": ([((29 * i) % 120, 1) for i in range(40)] + [(0, 60), (50, 30), (3, 2)],
                            32, 2, 64, "bf16", 16, {}),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_batches_match_oracle(name):
    seqs, Hq, Hkv, d, kv, bs, extra = SMALL[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of(name),
                     name=name, **extra)
    full_check(w)


FORCED_ROWS = ["prefill_g4", "prefill_g8_d64", "prefill_g16", "chunked", "ragged_tails",
               "prefill_bs256", "mixed", "prefill_bs48", "prefill_bs400"]


@pytest.mark.parametrize("rows", [128, 256])
@pytest.mark.parametrize("name", FORCED_ROWS)
def test_both_q_block_shapes_match_oracle(name, rows):
    # bf16 Q-block kernel with 4 waves (128 rows, two workgroups per CU) and
    # 8 waves (256 rows), whichever the tuned rule would pick
    seqs, Hq, Hkv, d, kv, bs, extra = SMALL[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of(name),
                     name=f"{name}_rows{rows}", **extra)
    with qblock_rows(rows):
        att = attention_for(w)
    assert att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]))["block_m"] == rows
    out = run_gpu(w, att)
    T = valid_token_count(w)
    check_close(out[:T], oracle_full(w)[:T], w.kv_fp8, w.name)
    assert (out[T:].float() == SENTINEL).all()


def test_shuffled_mixed_order():
    seqs = [(c, 1) for c in (900, 20, 3000, 450)] + [(c, q) for c, q in ((0, 70), (250, 33))]
    order = [4, 0, 2, 5, 1, 3]
    w = W.make_batch([seqs[i] for i in order], 16, 4, 128, seed=5, name="shuffled")
    full_check(w)


def test_config1_full():
    full_check(W.make_config(1))


@pytest.mark.parametrize("k", [2, 3, 4, 5])
def test_benchmark_batches_full(k):
    # Every row of the full-size batch, element by element, in the launch
    # configuration the benchmark times.
    w = W.make_config(k, device="cuda")
    out = run_gpu(w)
    wc = w.to("cpu")
    del w
    torch.cuda.empty_cache()
    ref = oracle_full(wc)
    T = valid_token_count(wc)
    mx, mean = check_close(out[:T], ref[:T], wc.kv_fp8, wc.name)
    print(f"{wc.name}: {T} rows x {wc.num_q_heads} heads, max abs {mx:.3e}, mean abs {mean:.3e}")


def test_config4_shuffled_sampled():
    w = W.make_config(4, device="cuda", shuffle=True)
    out = run_gpu(w)
    rows = sample_rows(w, 256, seed=44)
    ref = oracle_rows(w, rows)
    check_close(torch.stack([out[t, h] for t, h in rows]), ref, False, "config4-shuffled")


def test_deterministic_bitwise():
    w = W.make_config(4, device="cuda")
    att = attention_for(w)
    a = run_gpu(w, att)
    b = run_gpu(w, att)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_empty_batch_is_a_no_op():
    w = W.make_batch([], 8, 2, 128, seed=1, pool_blocks=2)
    out = run_gpu(w)
    assert out.shape[0] == 0
    w = W.make_batch([(10, 0)], 8, 2, 128, seed=1, token_pad=3)
    out = run_gpu(w)
    assert (out.float() == SENTINEL).all()
