"""Parity where the online softmax must move its reference maximum
(Sec. 4.1, Eq. 2) and where the log-sum-exp merge combines segments whose
maxima are far apart (Sec. 4.5).

With N(0,1) inputs at scale 1/sqrt(d) every score stays within a few units
of the first tile's maximum, so the kernels' rescale paths never run.  These
batches force them, in two ways:
  * large logits: Q drawn with a standard deviation of 16 or 32;
  * planted keys: a key aligned with one query token's heads, placed late in
    the sequence, so that its tile's maximum rises far above the maxima of
    the tiles before it.
Each case first shows, from the oracle's per-key scores (log2 units), that
its inputs cross the threshold of the kernel that computes them:
  * Q-block kernel (every cache dtype and head size): the reference is the
    first 64-key tile's row max and moves when a weight exceeds 2^12, so
    some later tile's max must exceed the first tile's max by more than 12;
  * decode kernel: the running max moves when a decode step's max exceeds
    it by more than 8;
  * merge: the pieces of one split row must have maxima more than 20 apart.
Then every row is compared with the oracle at the usual tolerances.
"""
import numpy as np
import pytest
import torch

from paper_2511_11581_amd import pa
from paper_2511_11581_amd import workloads as W
from gpu_util import (SENTINEL, attention_for, check_close, decode_min_steps, jumps_over_running_max,
                      oracle_full, row_scores_log2, run_gpu, seed_of, tile_maxima, valid_token_count)

pytestmark = pytest.mark.gpu

TILE = 64   # keys per Q-block tile


def _rows_of_tokens(w, tokens):
    G = w.num_q_heads // w.num_kv_heads
    return [(t, h) for t in tokens for h in range(w.num_q_heads)]


def _prefill_jump(w, rows):
    """Largest rise, over the rows, of a later tile's max over the first
    tile's max (the Q-block kernel's reference)."""
    best = float("-inf")
    for s in row_scores_log2(w, rows):
        tm = tile_maxima(s, 0, len(s), TILE)
        if len(tm) < 2:
            continue
        best = max(best, max(tm[1:]) - tm[0])
    return best


def _decode_pieces(att, w):
    qsl = w.query_start_loc.cpu().tolist()
    sl = w.seq_lens.cpu().tolist()
    return pa.pa_decode_pieces(att.handle, None, 0, sl, qsl, w.num_tokens,
                               int(w.block_table.shape[1]))


def _decode_crossings(att, w):
    """(largest rise of a decode step's max over the running max inside one
    piece, largest spread of piece maxima within one split row), over all
    decode rows, from the partition the device computes."""
    G = w.num_q_heads // w.num_kv_heads
    ks = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]))["decode_step"]
    pieces = _decode_pieces(att, w)
    qsl = w.query_start_loc.cpu().tolist()
    by_pair = {}
    for pc in pieces:
        by_pair.setdefault((pc["seq"], pc["kv_head"]), []).append((pc["first_key"], pc["end_key"]))
    rows = [(qsl[i], g * G + hh) for (i, g) in by_pair for hh in range(G)]
    scores = row_scores_log2(w, rows)
    step_jump, spread = float("-inf"), float("-inf")
    for (t, h), s in zip(rows, scores):
        i = qsl.index(t)
        segs = by_pair[(i, h // G)]
        maxima = []
        for a, b in segs:
            tm = tile_maxima(s, a, b, ks)
            maxima.append(max(tm))
            if len(tm) > 1:
                step_jump = max(step_jump, jumps_over_running_max(tm))
        if len(segs) > 1:
            spread = max(spread, max(maxima) - min(maxima))
    return step_jump, spread


def _full(w, att):
    out = run_gpu(w, att)
    ref = oracle_full(w)
    T = valid_token_count(w)
    check_close(out[:T], ref[:T], w.kv_fp8, w.name)
    assert (out[T:].float() == SENTINEL).all()


PREFILL = {
    # name: (seqs, Hq, Hkv, d, kv, bs, q_scale, spikes (seq, key, token, c), rows' tokens)
    "qblock_qx16": ([(0, 700), (300, 200)], 8, 2, 128, "bf16", 16, 16.0, (), [5, 300, 699, 750, 899]),
    "qblock_qx32_g8_d64": ([(0, 500), (1000, 64)], 16, 2, 64, "bf16", 32, 32.0, (), [100, 499, 530]),
    "qblock_spike_g1": ([(0, 400), (500, 100)], 4, 4, 128, "bf16", 16, 1.0,
                        [(0, 300, 350, 8.0), (1, 520, 90, 8.0)], [350, 490]),
    "qblock_spike_g4": ([(0, 1000), (200, 300)], 8, 2, 128, "bf16", 16, 1.0,
                        [(0, 700, 900, 6.0), (1, 410, 250, 6.0)], [900, 1250]),
    "prefill_fp8_spike": ([(0, 300), (700, 130)], 8, 2, 128, "fp8", 16, 1.0,
                          [(0, 200, 250, 8.0), (1, 750, 100, 8.0)], [250, 400]),
    "prefill_fp8_qx16_d64": ([(0, 400)], 8, 2, 64, "fp8", 64, 16.0, (), [100, 250, 399]),
    "prefill_fp8_qx32_g8": ([(0, 260), (900, 40)], 16, 2, 128, "fp8", 16, 32.0, (), [200, 290]),
}


@pytest.mark.parametrize("name", list(PREFILL))
def test_prefill_rescale(name):
    seqs, Hq, Hkv, d, kv, bs, qs, spikes, toks = PREFILL[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of(name), name=name,
                     q_scale=qs, spikes=spikes)
    jump = _prefill_jump(w, _rows_of_tokens(w, toks))
    assert jump > 12.0, f"{name}: inputs rise only {jump:.1f} log2 units over the first tile (need > 12)"
    _full(w, attention_for(w))


DECODE = {
    # name: (seqs, Hq, Hkv, d, kv, bs, q_scale, spikes, minimum decode share)
    # unsplit rows (one worker per (sequence, kv head)): the step rescale
    "decode_spike_unsplit": ([(3000, 1), (1500, 1), (700, 1), (5000, 1)], 8, 2, 128, "bf16", 16, 1.0,
                             [(0, 2500, 0, 6.0), (1, 1200, 0, 6.0), (2, 650, 0, 6.0), (3, 4000, 0, 6.0)],
                             4096),
    "decode_fp8_spike_unsplit": ([(3000, 1), (900, 1), (6000, 1)], 16, 2, 128, "fp8", 16, 1.0,
                                 [(0, 2000, 0, 8.0), (1, 800, 0, 8.0), (2, 5500, 0, 8.0)], 4096),
    "decode_d64_qx16_unsplit": ([(2000, 1), (513, 1), (4096, 1)], 4, 2, 64, "bf16", 32, 16.0, (), 4096),
    "decode_fp8_d64_qx32_unsplit": ([(1500, 1), (3333, 1)], 8, 2, 64, "fp8", 16, 32.0, (), 4096),
    # split rows: merges of pieces whose maxima are far apart, with pieces of
    # at least 8 or 16 steps (rescales inside the pieces too) and with the
    # default partition (pieces of one step)
    "merge_spike": ([(6000, 1), (9000, 1)], 8, 2, 128, "bf16", 16, 1.0,
                    [(0, 4500, 0, 8.0), (1, 7000, 0, 8.0)], 8),
    "merge_fp8_spike_g8": ([(20000, 1), (3000, 1)], 16, 2, 128, "fp8", 16, 1.0,
                           [(0, 15000, 0, 10.0), (1, 2500, 0, 10.0)], 16),
    "merge_qx32_d64": ([(8000, 1), (2000, 1)], 8, 4, 64, "bf16", 16, 32.0, (), 8),
    "merge_one_step_pieces": ([(6000, 1), (9000, 1)], 8, 2, 128, "bf16", 16, 1.0,
                              [(0, 4500, 0, 8.0), (1, 7000, 0, 8.0)], None),
}


@pytest.mark.parametrize("name", list(DECODE))
def test_decode_rescale_and_merge(name):
    seqs, Hq, Hkv, d, kv, bs, qs, spikes, share = DECODE[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of(name), name=name,
                     q_scale=qs, spikes=spikes)
    if share is None:
        att = attention_for(w)
    else:
        with decode_min_steps(share):
            att = attention_for(w)
    step_jump, spread = _decode_crossings(att, w)
    if share is not None:   # pieces of several steps: the rescale inside a piece
        assert step_jump > 8.0, f"{name}: a step max rises only {step_jump:.1f} over the running max"
    if name.startswith("merge"):
        assert spread > 20.0, f"{name}: piece maxima of a split row differ by only {spread:.1f}"
    else:
        assert spread == float("-inf"), f"{name}: expected unsplit rows"
    _full(w, att)


def test_mixed_batch_with_spikes():
    # decode and prefill rows of one call, each with a planted key
    seqs = [(2500, 1), (0, 300), (900, 1), (400, 120)]
    spikes = [(0, 2000, 0, 7.0), (1, 250, 280, 7.0), (2, 880, 0, 7.0), (3, 450, 100, 7.0)]
    w = W.make_batch(seqs, 32, 8, 128, seed=seed_of("mixed_spikes"), name="mixed_spikes",
                     spikes=spikes)
    _full(w, attention_for(w))
