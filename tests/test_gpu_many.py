"""Batches of thousands of sequences, past the sizes the fast paths hold:
a decode list longer than the decode kernel's LDS copy (~5000 entries for
these shapes: the list stays in the workspace, no fused planning), both
decode modes (whole pairs, split with merges), and more Q-blocks than the
plan kernel sorts in LDS (8192; then batch order, prefix sums read from
the workspace).  Plain and hinted calls, every row against the oracle."""
import pytest
import torch

from paper_2511_11581_amd import workloads as W
from gpu_util import SENTINEL, attention_for, check_close, oracle_full, valid_token_count

pytestmark = pytest.mark.gpu

MANY = {
    # name: (seqs [(ctx, q)], Hq, Hkv, d, kv)
    "decode_6000_whole": ([((37 * i) % 100, 1) for i in range(6000)], 8, 2, 64, "bf16"),
    "decode_6000_split": ([((37 * i) % 300, 1) for i in range(6000)], 8, 2, 64, "bf16"),
    "decode_5200_fp8_split": ([((53 * i) % 280 + 1, 1) for i in range(5200)], 16, 2, 64, "fp8"),
    "prefill_9000_qblocks": ([((13 * i) % 60, 2) for i in range(9000)], 8, 2, 64, "bf16"),
    "mixed_5000": ([((29 * i) % 250, 1) for i in range(5000)] + [((7 * i) % 90, 40) for i in range(60)],
                   8, 2, 64, "bf16"),
}


@pytest.mark.parametrize("name", list(MANY))
def test_many_sequences_match_oracle(name):
    seqs, Hq, Hkv, d, kv = MANY[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, seed=len(seqs), name=name, token_pad=2)
    wd = w.to("cuda")
    att = attention_for(w)
    plan = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]))
    if name.startswith("decode"):
        assert plan["decode_whole_units"] == (1 if "whole" in name else 0)
    ref = None
    T = valid_token_count(w)
    hint = (sum(1 for _, q in seqs if q == 1), max(q for _, q in seqs))
    for h in (None, hint):
        out = torch.full(wd.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
        att.forward(wd.q, wd.k_cache, wd.v_cache, wd.block_table, wd.seq_lens, wd.query_start_loc,
                    w.scale, out=out, hint=h)
        torch.cuda.synchronize()
        out = out.cpu()
        if ref is None:
            ref = oracle_full(w)[:T]
        check_close(out[:T], ref, w.kv_fp8, f"{name} hint={h is not None}")
        assert (out[T:].float() == SENTINEL).all()
