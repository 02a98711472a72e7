"""GPU parity of the ablation's rungs (the optimisation ladder of Sec. 7)
against the oracle, to the same tolerance as the main path: the baseline
decomposition (pa_forward_baseline: one wave per (query token, query head),
one page per tile; Sec. 4 / App. A) and Q-blocks without the split-KV
decode kernel (PA_FLAG_NO_SPLIT_KV: single-token rows as Q-blocks of one
token, Sec. 4.4, no split and no merge)."""
import pytest
import torch

from paper_2511_11581_amd import workloads as W
from gpu_util import (SENTINEL, attention_for, check_close, oracle_full, run_gpu, seed_of,
                      valid_token_count)

pytestmark = pytest.mark.gpu


def _baseline(w):
    wd = w.to("cuda")
    att = attention_for(w)
    out = torch.full(wd.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
    att.forward_baseline(wd.q, wd.k_cache, wd.v_cache, wd.block_table, wd.seq_lens,
                         wd.query_start_loc, w.scale, out=out)
    torch.cuda.synchronize()
    return out.cpu()


@pytest.mark.parametrize("name,seqs,Hq,Hkv,d,kv,bs", [
    ("mixed_g4", [(300, 1), (0, 70), (45, 33), (1000, 1)], 16, 4, 128, "bf16", 16),
    ("prefill_g8_d64_bs32", [(0, 77), (40, 20)], 16, 2, 64, "bf16", 32),
    ("decode_fp8", [(600, 1), (9, 1), (2000, 1)], 16, 2, 128, "fp8", 16),
])
def test_baseline_matches_oracle(name, seqs, Hq, Hkv, d, kv, bs):
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of(name), name=name)
    got = _baseline(w)
    T = valid_token_count(w)
    ref = oracle_full(w)
    check_close(got[:T], ref[:T], w.kv_fp8, name)


def test_baseline_config1():
    w = W.make_config(1)
    got = _baseline(w)
    T = valid_token_count(w)
    check_close(got[:T], oracle_full(w)[:T], w.kv_fp8, "config1")


@pytest.mark.parametrize("name,seqs,Hq,Hkv,d,kv,bs", [
    ("decode_g4", [(17, 1), (64, 1), (100, 1), (255, 1), (3000, 1)], 8, 2, 64, "bf16", 16),
    ("decode_g8_long", [(9000, 1), (257, 1), (0, 1)], 16, 2, 128, "bf16", 16),
    ("mixed_g4", [(300, 1), (0, 70), (45, 33), (1000, 1)], 16, 4, 128, "bf16", 48),
    ("decode_fp8_g8", [(600, 1), (9, 1), (2000, 1)], 16, 2, 128, "fp8", 16),
    ("mixed_fp8_d64", [(0, 50), (130, 1), (60, 20), (5000, 1)], 8, 2, 64, "fp8", 32),
])
def test_qblock_rung_without_split_matches_oracle(name, seqs, Hq, Hkv, d, kv, bs):
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of("nosplit" + name),
                     name=name)
    att = attention_for(w, no_split_kv=True)
    plan = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]))
    assert plan["prefill_launch"] == 1
    got = run_gpu(w, att)
    T = valid_token_count(w)
    check_close(got[:T], oracle_full(w)[:T], w.kv_fp8, name)
    assert (got[T:].float() == SENTINEL).all()
    # the decode kernel found no rows: the split partials were never used
    assert torch.isfinite(got[:T].float()).all()


def test_qblock_rung_config1():
    w = W.make_config(1)
    got = run_gpu(w, attention_for(w, no_split_kv=True))
    T = valid_token_count(w)
    check_close(got[:T], oracle_full(w)[:T], w.kv_fp8, "config1-no-split")
