"""GPU parity of the ablation's baseline decomposition (pa_forward_baseline:
one wave per (query token, query head), one page per tile; the paper's
Sec. 4 / App. A design) against the oracle, to the same tolerance as the
main path."""
import pytest
import torch

from paper_2511_11581_amd import workloads as W
from gpu_util import SENTINEL, attention_for, check_close, oracle_full, valid_token_count

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
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=len(name), name=name)
    got = _baseline(w)
    T = valid_token_count(w)
    ref = oracle_full(w)
    check_close(got[:T], ref[:T], w.kv_fp8, name)


def test_baseline_config1():
    w = W.make_config(1)
    got = _baseline(w)
    T = valid_token_count(w)
    check_close(got[:T], oracle_full(w)[:T], w.kv_fp8, "config1")
