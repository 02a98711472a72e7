"""Randomised batches through the C ABI against the fp64 oracle.

Each case draws, from its own seeded generator: the head layout (G from 1
to 16, d 64 or 128), the cache dtype, the block size (powers of two and
not), 1..40 sequences mixing decode rows, short chunks and long prefills
over contexts up to 20K keys, padding rows past the batch, and whether the
host hint is given.  Every valid row is compared with the oracle, and the
padding rows must keep their sentinel.
"""
import pytest
import torch

from paper_2511_11581_amd import workloads as W
from gpu_util import SENTINEL, attention_for, check_close, oracle_full, valid_token_count

pytestmark = pytest.mark.gpu

HEADS = [(8, 2, 64), (32, 8, 128), (16, 2, 128), (8, 8, 128), (64, 8, 128), (16, 1, 64), (4, 4, 64),
         (16, 1, 128), (4, 2, 128), (16, 8, 64)]
BLOCKS = [16, 32, 48, 64, 400]
MAX_KEYS = 60_000          # keys of the batch (cache size)
MAX_WORK = 2e9             # (query row, key) pairs x query heads x d: the oracle's work


def draw(seed):
    g = torch.Generator().manual_seed(7000 + seed)

    def ri(lo, hi):
        return int(torch.randint(lo, hi + 1, (1,), generator=g))

    Hq, Hkv, d = HEADS[ri(0, len(HEADS) - 1)]
    kv = "fp8" if ri(0, 2) == 0 else "bf16"
    bs = BLOCKS[ri(0, len(BLOCKS) - 1)]
    seqs = []
    for _ in range(ri(1, 40)):
        kind = ri(0, 9)
        q = 1 if kind < 6 else (ri(2, 64) if kind < 8 else ri(65, 400))
        ctx = ri(0, 3000) if ri(0, 4) else ri(0, 20000)
        seqs.append((ctx, q))
    # shrink the contexts until the cache and the oracle's work fit
    while (sum(c + q for c, q in seqs) > MAX_KEYS or
           sum(q * (c + q) for c, q in seqs) * Hq * d > MAX_WORK):
        seqs = [(c // 2, q) for c, q in seqs]
        if all(c == 0 for c, _ in seqs):
            seqs = [(0, max(1, q // 2)) for _, q in seqs]
    return seqs, Hq, Hkv, d, kv, bs, ri(0, 1) == 1, ri(0, 3)


@pytest.mark.parametrize("seed", range(40))
def test_random_batch_matches_oracle(seed):
    seqs, Hq, Hkv, d, kv, bs, hinted, pad = draw(seed)
    name = f"random{seed} (S={len(seqs)}, {Hq}/{Hkv}, d {d}, {kv}, bs {bs}, hint {hinted})"
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed, name=name,
                     token_pad=pad)
    wd = w.to("cuda")
    att = attention_for(w)
    out = torch.full(wd.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
    hint = (sum(1 for _, q in seqs if q == 1), max(q for _, q in seqs)) if hinted else None
    att.forward(wd.q, wd.k_cache, wd.v_cache, wd.block_table, wd.seq_lens, wd.query_start_loc,
                w.scale, out=out, hint=hint)
    torch.cuda.synchronize()
    out = out.cpu()
    T = valid_token_count(w)
    check_close(out[:T], oracle_full(w)[:T], w.kv_fp8, name)
    assert (out[T:].float() == SENTINEL).all(), name
