"""pa_forward_noalloc (for callers that cannot allocate device memory)
against pa_forward: the same kernels on the library's static scratch
instead of the handle's workspace.  Two calls in a row on one handle, the
second with a smaller batch, each bitwise equal to pa_forward's output and
within the oracle tolerances; rows past query_start_loc[S] untouched."""
import pytest
import torch

from paper_2511_11581_amd import pa
from paper_2511_11581_amd import workloads as W
from gpu_util import SENTINEL, attention_for, check_close, oracle_full, seed_of, valid_token_count

pytestmark = pytest.mark.gpu


def _handle_without_workspace(w):
    kvd = pa.PA_DTYPE_FP8_E4M3 if w.kv_fp8 else pa.PA_DTYPE_BF16
    cfg = pa.make_config(w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size, kvd, w.k_scale,
                         w.v_scale)
    return pa.pa_create(cfg)


def _args(w):
    return (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc, w.scale)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_noalloc_matches_pa_forward_twice_second_smaller(kv):
    big = W.make_batch([(1200, 1), (0, 300), (30, 1), (400, 65), (5000, 1), (0, 2)], 32, 8, 128,
                       kv_dtype=kv, seed=seed_of("noalloc_big" + kv), token_pad=3, device="cuda")
    # the second, smaller call: the first three sequences on the same cache
    # (the handle's fp8 scales are those of this cache)
    small = W.Workload(**{**big.__dict__})
    T3 = int(big.query_start_loc[3])
    small.q = big.q[:T3].contiguous()
    small.block_table = big.block_table[:3].contiguous()
    small.seq_lens = big.seq_lens[:3].contiguous()
    small.query_start_loc = big.query_start_loc[:4].contiguous()
    small.ctx_lens, small.q_lens = big.ctx_lens[:3], big.q_lens[:3]
    h = _handle_without_workspace(big)
    try:
        for w in (big, small):
            att = attention_for(w)
            ref = torch.full(w.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
            att.forward(*_args(w), out=ref)
            out = torch.full(w.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
            pa.pa_forward_noalloc(h, *_args(w), out)
            torch.cuda.synchronize()
            T = valid_token_count(w)
            assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), "differs from pa_forward"
            check_close(out.cpu()[:T], oracle_full(w)[:T], w.kv_fp8, "noalloc")
            assert (out[T:].float() == SENTINEL).all()
            att.close()
    finally:
        pa.pa_destroy(h)


def test_noalloc_rejects_a_batch_beyond_the_static_scratch():
    # 10^9 query rows (stride-0 views, nothing is read): the Q-block work
    # list alone needs ~375 MB, more than the scratch holds; refused before
    # launch.
    w = W.make_batch([(10, 1)], 8, 2, 128, seed=1, device="cuda")
    T = 1_000_000_000
    q = torch.zeros(1, 8, 128, dtype=torch.bfloat16, device="cuda").expand(T, 8, 128)
    out = torch.zeros(1, 8, 128, dtype=torch.bfloat16, device="cuda").expand(T, 8, 128)
    h = _handle_without_workspace(w)
    try:
        with pytest.raises(pa.PaError) as ei:
            pa.pa_forward_noalloc(h, q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                                  w.query_start_loc, w.scale, out)
        assert ei.value.status == pa.PA_ERR_WORKSPACE and "static scratch" in str(ei.value)
    finally:
        pa.pa_destroy(h)
