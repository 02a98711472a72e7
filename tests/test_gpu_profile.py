"""PA_FLAG_PROFILE: per-kernel launch counts and durations (pa_profile_read),
stamped by the runtime on each kernel's own dispatch.  Profiling changes no
result, and the kernels' summed durations fit inside the calls' wall time."""
import pytest
import torch

from paper_2511_11581_amd import pa
from paper_2511_11581_amd import workloads as W
from gpu_util import SENTINEL, seed_of

pytestmark = pytest.mark.gpu

CASES = {
    # name: (seqs, Hq, Hkv, d, kv, bs, hinted)
    "mixed": ([(1200, 1), (0, 90), (30, 1), (400, 65), (5000, 1), (0, 2)], 16, 4, 128, "bf16", 16, False),
    "mixed_fp8_d64": ([(0, 300), (130, 1), (60, 20), (9000, 1)], 8, 2, 64, "fp8", 32, False),
    "decode_only_hinted": ([(17, 1), (6400, 1), (100, 1), (2550, 1)], 32, 8, 128, "bf16", 16, True),
    "prefill_only_hinted": ([(0, 700), (40, 77), (0, 2)], 32, 8, 128, "bf16", 16, True),
}
CALLS = 12


def _handle(w, profile):
    return pa.PagedAttention(w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size, w.k_cache.dtype,
                             w.k_scale, w.v_scale, max_tokens=w.num_tokens, max_seqs=w.num_seqs,
                             max_blocks_per_seq=int(w.block_table.shape[1]), profile=profile)


def _calls(w, att, hint, n):
    out = torch.full(w.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    att.forward(*args, out=out, hint=hint)   # warm-up (not read from the profile: reset below)
    torch.cuda.synchronize()
    att.profile(reset=True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(n):
        att.forward(*args, out=out, hint=hint)
    ev1.record()
    torch.cuda.synchronize()
    return out.cpu(), ev0.elapsed_time(ev1)


@pytest.mark.parametrize("name", list(CASES))
def test_profile_counts_durations_and_results(name):
    seqs, Hq, Hkv, d, kv, bs, hinted = CASES[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of(name), name=name,
                     device="cuda")
    hint = (sum(1 for q in w.q_lens if q == 1), max(w.q_lens)) if hinted else None
    plain = _handle(w, profile=False)
    ref, _ = _calls(w, plain, hint, 1)
    att = _handle(w, profile=True)
    got, wall_ms = _calls(w, att, hint, CALLS)
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), f"{name}: profiling changed the output"

    prof = att.profile(reset=True)
    plan = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]), hint)
    has_decode = any(q == 1 for q in w.q_lens)
    has_prefill = any(q >= 2 for q in w.q_lens)
    launched = {k: n for k, (n, _) in prof.items()}
    # every kernel the batch needs ran once per call; a hint rules the others out
    assert launched["decode"] == (CALLS if has_decode else 0), (name, prof)
    assert launched["prefill"] == (CALLS if has_prefill else 0), (name, prof)
    assert launched["merge"] in ((CALLS if plan["merge_launch"] and has_decode else 0),), (name, prof, plan)
    if not hinted:
        assert launched["plan"] == CALLS, (name, prof)
    total = 0.0
    for k, (n, ms) in prof.items():
        if n:
            assert ms > 0.0, (name, k, prof)
        total += ms
    # the kernels of one stream run one after another inside the timed calls
    assert total <= wall_ms * 1.02 + 0.01, f"{name}: kernels {total:.3f} ms > wall {wall_ms:.3f} ms ({prof})"
    plain.close()
    att.close()
