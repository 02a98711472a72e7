"""pa_forward_hinted: the host's knowledge of the batch (number of
single-token rows, longest query; the metadata of Sec. 6.1) skips launches
that would find no work, with the same results as pa_forward."""
import pytest
import torch

from paper_2511_11581_amd import pa
from paper_2511_11581_amd import workloads as W
from gpu_util import SENTINEL, attention_for, check_close, oracle_full, seed_of, valid_token_count

pytestmark = pytest.mark.gpu


def _hint_of(w):
    return (sum(1 for q in w.q_lens if q == 1), max(w.q_lens + [0]))


def _run(w, att, hint):
    wd = w.to("cuda")
    out = torch.full(wd.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
    att.forward(wd.q, wd.k_cache, wd.v_cache, wd.block_table, wd.seq_lens, wd.query_start_loc,
                w.scale, out=out, hint=hint)
    torch.cuda.synchronize()
    return out.cpu()


CASES = {
    "decode_only": ([(17, 1), (64, 1), (100, 1), (255, 1), (4000, 1)], 8, 2, 64, "bf16", 16),
    "prefill_only": ([(0, 300), (40, 77), (0, 2)], 16, 4, 128, "bf16", 16),
    "mixed": ([(1200, 1), (0, 90), (30, 1), (400, 65), (5000, 1), (0, 2)], 32, 8, 128, "fp8", 48),
    "decode_only_fp8": ([(3000, 1), (9, 1)], 16, 2, 128, "fp8", 16),
    # small mixed batches in other kernel shapes: every row as Q-blocks when hinted
    "mixed_d64": ([(300, 1), (0, 50), (40, 1), (100, 20), (700, 1)], 8, 2, 64, "bf16", 16),
    "mixed_fp8_d64": ([(0, 50), (130, 1), (60, 20), (2000, 1)], 8, 2, 64, "fp8", 32),
}


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("no_split", [False, True])
def test_hinted_equals_plain_forward(name, no_split):
    seqs, Hq, Hkv, d, kv, bs = CASES[name]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of("hint" + name),
                     name=name, token_pad=2)
    att = attention_for(w, no_split_kv=no_split)
    plain = _run(w, att, None)
    hint = _hint_of(w)
    hinted = _run(w, att, hint)
    route = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]), hint)["prefill_qmin"]
    if name.startswith("mixed"):   # small mixed batches: every row as Q-blocks when hinted
        assert route == 1
    if route == 1 and not no_split:
        ref = _run(w, attention_for(w, no_split_kv=True), None)   # the no-split path's kernels
    else:
        ref = plain
    assert torch.equal(ref.view(torch.int16), hinted.view(torch.int16))
    unknown = _run(w, att, (-1, -1))
    assert torch.equal(plain.view(torch.int16), unknown.view(torch.int16))
    T = valid_token_count(w)
    check_close(hinted[:T], oracle_full(w)[:T], w.kv_fp8, name)
    assert (hinted[T:].float() == SENTINEL).all()


def test_validate_reports_a_violated_hint():
    seqs, Hq, Hkv, d, kv, bs = CASES["mixed"]
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=3, name="hint_bad")
    att = attention_for(w, validate=True)
    for bad in ((0, -1), (-1, 1), (-1, 64)):   # decode rows exist; q up to 90
        with pytest.raises(pa.PaError) as ei:
            _run(w, att, bad)
        assert ei.value.status == pa.PA_ERR_DEVICE and "hint" in str(ei.value)
    _run(w, att, _hint_of(w))   # the true hint passes validation


def test_hint_fields_are_checked_on_the_host():
    w = W.make_batch([(10, 1)], 8, 2, 128, seed=1).to("cuda")
    att = attention_for(w)
    with pytest.raises(pa.PaError) as ei:
        _run(w, att, (-2, 1))
    assert ei.value.status == pa.PA_ERR_INVALID_ARG


@pytest.mark.parametrize("k", [1, 2, 5])
def test_decode_batches_without_plan_launch_bitwise(k):
    # decode-only batches with the hint: the decode kernel builds the decode
    # list in LDS itself (no plan launch) and publishes it for the merge;
    # same bits as the plan + decode + merge launches, call after call
    w = W.make_config(k, device="cuda")
    att = attention_for(w)
    plain = _run(w, att, None)
    for _ in range(2):
        fused = _run(w, att, _hint_of(w))
        assert torch.equal(plain.view(torch.int16), fused.view(torch.int16))


def test_in_kernel_list_merge_with_far_apart_piece_maxima():
    seqs = [(6000, 1), (9000, 1), (300, 1)]
    w = W.make_batch(seqs, 8, 2, 128, seed=seed_of("fused_spike"), name="fused_spike",
                     spikes=[(0, 4500, 0, 8.0), (1, 7000, 0, 8.0)])
    att = attention_for(w)
    out = _run(w, att, _hint_of(w))
    T = valid_token_count(w)
    check_close(out[:T], oracle_full(w)[:T], w.kv_fp8, "fused_spike")
    assert torch.equal(out.view(torch.int16), _run(w, att, None).view(torch.int16))


def test_in_kernel_list_replays_from_a_hip_graph():
    w = W.make_batch([(5000, 1), (17, 1), (2500, 1), (900, 1)], 32, 8, 128,
                     seed=seed_of("fused_graph"), name="fused_graph").to("cuda")
    att = attention_for(w)
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    hint = _hint_of(w)
    eager = torch.empty_like(w.q)
    att.forward(*args, out=eager, hint=hint)
    torch.cuda.synchronize()
    out = torch.empty_like(w.q)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        att.forward(*args, out=out, hint=hint)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        att.forward(*args, out=out, hint=hint)
    for rep in range(4):
        out.fill_(SENTINEL)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), f"replay {rep}"


def test_whole_pairs_replay_from_a_hip_graph_with_new_metadata():
    # Short sequences (table width 13 blocks of 16 = 6.5 steps of 32 keys):
    # whole pairs per workgroup, merged inside it, the decode list built in
    # the kernel (hinted decode-only call), no merge launch.  The graph
    # captured on batch A replays on batch B's contents (same shapes, other
    # lengths), and on A again, bitwise equal to the eager call.
    seqs_a = [((37 * i) % 200, 1) for i in range(70)]
    seqs_b = [((53 * i + 11) % 200, 1) for i in range(70)]
    need = max(sum((c + q + 15) // 16 for c, q in s) for s in (seqs_a, seqs_b))
    wa = W.make_batch(seqs_a, 32, 8, 128, seed=seed_of("whole_a"), pool_blocks=need, table_width=13,
                      name="whole_a").to("cuda")
    wb = W.make_batch(seqs_b, 32, 8, 128, seed=seed_of("whole_b"), pool_blocks=need, table_width=13,
                      name="whole_b").to("cuda")
    att = attention_for(wa, max_blocks=13)
    assert att.plan(wa.num_tokens, wa.num_seqs, 13)["decode_whole_units"] == 1
    args = (wa.q, wa.k_cache, wa.v_cache, wa.block_table, wa.seq_lens, wa.query_start_loc, wa.scale)
    hint = _hint_of(wa)
    eager = torch.empty_like(wa.q)
    att.forward(*args, out=eager, hint=hint)
    torch.cuda.synchronize()
    T = valid_token_count(wa)
    check_close(eager.cpu()[:T], oracle_full(wa)[:T], False, "whole pairs, eager")
    out = torch.empty_like(wa.q)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        att.forward(*args, out=out, hint=hint)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        att.forward(*args, out=out, hint=hint)
    saved = [x.clone() for x in args[:6]]
    for dst, src in zip(args[:6], (wb.q, wb.k_cache, wb.v_cache, wb.block_table, wb.seq_lens,
                                   wb.query_start_loc)):
        dst.copy_(src)
    for rep in range(2):
        out.fill_(SENTINEL)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check_close(out.cpu()[:T], oracle_full(wb)[:T], False, f"whole pairs, replay {rep} on batch B")
    for dst, src in zip(args[:6], saved):
        dst.copy_(src)
    out.fill_(SENTINEL)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), "replay on batch A"
