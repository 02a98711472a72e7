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


def _prefill_seqs(n, seed, ctx_max=3000, q_max=600):
    g = torch.Generator().manual_seed(seed)
    return [(int(torch.randint(0, ctx_max + 1, (1,), generator=g)),
             int(torch.randint(2, q_max + 1, (1,), generator=g))) for _ in range(n)]


FUSED = {
    # name: (seqs, Hq, Hkv, d, kv, bs, forced Q-block rows or None, hinted)
    "pf8_short_prompts": ([(0, 200)] * 8, 32, 8, 128, "bf16", 16, None, True),
    "pf16_g4": (_prefill_seqs(16, 1, 2000, 120), 32, 8, 128, "bf16", 16, None, True),
    "pf9_g8_d64": (_prefill_seqs(9, 2, 3000, 200), 16, 2, 64, "bf16", 32, None, True),
    "pf6_fp8": (_prefill_seqs(6, 3, 3000, 150), 32, 8, 128, "fp8", 16, None, True),
    "pf5_fp8_d64": (_prefill_seqs(5, 7, 3000, 150), 16, 4, 64, "fp8", 16, None, True),
    "pf5_rows128": (_prefill_seqs(5, 4, 3000, 300), 32, 8, 128, "bf16", 16, 128, True),
    "pf4_g1_bs400": (_prefill_seqs(4, 5, 1500, 300), 8, 8, 128, "bf16", 400, None, True),
    "pf3_long_ctx": ([(40000, 130), (0, 2), (9000, 700)], 32, 8, 128, "bf16", 16, None, True),
    # a small mixed batch run as Q-blocks only (single-token rows included)
    "mixed_small_unified": ([(300, 1), (0, 50), (40, 1), (100, 20), (700, 1)], 8, 2, 64, "bf16", 16, None,
                            True),
    # beyond the route: more sequences, or more Q-blocks than two rounds
    "pf17_planned": (_prefill_seqs(17, 6, 800, 100), 32, 8, 128, "bf16", 16, None, True),
    "pf4_beyond_two_rounds": ([(0, 3000), (0, 2048), (0, 1500), (0, 1000)], 32, 8, 128, "bf16", 16, None, True),
}


@pytest.mark.parametrize("name", list(FUSED))
def test_fused_plan_route(name, monkeypatch):
    # Batches of at most 16 sequences with no split-KV decode launch, whose
    # Q-blocks fit two rounds of workgroups, launch the Q-block kernel alone,
    # each workgroup deriving its record; the results equal the planned
    # launch's bit for bit (a Q-block's result does not depend on which
    # workgroup computes it) and the oracle's within tolerance.
    seqs, Hq, Hkv, d, kv, bs, rows, hinted = FUSED[name]
    if rows is not None:
        monkeypatch.setenv("PA_QBLOCK_ROWS", str(rows))
    w = W.make_batch(seqs, Hq, Hkv, d, kv_dtype=kv, block_size=bs, seed=seed_of("fused" + name),
                     name=name, token_pad=3)
    wd = w.to("cuda")
    att = pa.PagedAttention(w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size,
                            w.k_cache.dtype, w.k_scale, w.v_scale, max_tokens=w.num_tokens,
                            max_seqs=w.num_seqs, max_blocks_per_seq=int(w.block_table.shape[1]),
                            profile=True)

    def run(hint):
        out = torch.full(wd.q.shape, SENTINEL, dtype=torch.bfloat16, device="cuda")
        att.profile(reset=True)
        att.forward(wd.q, wd.k_cache, wd.v_cache, wd.block_table, wd.seq_lens,
                    wd.query_start_loc, w.scale, out=out, hint=hint)
        torch.cuda.synchronize()
        return out.cpu(), att.profile(reset=True)

    hint = _hint_of(w)
    plan = att.plan(w.num_tokens, w.num_seqs, int(w.block_table.shape[1]), hint)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    no_decode = plan["prefill_qmin"] == 1 or hint[0] == 0   # no split-KV decode launch
    fused_route = (w.num_seqs <= 16 and no_decode and plan["prefill_launch"] == 1
                   and plan["prefill_units"] <= 2 * cus * (256 // plan["block_m"]))
    # the planned launch: the unhinted call (the plan kernel in front of the
    # Q-blocks; for the mixed batch the decode rows split instead)
    planned, prof_p = run(None)
    fused, prof_f = run(hint)
    assert prof_p["plan"][0] == 1 and prof_p["prefill"][0] == 1
    assert prof_f["prefill"][0] == 1 and prof_f["decode"][0] == 0
    assert prof_f["plan"][0] == (0 if fused_route else 1), (name, plan)
    T = valid_token_count(w)
    if plan["prefill_qmin"] == 2:   # the same Q-blocks either way: equal bit for bit
        assert torch.equal(planned.view(torch.int16), fused.view(torch.int16)), name
    check_close(fused[:T], oracle_full(w)[:T], w.kv_fp8, name)
    assert (fused[T:].float() == SENTINEL).all()
    att.close()


def test_plan_free_q_blocks_replay_from_a_hip_graph_with_new_metadata():
    # A hinted prefill batch small enough that each Q-block workgroup finds
    # its own work item (no plan launch): the graph captured on batch A
    # replays on batch B's contents (same shapes, other lengths and
    # contexts), each replay checked against the oracle, and on A again,
    # bitwise equal to the eager call.
    seqs_a = [(500, 100), (0, 50), (230, 30), (61, 20), (399, 40), (7, 60)]
    seqs_b = [(30, 60), (420, 40), (0, 20), (300, 30), (125, 50), (530, 100)]
    need = max(sum((c + q + 15) // 16 for c, q in s) for s in (seqs_a, seqs_b))
    wa = W.make_batch(seqs_a, 32, 8, 128, seed=seed_of("pfree_a"), pool_blocks=need, table_width=40,
                      name="pfree_a").to("cuda")
    wb = W.make_batch(seqs_b, 32, 8, 128, seed=seed_of("pfree_b"), pool_blocks=need, table_width=40,
                      name="pfree_b").to("cuda")
    att = attention_for(wa, max_blocks=40)
    hint = (0, 100)
    p = att.plan(wa.num_tokens, wa.num_seqs, 40, hint)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert wa.num_seqs <= 16 and p["prefill_units"] <= cus * (256 // p["block_m"])   # the plan-free route
    args = (wa.q, wa.k_cache, wa.v_cache, wa.block_table, wa.seq_lens, wa.query_start_loc, wa.scale)
    eager = torch.empty_like(wa.q)
    att.forward(*args, out=eager, hint=hint)
    torch.cuda.synchronize()
    T = valid_token_count(wa)
    check_close(eager.cpu()[:T], oracle_full(wa)[:T], False, "plan-free Q-blocks, eager")
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
    TB = valid_token_count(wb)
    for rep in range(2):
        out.fill_(SENTINEL)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check_close(out.cpu()[:TB], oracle_full(wb)[:TB], False, f"plan-free Q-blocks, replay {rep} on batch B")
    for dst, src in zip(args[:6], saved):
        dst.copy_(src)
    out.fill_(SENTINEL)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), "replay on batch A"
