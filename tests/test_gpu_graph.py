"""HIP-graph capture of pa_forward (Sec. 6.2: launches recorded once and
replayed; Sec. 4.7: a launch grid that does not depend on the batch's
lengths).  pa_forward allocates nothing and never synchronises, and its
grids depend only on host-visible shapes, so a captured call replays
correctly with whatever metadata and cache contents the captured tensors
hold at replay time."""
import pytest
import torch

from gpu_util import SENTINEL, attention_for, check_close, oracle_full, run_gpu, valid_token_count
from paper_2511_11581_amd import workloads as W

pytestmark = pytest.mark.gpu

# decode rows, prefill rows and a chunked-prefill row in one batch
SEQS_A = [(1200, 1), (0, 90), (30, 1), (400, 65), (5000, 1), (0, 2)]
# same query lengths (same token count), other contexts, different order of
# decode and prefill rows
SEQS_B = [(3000, 1), (10, 90), (700, 1), (0, 65), (40, 1), (2500, 2)]


def _capture(att, w, out):
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        att.forward(*args, out=out)          # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        att.forward(*args, out=out)
    return g


def test_graph_replays_match_eager_bitwise():
    w = W.make_batch(SEQS_A, 32, 8, 128, seed=21, name="graph_a").to("cuda")
    att = attention_for(w)
    eager = run_gpu(w, att)
    out = torch.empty_like(w.q)
    g = _capture(att, w, out)
    T = valid_token_count(w)
    for rep in range(4):
        out.fill_(SENTINEL)                  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = out.cpu()
        assert torch.equal(got[:T], eager[:T]), f"replay {rep} differs from the eager call"


def test_graph_replay_follows_new_metadata_and_cache():
    # both batches in pools and tables of the same shape
    need = max(sum((c + q + 15) // 16 for c, q in s) for s in (SEQS_A, SEQS_B))
    width = max((c + q + 15) // 16 for s in (SEQS_A, SEQS_B) for c, q in s)
    wa = W.make_batch(SEQS_A, 32, 8, 128, seed=22, pool_blocks=need, table_width=width,
                      name="graph_a").to("cuda")
    wb = W.make_batch(SEQS_B, 32, 8, 128, seed=23, pool_blocks=need, table_width=width,
                      name="graph_b").to("cuda")
    assert wa.q.shape == wb.q.shape and wa.block_table.shape == wb.block_table.shape
    att = attention_for(wa, max_blocks=width)
    out = torch.empty_like(wa.q)
    g = _capture(att, wa, out)
    # the captured tensors now take batch B's contents
    for dst, src in ((wa.q, wb.q), (wa.k_cache, wb.k_cache), (wa.v_cache, wb.v_cache),
                     (wa.block_table, wb.block_table), (wa.seq_lens, wb.seq_lens),
                     (wa.query_start_loc, wb.query_start_loc)):
        dst.copy_(src)
    for rep in range(3):
        out.fill_(SENTINEL)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        T = valid_token_count(wb)
        check_close(out.cpu()[:T], oracle_full(wb)[:T], False, f"graph replay {rep} on batch B")
