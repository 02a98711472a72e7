"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: torch's
fp64 scaled-dot-product attention on dense data, exact invariants, closed
forms, torch's fp8/bf16 decoders and the paper's worked partition example
(arxiv 2511.11581, Sec. 4.5, Fig. 4).
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2511_11581_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# Test-local construction of a paged cache from dense per-sequence K/V.
# (The oracle walks the table; these helpers scatter into it.)

def paged_from_dense(ks, vs, block_size, pool_extra=3, seed=0, poison=True):
    """ks/vs: list of [L_i, Hkv, d] tensors (bf16 or fp8).  Returns (k_cache,
    v_cache, block_table, seq_lens) with blocks placed at random physical ids."""
    g = torch.Generator().manual_seed(seed)
    L = [k.shape[0] for k in ks]
    nblk = [(x + block_size - 1) // block_size for x in L]
    NB = sum(nblk) + pool_extra
    Hkv, d = ks[0].shape[1], ks[0].shape[2]
    dt = ks[0].dtype
    perm = torch.randperm(NB, generator=g)
    MB = max(nblk + [1])
    table = torch.full((len(ks), MB), -1, dtype=torch.int32)
    kc = torch.zeros((NB, block_size, Hkv, d), dtype=torch.float32).to(dt)
    vc = torch.zeros_like(kc)
    if poison:
        if dt == torch.bfloat16:
            kc.view(torch.int16).fill_(0x7FC0)
            vc.view(torch.int16).fill_(0x7FC0)
        else:
            kc.view(torch.uint8).fill_(0x7F)
            vc.view(torch.uint8).fill_(0x7F)
    off = 0
    for i, (k, v) in enumerate(zip(ks, vs)):
        for b in range(nblk[i]):
            phys = int(perm[off + b])
            table[i, b] = phys
            lo, hi = b * block_size, min(L[i], (b + 1) * block_size)
            kc[phys, : hi - lo] = k[lo:hi]
            vc[phys, : hi - lo] = v[lo:hi]
        off += nblk[i]
    return kc, vc, table, torch.tensor(L, dtype=torch.int32)


def to_f64(t, scale=1.0):
    return t.to(torch.float64) * scale


def sdpa_reference(q, ks, vs, seqs, G, scale, k_scale=1.0, v_scale=1.0):
    """torch fp64 SDPA per sequence with an explicit bottom-right causal mask
    and KV heads repeated G times.  Returns [T, Hq, d]."""
    outs = []
    t0 = 0
    for (c, ql), k, v in zip(seqs, ks, vs):
        L = c + ql
        qq = to_f64(q[t0:t0 + ql]).permute(1, 0, 2)[None]            # [1, Hq, ql, d]
        kk = to_f64(k, k_scale).repeat_interleave(G, dim=1).permute(1, 0, 2)[None]
        vv = to_f64(v, v_scale).repeat_interleave(G, dim=1).permute(1, 0, 2)[None]
        mask = torch.arange(L)[None, :] <= (c + torch.arange(ql))[:, None]
        o = F.scaled_dot_product_attention(qq, kk, vv, attn_mask=mask, scale=scale)
        outs.append(o[0].permute(1, 0, 2))
        t0 += ql
    return torch.cat(outs, 0).numpy()


def lse_reference(q, ks, seqs, G, scale, k_scale=1.0):
    """Natural-log log-sum-exp of every row's causal scores, [T, Hq] (torch
    fp64 logsumexp over an explicit dense score matrix)."""
    outs = []
    t0 = 0
    for (c, ql), k in zip(seqs, ks):
        L = c + ql
        qq = to_f64(q[t0:t0 + ql]).permute(1, 0, 2)                  # [Hq, ql, d]
        kk = to_f64(k, k_scale).repeat_interleave(G, dim=1).permute(1, 2, 0)  # [Hq, d, L]
        s = scale * (qq @ kk)
        mask = torch.arange(L)[None, :] <= (c + torch.arange(ql))[:, None]
        s = s.masked_fill(~mask[None], float("-inf"))
        outs.append(torch.logsumexp(s, dim=-1).permute(1, 0))
        t0 += ql
    return torch.cat(outs, 0).numpy()


def rand_dense(seqs, Hq, Hkv, d, seed, fp8=False):
    g = torch.Generator().manual_seed(seed)
    T = sum(q for _, q in seqs)
    q = torch.randn(T, Hq, d, generator=g).to(torch.bfloat16)
    ks, vs = [], []
    for c, ql in seqs:
        L = c + ql
        k = torch.randn(L, Hkv, d, generator=g)
        v = torch.randn(L, Hkv, d, generator=g)
        if fp8:
            ks.append((k * 40).clamp(-448, 448).to(torch.float8_e4m3fn))
            vs.append((v * 40).clamp(-448, 448).to(torch.float8_e4m3fn))
        else:
            ks.append(k.to(torch.bfloat16))
            vs.append(v.to(torch.bfloat16))
    return q, ks, vs


def qsl_of(seqs):
    return torch.tensor([0] + list(np.cumsum([q for _, q in seqs])), dtype=torch.int32)


CASES = [
    # (seqs, Hq, Hkv, d, block_size, fp8)
    ([(0, 5), (3, 1), (7, 4), (0, 1)], 4, 2, 8, 4, False),
    ([(10, 1), (0, 9), (5, 6)], 8, 2, 16, 16, False),
    ([(2, 3), (17, 1)], 3, 3, 8, 3, False),           # MHA, non-power-of-two block
    ([(0, 7), (11, 2)], 8, 1, 8, 5, False),           # MQA
    ([(4, 2), (9, 1), (0, 3)], 4, 2, 8, 4, True),     # fp8 cache
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_matches_dense_fp64_sdpa(case):
    seqs, Hq, Hkv, d, bs, fp8 = CASES[case]
    q, ks, vs = rand_dense(seqs, Hq, Hkv, d, seed=100 + case, fp8=fp8)
    kc, vc, table, sl = paged_from_dense(ks, vs, bs, seed=case)
    scale = 1.0 / math.sqrt(d)
    ksc, vsc = (0.03, 0.02) if fp8 else (1.0, 1.0)
    ref = sdpa_reference(q, ks, vs, seqs, Hq // Hkv, scale, ksc, vsc)
    out, lse = oracle.forward(q, kc, vc, table, sl, qsl_of(seqs), scale, k_scale=ksc, v_scale=vsc,
                              with_lse=True)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lse_reference(q, ks, seqs, Hq // Hkv, scale, ksc),
                               rtol=0, atol=1e-12)


def test_block_permutation_invariance():
    w = W.make_batch([(20, 1), (0, 13), (37, 4)], 4, 2, 16, block_size=4, seed=3, pool_blocks=40)
    base = oracle.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                          w.query_start_loc, w.scale)
    g = torch.Generator().manual_seed(9)
    perm = torch.randperm(w.num_blocks, generator=g)           # old id -> new id
    kc = torch.empty_like(w.k_cache)
    vc = torch.empty_like(w.v_cache)
    kc[perm] = w.k_cache
    vc[perm] = w.v_cache
    table = w.block_table.clone()
    valid = table >= 0
    table[valid] = perm[table[valid].long()].to(torch.int32)
    out = oracle.forward(w.q, kc, vc, table, w.seq_lens, w.query_start_loc, w.scale)
    assert np.array_equal(out, base)


def test_single_key_returns_its_v_row():
    w = W.make_batch([(0, 1), (0, 1)], 6, 3, 16, block_size=16, seed=4)
    out = oracle.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                         w.query_start_loc, w.scale)
    for i in range(2):
        blk = int(w.block_table[i, 0])
        for h in range(6):
            expect = w.v_cache[blk, 0, h // 2].to(torch.float64).numpy()
            assert np.array_equal(out[i, h], expect)


def test_constant_v_returns_constant():
    w = W.make_batch([(30, 1), (0, 9), (12, 5)], 8, 2, 16, block_size=8, seed=5)
    c = torch.randn(2, 16, generator=torch.Generator().manual_seed(1)).to(torch.bfloat16)
    v = w.v_cache.clone()
    v[:] = c  # every slot of every block: V[p, g, :] = c[g, :]
    out = oracle.forward(w.q, w.k_cache, v, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    T = int(w.query_start_loc[-1])
    for h in range(8):
        np.testing.assert_allclose(out[:T, h], np.broadcast_to(c[h // 4].double().numpy(), (T, 16)),
                                   rtol=0, atol=1e-14)


def test_weights_sum_to_one_and_are_causal():
    w = W.make_batch([(9, 6), (40, 1)], 4, 1, 16, block_size=16, seed=6)
    rows = [(t, h) for t in range(7) for h in range(4)]
    out, wts = oracle.rows(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                           w.query_start_loc, w.scale, rows, max_keys=48)
    for k, (t, h) in enumerate(rows):
        nkeys = 9 + t + 1 if t < 6 else 41
        assert abs(wts[k].sum() - 1.0) <= 1e-12
        assert (wts[k, :nkeys] > 0).all()
        assert (wts[k, nkeys:] == 0).all()


def test_zero_keys_give_uniform_average():
    seqs = [(5, 4), (0, 6)]
    q, ks, vs = rand_dense(seqs, 4, 2, 8, seed=7)
    ks = [torch.zeros_like(k) for k in ks]
    kc, vc, table, sl = paged_from_dense(ks, vs, 4, seed=7)
    out = oracle.forward(q, kc, vc, table, sl, qsl_of(seqs), 0.5)
    t = 0
    for (c, ql), v in zip(seqs, vs):
        vd = v.double().numpy()
        for j in range(ql):
            for h in range(4):
                np.testing.assert_allclose(out[t + j, h], vd[: c + j + 1, h // 2].mean(0),
                                           rtol=0, atol=1e-14)
        t += ql


def test_two_keys_closed_form():
    # A 2-token prompt: row 0 sees key 0 only; row 1 mixes V0 and V1 with
    # weight sigmoid(s1 - s0) on V1, s_p = scale * <q, k_p>.
    seqs = [(0, 2)]
    q, ks, vs = rand_dense(seqs, 2, 1, 8, seed=8)
    kc, vc, table, sl = paged_from_dense(ks, vs, 16, seed=8)
    scale = 0.7
    out = oracle.forward(q, kc, vc, table, sl, qsl_of(seqs), scale)
    k = ks[0].double().numpy()[:, 0]
    v = vs[0].double().numpy()[:, 0]
    for h in range(2):
        qq = q[1, h].double().numpy()
        s0, s1 = scale * qq @ k[0], scale * qq @ k[1]
        sig = 1.0 / (1.0 + math.exp(-(s1 - s0)))
        np.testing.assert_allclose(out[1, h], v[0] + (v[1] - v[0]) * sig, rtol=0, atol=1e-13)
        np.testing.assert_array_equal(out[0, h], v[0])


def test_split_merge_identity():
    w = W.make_batch([(200, 3)], 4, 2, 16, block_size=16, seed=9)
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    rng = np.random.default_rng(0)
    for t, h in [(0, 0), (1, 3), (2, 1)]:
        nkeys = 200 + t + 1
        ref = oracle.rows(*args, [(t, h)])[0]
        for trial in range(4):
            cuts = sorted(rng.integers(0, nkeys + 1, size=trial + 2).tolist())
            bounds = [0] + cuts + [nkeys]       # may contain empty segments
            parts = [oracle.segment(*args, t, h, a, b) for a, b in zip(bounds[:-1], bounds[1:])]
            acc = np.stack([p[0] for p in parts])
            m = np.array([p[1] for p in parts])
            l = np.array([p[2] for p in parts])
            np.testing.assert_allclose(oracle.merge(acc, m, l), ref, rtol=0, atol=1e-13)
        # all segments but one empty
        parts = [oracle.segment(*args, t, h, 0, 0), oracle.segment(*args, t, h, 0, nkeys),
                 oracle.segment(*args, t, h, nkeys, nkeys)]
        acc = np.stack([p[0] for p in parts])
        out = oracle.merge(acc, np.array([p[1] for p in parts]), np.array([p[2] for p in parts]))
        np.testing.assert_allclose(out, ref, rtol=0, atol=1e-15)


def test_segment_partition_matches_paper_example():
    with open(os.path.join(GOLDEN, "fig4_segments.txt")) as f:
        lines = [x for x in f.read().splitlines() if x and not x.startswith("#")]
    for line in lines:
        head, tail = line.split("|")
        n, tps = (int(x) for x in head.split())
        expect = [tuple(int(x) for x in part.split()) for part in tail.split(";")]
        assert oracle.segment_ranges(n, tps) == expect
    # ragged tail: the last segment is shorter, none is empty
    assert oracle.segment_ranges(30, 8) == [(0, 8), (8, 16), (16, 24), (24, 30)]


def test_decode_equals_last_prefill_row():
    L = 77
    w = W.make_batch([(0, L)], 8, 2, 16, block_size=16, seed=10)
    pre = oracle.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                         w.query_start_loc, w.scale)
    qdec = w.q[L - 1:L].clone()
    dec = oracle.forward(qdec, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                         torch.tensor([0, 1], dtype=torch.int32), w.scale)
    assert np.array_equal(dec[0], pre[L - 1])


def test_chunked_prefill_equals_whole_prefill():
    L, a = 90, 37
    w = W.make_batch([(0, L)], 4, 4, 16, block_size=8, seed=11)
    whole = oracle.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                           w.query_start_loc, w.scale)
    chunk = oracle.forward(w.q[a:].clone(), w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                           torch.tensor([0, L - a], dtype=torch.int32), w.scale)
    assert np.array_equal(chunk, whole[a:])


def test_gqa_equals_repeated_head_mha():
    G = 4
    w = W.make_batch([(12, 3), (30, 1)], 8, 2, 16, block_size=16, seed=12)
    gqa = oracle.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                         w.query_start_loc, w.scale)
    kc = w.k_cache.repeat_interleave(G, dim=2).contiguous()
    vc = w.v_cache.repeat_interleave(G, dim=2).contiguous()
    mha = oracle.forward(w.q, kc, vc, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    assert np.array_equal(gqa, mha)


def test_fp8_decoder_matches_torch_for_all_codes():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = np.array([oracle.fp8e4m3_to_f64(c) for c in range(256)])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(ours))
    assert np.array_equal(ref[~nan], ours[~nan])
    assert nan.sum() == 2  # 0x7F and 0xFF


def test_bf16_decoder_matches_torch():
    g = torch.Generator().manual_seed(13)
    bits = torch.randint(0, 1 << 16, (4096,), generator=g, dtype=torch.int32)
    bits = torch.cat([bits, torch.tensor([0, 0x8000, 0x7F80, 0xFF80, 0x0001, 0x3F80])])
    b16 = (bits - (bits >= 32768).int() * 65536).to(torch.int16)
    ref = b16.view(torch.bfloat16).to(torch.float64).numpy()
    ours = np.array([oracle.bf16_to_f64(int(b) & 0xFFFF) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(ours))
    assert np.array_equal(ref[~nan], ours[~nan])


def test_poison_never_reaches_the_output():
    w = W.make_batch([(33, 1), (0, 7), (5, 2)], 4, 2, 16, block_size=16, seed=14,
                     pool_blocks=12, token_pad=3, table_width=6)
    out = oracle.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens,
                         w.query_start_loc, w.scale)
    T = int(w.query_start_loc[-1])
    assert np.isfinite(out[:T]).all()
    assert np.isnan(out[T:]).all()  # padding rows untouched


def test_threads_and_rows_agree_bitwise():
    w = W.make_batch([(100, 1), (0, 33), (64, 16)], 8, 2, 32, block_size=16, seed=15)
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    a = oracle.forward(*args, threads=1)
    b = oracle.forward(*args, threads=8)
    assert np.array_equal(a, b)
    sel = [(0, 5), (17, 2), (49, 7)]
    r = oracle.rows(*args, sel)
    for k, (t, h) in enumerate(sel):
        assert np.array_equal(r[k], a[t, h])


@pytest.mark.parametrize("bad", ["qsl0", "decreasing", "q_gt_L", "blk_oob", "L_gt_table"])
def test_malformed_metadata_is_rejected(bad):
    w = W.make_batch([(10, 2), (3, 1)], 4, 2, 8, block_size=4, seed=16, pool_blocks=8)
    qsl = w.query_start_loc.clone()
    sl = w.seq_lens.clone()
    bt = w.block_table.clone()
    if bad == "qsl0":
        qsl[0] = 1
    elif bad == "decreasing":
        qsl[1] = 3
        qsl[2] = 2
    elif bad == "q_gt_L":
        sl[1] = 0
    elif bad == "blk_oob":
        bt[0, 0] = 8
    elif bad == "L_gt_table":
        sl[0] = bt.shape[1] * 4 + 1
    with pytest.raises(oracle.OracleError):
        oracle.forward(w.q, w.k_cache, w.v_cache, bt, sl, qsl, w.scale)


def test_gather_walks_the_table():
    w = W.make_batch([(20, 1), (0, 5)], 4, 2, 8, block_size=4, seed=17, pool_blocks=16)
    kd, vd = oracle.gather(w.k_cache, w.v_cache, w.block_table, w.seq_lens)
    kb = w.k_cache.view(torch.int16).numpy().view(np.uint8)
    for i, L in enumerate(w.seq_len_list):
        for p in range(L):
            blk = int(w.block_table[i, p // 4])
            assert np.array_equal(kd[i, p].reshape(-1), kb[blk, p % 4].reshape(-1))
