"""Host-side tests of the C ABI: the library loads and exports every function
declared in include/pa.h, the header is plain C whose struct layout matches
the binding, and the launch planner's decisions (no GPU needed)."""
import ctypes
import itertools
import os
import re
import subprocess

import pytest
import torch

from paper_2511_11581_amd import pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pa.h")
GOLDEN = os.path.join(ROOT, "tests", "golden")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pa_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = pa.load_library()
    declared = header_functions()
    assert sorted(pa.EXPORTS) == declared
    for name in declared:
        assert hasattr(lib, name), name


def test_header_is_plain_c_and_matches_binding_layout(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(r'''
#include <stddef.h>
#include <stdio.h>
#include "pa.h"
int main(void) {
  printf("%zu %zu %zu %zu\n", sizeof(pa_tensor), offsetof(pa_tensor, shape), offsetof(pa_tensor, stride), sizeof(pa_config));
  printf("%zu %zu %zu %zu\n", offsetof(pa_config, workspace), offsetof(pa_config, workspace_bytes), sizeof(pa_plan_info), offsetof(pa_plan_info, decode_grid));
  printf("%zu\n", offsetof(pa_plan_info, workspace_bytes));
  return 0;
}
''')
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER),
                           str(src), "-o", str(exe)])
    vals = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    expect = [ctypes.sizeof(pa.pa_tensor), pa.pa_tensor.shape.offset, pa.pa_tensor.stride.offset,
              ctypes.sizeof(pa.pa_config), pa.pa_config.workspace.offset,
              pa.pa_config.workspace_bytes.offset, ctypes.sizeof(pa.pa_plan_info),
              pa.pa_plan_info.decode_grid.offset, pa.pa_plan_info.workspace_bytes.offset]
    assert vals == expect


def cfg(Hq=32, Hkv=8, d=128, bs=16, kv=pa.PA_DTYPE_BF16):
    return pa.make_config(Hq, Hkv, d, bs, kv)


def plan(c, cus=256, T=1, S=1, MB=1):
    return pa.pa_plan(None, c, cus, T, S, MB)


def fig4_example():
    line = [x for x in open(os.path.join(GOLDEN, "fig4_segments.txt")).read().splitlines()
            if x and not x.startswith("#")][0]
    head, tail = line.split("|")
    n_tiles, tps = (int(x) for x in head.split())
    return n_tiles, tps, [tuple(int(x) for x in part.split()) for part in tail.split(";")]


def test_plan_reproduces_the_papers_partition_example(monkeypatch):
    # Fig. 4 (Sec. 4.5): the tiles of one long decode row are distributed over
    # segments of 8 tiles, here 32 tiles over 4 segments (the minimum share
    # set to the figure's segment length; the default is 1 step).
    n_tiles, tps, expect = fig4_example()
    monkeypatch.setenv("PA_DECODE_MIN_STEPS", str(tps))
    c = cfg(4, 1, 128)
    p = plan(c, cus=256, T=1, S=1, MB=n_tiles * 2)
    assert p["decode_step"] == 32 and p["decode_min_steps"] == tps
    L = n_tiles * p["decode_step"]
    pcs = pa.pa_decode_pieces(None, c, 256, [L], [0, 1], 1, n_tiles * 2)
    got = [(x["first_key"] // 32, x["end_key"] // 32) for x in pcs]
    assert got == expect
    assert len({x["worker"] for x in pcs}) == len(expect)
    # the first segment continues on the next worker (tail slot), the others
    # start inside the row (head slot); all of them are merged
    assert [x["slot"] for x in pcs] == [1] + [0] * (len(expect) - 1)


def check_partition(c, cus, seq_lens, qsl, T, MB):
    """Every decode row's keys are covered once, in order, by pieces of
    consecutive workers; a worker computes the HU adjacent kv heads of a unit
    together (the same keys for each); the workers' unit step counts differ
    by at most one."""
    p = plan(c, cus=cus, T=T, S=len(seq_lens), MB=MB)
    KS = p["decode_step"]
    HU = p["decode_unit_heads"]
    pcs = pa.pa_decode_pieces(None, c, cus, seq_lens, qsl, T, MB)
    cap = MB * c.block_size
    rows = {}
    for x in pcs:
        rows.setdefault((x["seq"], x["kv_head"]), []).append(x)
    decode = [i for i in range(len(seq_lens))
              if qsl[i + 1] - qsl[i] == 1 and 0 <= qsl[i] < T and min(seq_lens[i], cap) >= 1]
    assert sorted(rows) == sorted((i, g) for i in decode for g in range(c.num_kv_heads))
    for (i, g), lst in rows.items():
        L = min(seq_lens[i], cap)
        assert lst[0]["first_key"] == 0 and lst[-1]["end_key"] == L
        for x, y in zip(lst, lst[1:]):
            assert x["end_key"] == y["first_key"] and y["worker"] == x["worker"] + 1
            assert x["end_key"] % KS == 0
        if len(lst) == 1:
            assert lst[0]["slot"] == -1
        else:
            assert lst[0]["slot"] == 1 and all(x["slot"] == 0 for x in lst[1:])
    # unit pieces: HU consecutive entries, heads HU u .. HU u + HU - 1, same keys
    assert len(pcs) % HU == 0
    for i in range(0, len(pcs), HU):
        grp = pcs[i:i + HU]
        assert [x["kv_head"] for x in grp] == list(range(grp[0]["kv_head"], grp[0]["kv_head"] + HU))
        assert grp[0]["kv_head"] % HU == 0
        assert all((x["seq"], x["worker"], x["first_key"], x["end_key"], x["slot"]) ==
                   (grp[0]["seq"], grp[0]["worker"], grp[0]["first_key"], grp[0]["end_key"], grp[0]["slot"])
                   for x in grp)
    steps = {}
    for x in pcs[::HU]:
        steps[x["worker"]] = steps.get(x["worker"], 0) + -(-(x["end_key"] - x["first_key"]) // KS)
        # a worker holds at most one piece per partial slot
    for w in steps:   # per unit piece (its HU heads share the slot, one row each)
        slots = [x["slot"] for x in pcs[::HU] if x["worker"] == w and x["slot"] >= 0]
        assert len(slots) == len(set(slots))
    if steps and p["decode_whole_units"]:
        # whole pairs: workgroup b takes pairs [b U / B, (b + 1) U / B) in
        # order, B = min(U, workgroups); a pair of nt steps is cut evenly
        # over the first min(4, nt) waves of its workgroup
        nw = p["decode_waves"]
        firsts = [x for x in pcs[::HU] if x["first_key"] == 0]   # one per pair, in order
        U = len(firsts)
        B = min(U, p["decode_workers"] // nw)
        for u, x in enumerate(firsts):
            b = next(b for b in range(B) if b * U // B <= u < (b + 1) * U // B)
            assert x["worker"] == b * nw
            row = rows[(x["seq"], x["kv_head"])]
            nt = -(-row[-1]["end_key"] // KS)
            n = min(nw, nt)
            assert [(y["first_key"] // KS, -(-y["end_key"] // KS)) for y in row] == \
                [(i * nt // n, (i + 1) * nt // n) for i in range(n)]
    elif steps:
        assert sorted(steps) == list(range(len(steps)))
        assert max(steps.values()) - min(steps.values()) <= 1
        total = sum(steps.values())   # steps of the unit space
        W = len(steps)
        assert W == min(p["decode_workers"], -(-total // p["decode_min_steps"]))
    return pcs


@pytest.mark.parametrize("seed", range(6))
def test_decode_partition_covers_every_key_once(seed):
    g = torch.Generator().manual_seed(seed)
    S = int(torch.randint(1, 200, (1,), generator=g))
    MB = int(torch.randint(1, 300, (1,), generator=g))
    bs = [16, 32, 64][seed % 3]
    q = torch.randint(0, 3, (S,), generator=g)
    q[torch.rand(S, generator=g) < 0.7] = 1
    L = torch.minimum(torch.randint(1, MB * bs + 1, (S,), generator=g) + q, torch.tensor(MB * bs))
    L = torch.maximum(L, q)
    qsl = [0] + torch.cumsum(q, 0).tolist()
    T = qsl[-1] + 3
    for Hq, Hkv, d, kv in [(32, 8, 128, pa.PA_DTYPE_BF16), (64, 8, 128, pa.PA_DTYPE_FP8_E4M3),
                           (8, 2, 64, pa.PA_DTYPE_BF16)]:
        check_partition(cfg(Hq, Hkv, d, bs, kv), [1, 80, 256][seed % 3], L.tolist(), qsl, T, MB)


def test_decode_partition_of_the_benchmark_decode_batch():
    # 64 decode rows up to 8193 keys: all 1024 workers busy, one step apart
    from paper_2511_11581_amd import workloads as W
    w = W.make_config(2, device="cpu", poison=False)
    c = cfg(32, 8, 128)
    pcs = check_partition(c, 256, w.seq_lens.tolist(), w.query_start_loc.tolist(), w.num_tokens,
                          int(w.block_table.shape[1]))
    assert len({x["worker"] for x in pcs}) == 1024


def test_plan_decode_grid_is_static():
    for S, MB in [(1, 1), (64, 513), (16, 8193)]:
        p = plan(cfg(), cus=256, T=S, S=S, MB=MB)
        whole = -(-MB * 16 // p["decode_step"]) <= 8
        assert p["decode_launch"] == 1 and p["merge_launch"] == (0 if whole else 1)
        assert p["decode_whole_units"] == (1 if whole else 0)
        assert p["decode_workers"] == 256 * 4
        assert p["decode_grid"] == [p["decode_workers"] // p["decode_waves"], 1, 1]
    assert plan(cfg(), cus=80, T=4, S=4, MB=4)["decode_workers"] == 80 * 4
    assert plan(cfg(64, 8, 128, 16, pa.PA_DTYPE_FP8_E4M3))["decode_step"] == 32
    assert plan(cfg(64, 8, 128, 16, pa.PA_DTYPE_FP8_E4M3))["decode_workers"] == 256 * 4
    assert plan(cfg(8, 2, 64))["decode_step"] == 32   # two heads per unit: 256-byte runs
    assert plan(cfg(8, 2, 64, 16, pa.PA_DTYPE_FP8_E4M3))["decode_step"] == 32  # two 64-byte heads per unit: 128-byte runs of fp8


def test_short_sequences_take_whole_pairs_without_merge(monkeypatch):
    # the tiny decode batch (contexts up to 255, table width 16 blocks of 16):
    # at most 8 steps per pair, so whole pairs per worker and no merge launch
    from paper_2511_11581_amd import workloads as W
    w = W.make_config(1, device="cpu", poison=False)
    c = cfg(8, 2, 64)
    MB = int(w.block_table.shape[1])
    p = plan(c, cus=256, T=w.num_tokens, S=w.num_seqs, MB=MB)
    assert p["decode_whole_units"] == 1 and p["merge_launch"] == 0
    pcs = check_partition(c, 256, w.seq_lens.tolist(), w.query_start_loc.tolist(), w.num_tokens, MB)
    # lengths 18, 65, 101, 256 (context + the new token) = 1, 3, 4, 8 steps of
    # 32 keys: one workgroup per sequence (Hkv 2 in one unit), its pieces on
    # 1, 3, 4, 4 waves
    assert w.seq_lens.tolist() == [18, 65, 101, 256]
    assert [sum(1 for x in pcs if x["seq"] == i and x["kv_head"] == 0) for i in range(4)] == [1, 3, 4, 4]
    assert {x["worker"] // 4 for x in pcs if x["seq"] == 3} == {3}
    # one step more than the limit (a wider table) splits again
    p = plan(c, cus=256, T=w.num_tokens, S=w.num_seqs, MB=8 * p["decode_step"] // 16 + 1)
    assert p["decode_whole_units"] == 0 and p["merge_launch"] == 1
    # PA_DECODE_WHOLE_STEPS=0 turns it off
    monkeypatch.setenv("PA_DECODE_WHOLE_STEPS", "0")
    p = plan(c, cus=256, T=w.num_tokens, S=w.num_seqs, MB=MB)
    assert p["decode_whole_units"] == 0 and p["merge_launch"] == 1
    pcs = check_partition(c, 256, w.seq_lens.tolist(), w.query_start_loc.tolist(), w.num_tokens, MB)
    assert len({x["worker"] for x in pcs}) == 16   # 16 steps in all, one per worker


def test_small_mixed_batch_runs_every_row_as_q_blocks(monkeypatch):
    # 8 single-token rows and 8 chunks of 128 tokens, contexts up to 4096
    from paper_2511_11581_amd import workloads as W
    c = cfg()
    T, S, MB = 8 + 8 * 128, 16, (4096 + 128) // 16 + 1
    p = plan(c, T=T, S=S, MB=MB)                     # pa_forward: split-KV decode + Q-blocks
    assert p["prefill_qmin"] == 2 and p["decode_launch"] == 1 and p["merge_launch"] == 1
    ph = pa.pa_plan(None, c, 256, T, S, MB, (8, 128))   # pa_forward_hinted: one Q-block launch
    assert ph["prefill_qmin"] == 1 and ph["decode_launch"] == 0 and ph["merge_launch"] == 0
    assert ph["prefill_units"] <= 256 * (256 // ph["block_m"])
    assert ph["workspace_bytes"] <= pa.pa_workspace_bytes(c, T, S, MB)
    # not for decode-only or prefill-only batches, tables past 8192 keys,
    # or more Q-blocks than one round of workgroups (the mixed benchmark batch)
    assert pa.pa_plan(None, c, 256, 8, 8, MB, (8, 1))["prefill_qmin"] == 2
    assert pa.pa_plan(None, c, 256, T, S, MB, (0, 128))["prefill_qmin"] == 2
    assert pa.pa_plan(None, c, 256, T, S, 8192 // 16 + 1, (8, 128))["prefill_qmin"] == 2
    seqs = W.config_seqs(4)[0]   # its shape only: 128 sequences, 4216 tokens
    T4, MB4 = sum(q for _, q in seqs), max(-(-(c + q) // 16) for c, q in seqs)
    assert pa.pa_plan(None, c, 256, T4, len(seqs), MB4, (120, 512))["prefill_qmin"] == 2
    monkeypatch.setenv("PA_UNIFY_MAX_KEYS", "0")
    assert pa.pa_plan(None, c, 256, T, S, MB, (8, 128))["prefill_qmin"] == 2


def test_decode_unit_heads_make_runs_of_256_bytes():
    F8 = pa.PA_DTYPE_FP8_E4M3
    assert plan(cfg(32, 8, 128))["decode_unit_heads"] == 1          # 256-byte bf16 rows
    assert plan(cfg(64, 8, 128, 16, F8))["decode_unit_heads"] == 2  # 128-byte fp8 rows
    assert plan(cfg(8, 2, 64))["decode_unit_heads"] == 2            # 128-byte bf16 rows
    assert plan(cfg(32, 8, 64, 16, F8))["decode_unit_heads"] == 4   # 64-byte fp8 rows
    assert plan(cfg(8, 2, 64, 16, F8))["decode_unit_heads"] == 2    # limited by Hkv
    assert plan(cfg(8, 1, 128, 16, F8))["decode_unit_heads"] == 1
    assert plan(cfg(12, 3, 128, 16, F8))["decode_unit_heads"] == 1  # Hkv odd


@pytest.mark.parametrize("kv,d,hkv", [("fp8", 128, 8), ("bf16", 64, 2), ("fp8", 64, 8)])
def test_decode_partition_with_head_units(kv, d, hkv):
    g = torch.Generator().manual_seed(d + hkv)
    S = 37
    L = torch.randint(1, 3000, (S,), generator=g).tolist()
    qsl = list(range(S + 1))
    dt = pa.PA_DTYPE_FP8_E4M3 if kv == "fp8" else pa.PA_DTYPE_BF16
    c = cfg(4 * hkv, hkv, d, 16, dt)
    assert plan(c)["decode_unit_heads"] > 1
    check_partition(c, 80, L, qsl, S, 200)


def test_plan_prefill_grid_bounds_the_q_blocks():
    p = plan(cfg(), cus=256, T=6589, S=4, MB=188)
    assert p["prefill_launch"] == 1
    assert p["block_m"] == 256 and p["block_q"] == 64   # bf16 caches: 8 waves x 32 rows
    # sum ceil(q_i / BLOCK_Q) <= ceil(T / BLOCK_Q) + S
    qs = [2048, 1024, 3000, 517]
    need = sum(-(-q // 64) for q in qs)
    assert p["prefill_units"] >= need * 8
    assert p["prefill_grid"][0] == p["prefill_units"]   # one workgroup per (Q-block, kv head)
    # fp8 caches: the 8-wave kernel (its staging needs 8 waves) for d = 128 and 64
    pf = plan(cfg(32, 8, 128, 16, pa.PA_DTYPE_FP8_E4M3), cus=256, T=6589, S=4, MB=188)
    assert pf["block_m"] == 256 and pf["block_q"] == 64
    pf64 = plan(cfg(32, 8, 64, 16, pa.PA_DTYPE_FP8_E4M3), cus=256, T=6589, S=4, MB=188)
    assert pf64["block_m"] == 256 and pf64["block_q"] == 64
    p1 = plan(cfg(), T=1, S=1, MB=4)
    assert p1["prefill_launch"] == 0


@pytest.mark.parametrize("S,q,ctx,Hq,rows", [
    (4, 2048, 0, 32, 256),      # varlen-prefill-like: long prompts, several grid waves
    (16, 4096, 4096, 32, 256),  # large batch over long keys
    (1, 64, 4096, 32, 128),     # short prompt on a long context: few units
    (64, 16, 4096, 32, 128),    # many short chunks
    (32, 256, 0, 64, 128),      # short prompts, G = 8
    (1, 4096, 0, 32, 256),
])
def test_plan_q_block_rows_follow_the_tuned_tree(S, q, ctx, Hq, rows):
    # The exported rule of the offline BLOCK_M sweep (Sec. 5 / Fig. 8): the
    # faster of the two Q-block shapes on each swept batch.
    MB = -(-(q + ctx) // 16)
    p = plan(cfg(Hq, 8, 128), cus=256, T=S * q, S=S, MB=MB)
    assert p["block_m"] == rows and p["block_q"] == rows // (Hq // 8)


def test_plan_q_block_rows_can_be_forced(monkeypatch):
    monkeypatch.setenv("PA_QBLOCK_ROWS", "128")
    assert plan(cfg(), cus=256, T=6589, S=4, MB=188)["block_m"] == 128
    monkeypatch.setenv("PA_QBLOCK_ROWS", "256")
    assert plan(cfg(), cus=256, T=64, S=4, MB=16)["block_m"] == 256
    monkeypatch.setenv("PA_QBLOCK_ROWS", "100")   # not a kernel shape: ignored
    assert plan(cfg(), cus=256, T=64, S=4, MB=16)["block_m"] == 128


@pytest.mark.parametrize("Hq,Hkv,d,bs,kv,status", [
    (32, 8, 128, 16, pa.PA_DTYPE_BF16, pa.PA_OK),
    (12, 4, 128, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),   # G = 3
    (64, 2, 128, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),   # G = 32
    (32, 8, 96, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),
    (32, 8, 128, 8, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),
    (32, 8, 128, 24, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),    # not a multiple of 16
    (32, 8, 128, 48, pa.PA_DTYPE_BF16, pa.PA_OK),
    (32, 8, 128, 528, pa.PA_DTYPE_FP8_E4M3, pa.PA_OK),
    (32, 8, 128, (1 << 20) + 16, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),
    (30, 8, 128, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_INVALID_ARG),
    (32, 8, 128, 16, pa.PA_DTYPE_F32, pa.PA_ERR_UNSUPPORTED),
    (32, 8, 128, 32, pa.PA_DTYPE_FP8_E4M3, pa.PA_OK),
])
def test_config_validation(Hq, Hkv, d, bs, kv, status):
    c = cfg(Hq, Hkv, d, bs, kv)
    info = pa.pa_plan_info()
    st = pa.load_library().pa_plan(None, ctypes.byref(c), 256, 10, 2, 4, None, ctypes.byref(info))
    assert st == status, pa.pa_last_error()
    if st != pa.PA_OK:
        assert pa.pa_last_error()


def test_workspace_bound_covers_every_plan():
    for Hq, Hkv, d in [(32, 8, 128), (8, 2, 64), (64, 8, 128), (16, 16, 128)]:
        c = cfg(Hq, Hkv, d)
        for S_max, MB_max in [(1, 1), (4, 16), (64, 513), (16, 8193), (128, 1025), (300, 40)]:
            bound = pa.pa_workspace_bytes(c, 10 * S_max, S_max, MB_max)
            for S, MB, cus, T in itertools.product(sorted({1, 2, 3, S_max // 2 or 1, S_max}),
                                                   sorted({1, MB_max // 3 or 1, MB_max}),
                                                   (1, 80, 256), (1, 2, 10)):
                p = plan(c, cus=cus, T=T * S, S=S, MB=MB)
                assert p["workspace_bytes"] <= bound, (Hq, Hkv, d, S, MB, cus, T)


def test_create_without_a_gpu_reports_a_device_error():
    if torch.cuda.is_available():
        pytest.skip("a GPU is visible")
    c = cfg()
    h = ctypes.c_void_p()
    st = pa.load_library().pa_create(ctypes.byref(c), ctypes.byref(h))
    assert st == pa.PA_ERR_DEVICE
    assert "hip" in pa.pa_last_error().lower()
