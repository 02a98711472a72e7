"""Offline tuning sweeps of the launcher's choices, exported as decision
rules (arxiv 2511.11581 Sec. 5 offline tuning, Lst. 2 decision trees;
Sec. 7 / Fig. 8 the tuned tree on prefill-heavy shapes).  Runs on one GPU:

    python -m paper_2511_11581_amd.tune [--out tune.json] [--only decode|qblock]

decode: the decode partition's minimum share (segment length = min_steps *
step keys, Sec. 4.5).  For each decode-only batch shape (S sequences of
length L) every candidate share is timed (decode + merge kernels, from the
library's per-kernel events); a depth-2 tree over (total decode steps per
worker group, sequences) is fitted to the best share.

qblock: the Q-block shape for bf16 caches, BLOCK_M = 256 rows (8 waves, one
workgroup per CU) or 128 rows (4 waves, two per CU), on prefill-heavy
batches (S sequences of q new tokens after ctx cached ones; short prompts,
small chunks, many sequences); every call of pa_forward is timed with HIP
events, and a depth-2 tree over host-visible features (grid waves of the
256-row grid over the CUs, query tokens per sequence) is fitted to the
best BLOCK_M."""
import argparse
import json
import os
import sys

SHARES = (1, 2, 4, 8, 16, 32)
SHAPES = [(s, l) for s in (1, 4, 16, 64, 128) for l in (1024, 8192, 32768)]
ROWS = (256, 128)
# (sequences, query tokens, context, query heads, kv heads)
QB_SHAPES = ([(s, q, c, 32, 8) for s in (1, 4, 16, 64) for q in (16, 64, 256, 1024, 4096)
              for c in (0, 4096) if s * q <= 65536]
             + [(s, q, 0, 64, 8) for s in (1, 8, 32) for q in (32, 256, 2048)])


def time_shape(S, L, share, steps=20, warmup=3):
    import torch
    from paper_2511_11581_amd import pa, workloads as W
    os.environ["PA_DECODE_MIN_STEPS"] = str(share)   # read when the handle is created
    w = W.make_batch([(L - 1, 1)] * S, 32, 8, 128, seed=S * 7 + L, name=f"tune{S}x{L}",
                     device="cuda", poison=False)
    att = pa.PagedAttention(32, 8, 128, 16, max_tokens=w.num_tokens, max_seqs=S,
                            max_blocks_per_seq=int(w.block_table.shape[1]), profile=True)
    out = torch.empty_like(w.q)
    for _ in range(warmup):
        att.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc,
                    w.scale, out=out)
    torch.cuda.synchronize()
    att.profile(reset=True)
    for _ in range(steps):
        att.forward(w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc,
                    w.scale, out=out)
    torch.cuda.synchronize()
    prof = att.profile(reset=True)
    plan = att.plan(w.num_tokens, S, int(w.block_table.shape[1]))
    us = (prof["decode"][1] + prof["merge"][1]) * 1e3 / steps   # (launches, total ms)
    total_steps = S * 8 // plan["decode_unit_heads"] * -(-L // plan["decode_step"])
    del w, att, out
    torch.cuda.empty_cache()
    return us, total_steps, plan["decode_workers"] // plan["decode_unit_heads"]


def time_qblock(S, q, ctx, Hq, Hkv, rows, steps=30, warmup=5):
    import torch
    from paper_2511_11581_amd import pa, workloads as W
    os.environ["PA_QBLOCK_ROWS"] = str(rows)   # read when the handle is created
    w = W.make_batch([(ctx, q)] * S, Hq, Hkv, 128, seed=S * 131 + q + ctx, name="tuneqb",
                     device="cuda", poison=False)
    att = pa.PagedAttention(Hq, Hkv, 128, 16, max_tokens=w.num_tokens, max_seqs=S,
                            max_blocks_per_seq=int(w.block_table.shape[1]))
    del os.environ["PA_QBLOCK_ROWS"]
    out = torch.empty_like(w.q)
    args = (w.q, w.k_cache, w.v_cache, w.block_table, w.seq_lens, w.query_start_loc, w.scale)
    for _ in range(warmup):
        att.forward(*args, out=out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        att.forward(*args, out=out)
    e1.record()
    torch.cuda.synchronize()
    plan = att.plan(w.num_tokens, S, int(w.block_table.shape[1]))
    us = e0.elapsed_time(e1) * 1e3 / steps
    del w, att, out
    torch.cuda.empty_cache()
    return us, plan


def qblock_features(S, T, Hq, Hkv, cus=256):
    """Host-visible features of the BLOCK_M rule (the same formula make_plan
    evaluates): waves of the 256-row grid over the CUs, tokens per sequence."""
    G = Hq // Hkv
    bq = 256 // G
    units = (-(-T // bq) + min(S, T // 2)) * Hkv
    return [units / cus, T / max(S, 1)]


def fit_tree(rows):
    from sklearn.tree import DecisionTreeClassifier, export_text
    X = [[r["steps_per_group"], r["seqs"]] for r in rows]
    y = [r["best_share"] for r in rows]
    tree = DecisionTreeClassifier(max_depth=2, random_state=0).fit(X, y)
    return export_text(tree, feature_names=["steps_per_group", "seqs"])


def fit_qblock_tree(rows):
    from sklearn.tree import DecisionTreeClassifier, export_text
    X = [r["features"] for r in rows]
    y = [r["best_rows"] for r in rows]
    tree = DecisionTreeClassifier(max_depth=2, random_state=0).fit(X, y)
    return export_text(tree, feature_names=["grid_waves_256", "tokens_per_seq"])


def sweep_qblock():
    rows = []
    for S, q, c, Hq, Hkv in QB_SHAPES:
        t = {}
        for r in ROWS:
            us, plan = time_qblock(S, q, c, Hq, Hkv, r)
            t[r] = us
        best = min(t, key=t.get)
        rows.append({"seqs": S, "q": q, "ctx": c, "heads": [Hq, Hkv], "us": t, "best_rows": best,
                     "features": qblock_features(S, S * q, Hq, Hkv),
                     "gain_vs_256": t[256] / t[best]})
        print(json.dumps(rows[-1]), flush=True)
    return {"rows_options": ROWS, "rows": rows, "tree": fit_qblock_tree(rows)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default="")
    ap.add_argument("--only", default="", choices=["", "decode", "qblock"])
    args = ap.parse_args()
    res = {}
    if args.only in ("", "qblock"):
        res["qblock"] = sweep_qblock()
        print(res["qblock"]["tree"], flush=True)
    if args.only == "qblock":
        if args.out:
            json.dump(res, open(args.out, "w"), indent=1)
        return 0
    rows = []
    for S, L in SHAPES:
        t = {}
        for share in SHARES:
            us, total, groups = time_shape(S, L, share)
            t[share] = us
        best = min(t, key=t.get)
        rows.append({"seqs": S, "len": L, "total_steps": total, "groups": groups,
                     "steps_per_group": total / groups, "us": t, "best_share": best,
                     "gain_vs_1": t[1] / t[best]})
        print(json.dumps(rows[-1]), flush=True)
    res["decode"] = {"shares": SHARES, "rows": rows, "tree": fit_tree(rows)}
    print(res["decode"]["tree"])
    if args.out:
        json.dump(res, open(args.out, "w"), indent=1)


if __name__ == "__main__":
    sys.exit(main())
