"""Offline tuning sweep of the decode partition's minimum share (segment
length = min_steps * step keys; arxiv 2511.11581 Sec. 4.5 segments, Sec. 5
offline tuning exported as decision rules).  Runs on one GPU:

    python -m paper_2511_11581_amd.tune [--out tune.json]

For each batch shape (decode rows only: S sequences of length L), every
candidate minimum share is timed (decode + merge kernels, from the
library's per-kernel events); the result lists the best share per shape and
a decision tree fitted to it over (total decode steps per worker, sequences)."""
import argparse
import json
import os
import sys

SHARES = (1, 2, 4, 8, 16, 32)
SHAPES = [(s, l) for s in (1, 4, 16, 64, 128) for l in (1024, 8192, 32768)]


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


def fit_tree(rows):
    from sklearn.tree import DecisionTreeClassifier, export_text
    X = [[r["steps_per_group"], r["seqs"]] for r in rows]
    y = [r["best_share"] for r in rows]
    tree = DecisionTreeClassifier(max_depth=2, random_state=0).fit(X, y)
    return export_text(tree, feature_names=["steps_per_group", "seqs"])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default="")
    args = ap.parse_args()
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
    res = {"shares": SHARES, "rows": rows, "tree": fit_tree(rows)}
    print(res["tree"])
    if args.out:
        json.dump(res, open(args.out, "w"), indent=1)


if __name__ == "__main__":
    sys.exit(main())
