"""Per-step kernel times of a decode run from a rocprofv3 kernel trace (measurement aid).

    python -m paper_2502_00085_amd.trace_steps <prefix>_kernel_trace.csv --prompt P --gc-interval g

Splits the dispatches that follow the n-th `k_init_prompt` (default: the 5th, which starts
the timed graph replay of bench.py) into decode steps at each attention launch, and reports
the decode pass (attention + top-b) against the garbage collection (the append kernel of a
collecting step plus the row copy launched before the next attention), overall and per
tenth of the run: the comparison of the paper's Figure 4 (Section 5.3).  A step collects
when the position after its new leaves, P + step, is a multiple of g (Alg 2).  In a run of
fused steps (the append inside the selection's merge kernel) the append has no launch of its
own: the merge kernel's time on collecting steps is compared with the other steps instead.
"""
from __future__ import annotations

import argparse
import csv

import numpy as np

KERNELS = ("k_init_prompt", "k_move_rows", "k_attn_mfma", "k_attn_valu", "k_attn_combine",
           "k_topb_chunk", "k_topb_final", "k_append_prune")


def kind(name: str):
    for k in KERNELS:
        if k in name:
            return k
    return None


def steps_of(path: str, run: int):
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"]))
    inits = [i for i, r in enumerate(rows) if kind(r["Kernel_Name"]) == "k_init_prompt"]
    end = inits[run + 1] if run + 1 < len(inits) else len(rows)
    steps, cur, move = [], None, 0.0
    for r in rows[inits[run] + 1:end]:
        k = kind(r["Kernel_Name"])
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        if k == "k_move_rows":
            move += us
        elif k in ("k_attn_mfma", "k_attn_valu"):
            cur = dict(attn=us, move=move, topb=0.0, append=0.0, fused=0.0)
            move = 0.0
            steps.append(cur)
        elif cur is None:
            continue
        elif k == "k_attn_combine":
            cur["attn"] += us
        elif k in ("k_topb_chunk", "k_topb_final"):
            cur["topb"] += us
            if k == "k_topb_final" and "true>" in r["Kernel_Name"]:
                cur["fused"] += us
        elif k == "k_append_prune":
            cur["append"] += us
    return steps


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("trace")
    ap.add_argument("--prompt", type=int, required=True)
    ap.add_argument("--gc-interval", type=int, default=1)
    ap.add_argument("--run", type=int, default=4, help="0-based index of the k_init_prompt that starts the run")
    a = ap.parse_args()
    st = steps_of(a.trace, a.run)
    K = len(st)
    att = np.array([s["attn"] for s in st])
    tb = np.array([s["topb"] for s in st])
    app = np.array([s["append"] for s in st])
    mv = np.array([s["move"] for s in st] + [0.0])
    dec = att + tb
    col = np.array([(a.prompt + i + 1) % a.gc_interval == 0 for i in range(K)])
    gc = np.array([app[i] + mv[i + 1] for i in range(K)])
    idx = np.nonzero(col)[0]
    print(f"steps {K}, collections {len(idx)}")
    print(f"decode pass (attention + top-b): {dec.mean():.2f} us (attention {att.mean():.2f}, top-b {tb.mean():.2f})")
    fz = np.array([s["fused"] for s in st])
    fused = bool(fz.any()) and not app.any()
    if fused and len(idx) and (~col).any():
        # the collection's share of a fused merge: its extra time on collecting steps
        extra = max(0.0, float(fz[col].mean() - fz[~col].mean()))
        gc = np.array([(extra if col[i] else 0.0) + mv[i + 1] for i in range(K)])
        print(f"fused selection + append kernel: {fz[col].mean():.2f} us on collecting steps, "
              f"{fz[~col].mean():.2f} us on the others")
    elif (~col).any():
        print(f"append kernel, no collection: {app[~col].mean():.2f} us")
    if len(idx):
        copies = [mv[i + 1] for i in idx if i + 1 < K]
        what = ("append + copy" if not fused else "the fused merge's extra time + copy" if (~col).any()
                else "the row copy only: every step collects, so the fused merge's share is not separable")
        if not fused:
            print(f"append kernel, collecting: {app[col].mean():.2f} us; row copy after it: {np.mean(copies):.2f} us")
        else:
            print(f"row copy after a collecting step: {np.mean(copies):.2f} us")
        print(f"collection ({what}): {gc[col].mean():.2f} us = {gc[col].mean() / dec.mean() * 100:.1f} % "
              f"of a decode pass; {gc[col].sum() / K / dec.mean() * 100:.2f} % per step")
    print("| steps | decode pass (µs) | collection (µs) |")
    print("|---|---|---|")
    for k in range(10):
        lo, hi = k * K // 10, (k + 1) * K // 10
        if hi <= lo:
            continue
        c = col[lo:hi]
        cg = f"{gc[lo:hi][c].mean():.1f}" if c.any() else "-"
        print(f"| {lo + 1}-{hi} | {dec[lo:hi].mean():.1f} | {cg} |")


if __name__ == "__main__":
    main()
