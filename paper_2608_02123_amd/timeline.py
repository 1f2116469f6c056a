"""Stage timeline of one round, from the library's timeline build.

``libpctree_timeline.so`` is the library with device wall-clock stamps at the
steps of every stage (include/pctree_profile.h lists them).  This tool runs a
few rounds of a synthetic workload through it, reads the stamps of the last
round and prints where the round's time goes: per stage, the keeper's merge
and selection and the first and last streaming workgroups' wait, head input,
stream and publish (single-launch round), or the wide stages' head and
merge-and-select launches (per-stage launches).

    python -m paper_2608_02123_amd.timeline [--workload qwen4b_b16]
        [--shape V,B,N,k,r,R,dtype] [--rounds 5] [--json OUT] [--save-tree OUT.npz]
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np

from . import pctree as P
from .synth import CONFIGS, Workload, make_inputs

KEEPER, FIRST, LAST, HEAD, MERGE = range(5)
ROUND = P.TIMELINE_STAGES - 1  # the keeper's round-level stamps


def run(w: Workload, rounds: int = 5):
    """Run `rounds` rounds of `w` through the timeline build; returns the last
    round's stamps (microseconds, [who][stage][event], NaN where not stamped)
    and its outputs."""
    if P._lib is not None and P.LIB_PATH != P.TIMELINE_LIB_PATH:
        raise RuntimeError("the default library is already loaded in this process")
    P.LIB_PATH = P.TIMELINE_LIB_PATH
    if not P.timeline_available():
        raise RuntimeError(f"{P.LIB_PATH} is not the timeline build")
    dev = P.device_inputs(make_inputs(w))
    b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, P.BF16 if w.dtype == "bf16" else P.F32,
                      mask=True, trace=True)
    b.bind(**dev)
    for _ in range(max(rounds - 1, 0)):
        b.launch()
    P.timeline_read()  # (waits for the rounds, then zeroes the stamps)
    out = b.launch(check=True)
    stamps = P.timeline_read()
    return stamps, {k: v.cpu().numpy() for k, v in out.items()}


def summarize(t: np.ndarray, B: int) -> dict:
    """Per-stage durations (microseconds) of one round's stamps."""
    res = {"stages": []}
    if not np.isnan(t[KEEPER, 0, 0]):  # single-launch round
        t0 = np.nanmin(t[FIRST, 0, :])
        for d in range(B):
            k, f, l = t[KEEPER, d], t[FIRST, d], t[LAST, d]
            res["stages"].append({
                "stage": d,
                "keeper_merge_us": k[1] - k[0],
                "keeper_select_us": k[2] - k[1],
                "first_inputs_us": f[1] - f[0],
                "first_stream_us": f[2] - f[1],
                "first_publish_us": f[3] - f[2],
                "last_inputs_us": l[1] - l[0],
                "last_stream_us": l[2] - l[1],
                "last_publish_us": l[3] - l[2],
                "selected_at_us": k[2] - t0,
            })
        sel = t[KEEPER, :B, 2]
        res["form"] = "single launch"
        res["stage_period_us"] = float(np.nanmean(np.diff(sel[1:]))) if B > 2 else float("nan")
        res["emission_us"] = float(t[KEEPER, ROUND, 1] - t[KEEPER, ROUND, 0])
        res["round_us"] = float(t[KEEPER, ROUND, 1] - t0)
    else:  # per-stage launches: the wide stages
        res["form"] = "per-stage launches"
        for d in range(B):
            h, m = t[HEAD, d], t[MERGE, d]
            if np.isnan(h[0]):
                continue
            res["stages"].append({
                "stage": d,
                "head_stream_us": h[1] - h[0],
                "head_us": h[2] - h[0],
                "head_to_merge_us": m[0] - h[2],
                "merge_rows_us": m[1] - m[0],
                "merge_select_us": m[2] - m[1],
                "stage_us": (t[HEAD, d + 1, 0] - h[0]) if d + 1 < B and not np.isnan(
                    t[HEAD, d + 1, 0]) else float("nan"),
            })
    for s in res["stages"]:
        for key, v in s.items():
            s[key] = None if isinstance(v, float) and np.isnan(v) else (
                round(float(v), 3) if key != "stage" else v)
    return res


def _table(res: dict) -> str:
    rows = res["stages"]
    if not rows:
        return "(no stage stamped)"
    keys = [k for k in rows[0] if k != "stage"]
    fmt = lambda v: "     -" if v is None else f"{v:6.2f}"  # noqa: E731
    lines = ["stage " + " ".join(k.replace("_us", "") for k in keys)]
    for s in rows:
        lines.append(f"{s['stage']:5d} " + " ".join(fmt(s[k]).rjust(len(k) - 3) for k in keys))
    return "\n".join(lines)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="qwen4b_b16", choices=sorted(CONFIGS))
    ap.add_argument("--shape", default=None,
                    help="V,B,N,k,r,R,dtype instead of a named workload (synthetic inputs)")
    ap.add_argument("--rounds", type=int, default=5)
    ap.add_argument("--json", default=None, help="write the per-stage summary here")
    ap.add_argument("--save-tree", default=None, help="write the last round's outputs (npz)")
    a = ap.parse_args(argv)
    if a.shape:
        V, B, N, k, r, R, dt = a.shape.split(",")
        w = Workload("shape", V=int(V), B=int(B), N=int(N), k=int(k), r=int(r), R=int(R),
                     dtype=dt, peak="uniform", seed=1)
    else:
        w = CONFIGS[a.workload]
    print(f"[timeline] {w.name}: V={w.V} B={w.B} N={w.N} k={w.k} r={w.r} R={w.R} {w.dtype}",
          flush=True)
    stamps, out = run(w, a.rounds)
    res = summarize(stamps, w.B)
    res["workload"] = w.name
    print(f"[timeline] {res['form']}", flush=True)
    print(_table(res), flush=True)
    for key in ("stage_period_us", "emission_us", "round_us"):
        if key in res:
            print(f"{key}: {res[key]:.2f}", flush=True)
    if a.json:
        with open(a.json, "w") as f:
            json.dump(res, f, indent=1)
    if a.save_tree:
        np.savez(a.save_tree, **out)
    return 0


if __name__ == "__main__":
    sys.exit(main())
