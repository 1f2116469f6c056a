"""The stage-timeline build on the GPU: the tool runs a round through
libpctree_timeline.so in a process of its own, and the tree must be the
default library's bit for bit (the stamps only store the clock), with every
stage stamped and each workgroup's stamps in order."""
from __future__ import annotations

import json
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

from paper_2608_02123_amd import pctree as P
from paper_2608_02123_amd.synth import CONFIGS, Workload, make_inputs

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KEYS = ("token", "parent", "depth", "position", "logprob", "count", "mask",
        "trace_token", "trace_parent_slot", "trace_score")


def say(msg):
    print(msg, flush=True)


CASES = [
    ("qwen4b_b7", ["--workload", "qwen4b_b7"], CONFIGS["qwen4b_b7"]),
    ("wide", ["--shape", "700,3,30,5,32,9,bf16"],
     Workload("shape", V=700, B=3, N=30, k=5, r=32, R=9, dtype="bf16", peak="uniform", seed=1)),
]


@pytest.mark.parametrize("label,args,w", CASES, ids=[c[0] for c in CASES])
def test_timeline_build_keeps_the_tree(tmp_path, label, args, w):
    jf, tf = tmp_path / "timeline.json", tmp_path / "tree.npz"
    cmd = [sys.executable, "-u", "-m", "paper_2608_02123_amd.timeline", *args, "--rounds", "3",
           "--json", str(jf), "--save-tree", str(tf)]
    say(f"[timeline] {label}: {' '.join(cmd[2:])}")
    r = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True, timeout=240)
    say(r.stdout[-3000:])
    assert r.returncode == 0, r.stderr[-3000:]
    res = json.load(open(jf))
    got = np.load(tf)

    dev = P.device_inputs(make_inputs(w))
    b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, P.BF16 if w.dtype == "bf16" else P.F32,
                      mask=True, trace=True)
    out = b.run(**dev, check=True)
    torch.cuda.synchronize()
    for key in KEYS:
        assert np.array_equal(got[key], out[key].cpu().numpy()), f"{label}: {key} differs"

    stages = res["stages"]
    if res["form"] == "single launch":
        assert [s["stage"] for s in stages] == list(range(w.B))
        for s in stages:
            for key, v in s.items():
                assert v is not None and v >= 0.0, (label, s["stage"], key, v)
        assert res["stage_period_us"] > 0.0 and res["round_us"] > res["emission_us"] > 0.0
    else:
        assert len(stages) == w.B  # more than 16 frontier rows: every stage is wide
        for s in stages:
            for key in ("head_stream_us", "head_us", "head_to_merge_us", "merge_rows_us",
                        "merge_select_us"):
                assert s[key] is not None and s[key] >= 0.0, (label, s["stage"], key)
            assert s["head_us"] >= s["head_stream_us"]
    say(f"[timeline] {label}: tree identical, {len(stages)} stages stamped in order")
