"""A round captured into a HIP graph and replayed.

Serving loops capture their per-step work into a graph and replay it; the
round's launches (a clear of the stage records, the single persistent launch
or the per-stage launches, the emission) must then give the tree of an
ordinary call on every replay.  A replay runs with the launch arguments of
the capture, the call's tag among them, so the test puts ordinary calls on
the same workspace between replays (each with a tag of its own) and checks
every replay bit for bit against the eager result.  The entry point that
allocates nothing is captured as well: it is meant for callers under
capture.
"""
from __future__ import annotations

import pytest
import torch

from paper_2608_02123_amd import pctree as P
from paper_2608_02123_amd.synth import CONFIGS, Workload, make_inputs
import compare as C

pytestmark = pytest.mark.gpu

KEYS = ("token", "parent", "depth", "position", "logprob", "count", "mask",
        "trace_token", "trace_parent_slot", "trace_score")

# (label, workload): the persistent form (R k' <= 16) and the per-stage form
# with wide stages (R k' > 16)
CASES = [
    ("tiny", CONFIGS["tiny"]),
    ("persistent-bf16", Workload("gp", V=9000, B=5, N=40, k=8, r=64, dtype="bf16",
                                peak="uniform", seed=11)),
    ("wide-bf16", Workload("gw", V=700, B=3, N=30, k=5, r=32, R=9, dtype="bf16",
                          peak="uniform", seed=12)),
]


def say(msg):
    print(msg, flush=True)


def _snapshot(out):
    return {k: v.clone() for k, v in out.items() if k in KEYS}


def _replay_and_check(label, g, b, launch_eager, ref):
    for rep in range(3):
        launch_eager()  # an ordinary call on the same workspace, its own tag
        for key in KEYS:
            b.out[key].fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for key in KEYS:
            assert torch.equal(b.out[key], ref[key]), f"{label} replay {rep}: {key} differs"
        say(f"[graph] {label}: replay {rep} identical to the eager call")


@pytest.mark.parametrize("label,w", CASES, ids=[c[0] for c in CASES])
def test_captured_round_replays_the_eager_tree(label, w):
    dt = P.BF16 if w.dtype == "bf16" else P.F32
    say(f"[graph] {label}: V={w.V} B={w.B} N={w.N} k={w.k} r={w.r} R={w.R} {w.dtype}")
    inp = make_inputs(w)
    dev = P.device_inputs(inp)
    b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, dt, mask=True, trace=True)
    ref = _snapshot(b.run(**dev, check=True))
    torch.cuda.synchronize()
    reps = C.compare_batch(ref, inp, w.k, w.N, label=f"graph {label}")
    assert all(r["exact"] for r in reps), f"{label}: eager tree not exact against the oracle"

    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b.launch()  # (first use on the capture stream outside the capture)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        b.launch()
    torch.cuda.synchronize()
    _replay_and_check(label, g, b, lambda: b.launch(), ref)


@pytest.mark.parametrize("label,w", CASES[1:], ids=[c[0] for c in CASES[1:]])
def test_captured_noalloc_round_replays_the_eager_tree(label, w):
    dt = P.BF16 if w.dtype == "bf16" else P.F32
    say(f"[graph] noalloc {label}")
    dev = P.device_inputs(make_inputs(w))
    ref_b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, dt, mask=True, trace=True)
    ref = _snapshot(ref_b.run(**dev, check=True))
    b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, dt, mask=True, trace=True, workspace=False)
    b.run_noalloc(**dev, check=True)  # the device's scratch address is looked up here
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        b.run_noalloc(**dev)
    torch.cuda.synchronize()
    _replay_and_check(f"noalloc {label}", g, b, lambda: b.run_noalloc(**dev), ref)
