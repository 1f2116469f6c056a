"""GPU tests of properties that must hold however a round is launched.

* The tree does not depend on how the vocabulary is sliced over workgroups
  (Alg. 1 defines it on whole rows): the single-launch round with the
  default slicing, with fewer slices, and the per-stage launches (another
  slicing and other kernels) must emit the same tree, and each must match
  the oracle.
* An abandoned single-launch round (its bounded waits give up) must leave
  count = -1 and padding in every output row, not the previous call's tree,
  and the next round must be whole again.  The test shortens the wait bound
  from the host (pctree_debug_set), so every workgroup still leaves through
  its own bounded wait: nothing hangs or faults.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2608_02123_amd import pctree as P
from paper_2608_02123_amd.synth import CONFIGS, make_inputs
import compare as C

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)


def _builder(w, **kw):
    return P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, P.BF16 if w.dtype == "bf16" else P.F32,
                         mask=True, trace=True, **kw)


def _run(b, dev, **launch):
    """One round with the given launch overrides (restored afterwards)."""
    P.debug_set(**launch)
    try:
        out = b.run(**dev)
        torch.cuda.synchronize()
    finally:
        P.debug_set()
    return {k: v.clone() for k, v in out.items()}


TREE_KEYS = ("token", "parent", "depth", "position", "count", "mask")


@pytest.mark.parametrize("name", ["tiny", "qwen4b_b7", "qwen4b_b16"])
def test_tree_independent_of_vocab_slicing(name):
    w = CONFIGS[name]
    inp = make_inputs(w)
    dev = P.device_inputs(inp)
    b = _builder(w)
    variants = {
        "single launch, one slice per CU": {},
        "single launch, at most 37 slices": {"round_slices": 37},
        "per-stage launches": {"force_multilaunch": True},
    }
    outs = {}
    for label, launch in variants.items():
        say(f"[launch] {name}: {label}")
        outs[label] = _run(b, dev, **launch)
        reps = C.compare_batch(outs[label], inp, w.k, w.N, label=f"{name}/{label}")
        assert all(r["exact"] for r in reps), f"{label}: tree not exact against the oracle"
    ref = outs["single launch, one slice per CU"]
    for label, out in outs.items():
        for key in TREE_KEYS:
            assert torch.equal(out[key], ref[key]), f"{label}: {key} differs"
        # scores: the same values up to the fp32 order of the slice merges
        np.testing.assert_allclose(out["logprob"].cpu().numpy(), ref["logprob"].cpu().numpy(),
                                   atol=C.SCORE_GUARD)


@pytest.mark.parametrize("mode", ["shared", "independent"])
def test_control_modes_independent_of_launch_form(mode):
    """The control scorings run in the single-launch round too (one shared
    row per request and stage): it must emit the tree of the per-stage
    launches, and both must match the oracle."""
    w = CONFIGS["qwen4b_b7"]
    inp = make_inputs(w)
    dev = P.device_inputs(inp)
    m = {"shared": P.MODE_SHARED, "independent": P.MODE_INDEPENDENT}[mode]
    b = _builder(w, mode=m)
    outs = {}
    for label, launch in {"single launch": {}, "per-stage launches": {"force_multilaunch": True}}.items():
        say(f"[launch] {mode}: {label}")
        outs[label] = _run(b, dev, **launch)
        reps = C.compare_batch(outs[label], inp, w.k, w.N, mode=mode, label=f"{mode}/{label}")
        # (parent-independent scores tie exactly: a + b = b + a across parents)
        assert all(r["exact"] or r["identical"] for r in reps), f"{label}: tree differs from the oracle"
    for key in TREE_KEYS:
        assert torch.equal(outs["single launch"][key], outs["per-stage launches"][key]), key
    np.testing.assert_allclose(outs["single launch"]["logprob"].cpu().numpy(),
                               outs["per-stage launches"]["logprob"].cpu().numpy(),
                               atol=C.SCORE_GUARD)


def test_abandoned_round_pads_every_output_then_recovers():
    w = CONFIGS["qwen4b_b7"]  # R * k' = 8 rows: the single-launch round
    inp = make_inputs(w)
    dev = P.device_inputs(inp)
    b = _builder(w)
    say("[launch] whole round")
    good = _run(b, dev)
    assert int(good["count"][0]) == w.N
    say("[launch] round whose waits give up at once")
    bad = _run(b, dev, wait_ticks=0)
    assert (bad["count"] == -1).all(), f"count {bad['count'].tolist()} (the round was not abandoned)"
    for key in ("token", "parent", "depth", "position"):
        assert (bad[key] == -1).all(), f"{key} is not padding after an abandoned round"
    assert torch.isneginf(bad["logprob"]).all(), "logprob is not -inf padding"
    assert (bad["mask"] == 0).all(), "mask words left after an abandoned round"
    with pytest.raises(P.RoundAborted):
        P.check_counts(bad["count"])
    say("[launch] next round with the default wait bound")
    again = _run(b, dev)
    P.check_counts(again["count"])
    for key in TREE_KEYS + ("logprob",):
        assert torch.equal(again[key], good[key]), f"{key} differs after the abandoned round"
    reps = C.compare_batch(again, inp, w.k, w.N, label="qwen4b_b7/after abort")
    assert reps[0]["exact"]


WIDE = [
    # V, B, N, k, r, R, dtype: more than 16 frontier rows per stage
    (2000, 3, 48, 16, 64, 2, "bf16"),
    (3000, 4, 40, 8, 128, 5, "f32"),
    (700, 3, 30, 5, 32, 9, "bf16"),
    (9000, 3, 64, 16, 512, 3, "bf16"),
]


@pytest.mark.parametrize("shape", WIDE, ids=lambda s: "V{}B{}N{}k{}r{}R{}{}".format(*s))
def test_wide_stages_without_row_bounds(shape):
    """Wide stages with their per-row bounds switched off: every logit is a
    candidate, every (row, slice) overflows its candidate slots and takes the
    exact per-slice path.  The tree must equal the bounded run's and the
    oracle's."""
    from paper_2608_02123_amd.synth import Workload

    V, B, N, k, r, R, dt = shape
    w = Workload("wu", V=V, B=B, N=N, k=k, r=r, R=R, dtype=dt, peak="uniform", seed=9)
    inp = make_inputs(w)
    dev = P.device_inputs(inp)
    b = _builder(w)
    say(f"[launch] wide {shape}: bounded")
    ref = _run(b, dev)
    say(f"[launch] wide {shape}: unbounded (exact path everywhere)")
    out = _run(b, dev, wide_unbounded=True)
    reps = C.compare_batch(out, inp, k, N, label=f"wide unbounded {shape}")
    for key in TREE_KEYS:
        assert torch.equal(out[key], ref[key]), f"{key} differs between bounded and unbounded"
    np.testing.assert_allclose(out["logprob"].cpu().numpy(), ref["logprob"].cpu().numpy(),
                               atol=C.SCORE_GUARD)
    assert all(r_["exact"] or r_["identical"] for r_ in reps)
