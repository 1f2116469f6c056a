"""GPU parity of the two control scorings of Sec. 5.3 and Sec. 4 against the
CPU oracle, through the C ABI: the Shared-Markov tree (the greedy chain's row
at each depth serves every parent) and parent-independent per-position
scoring (every parent of depth d gets log_softmax(L_d)).  Same comparator and
tolerances as the parent-conditioned parity tests."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import pctree_oracle as O
from paper_2608_02123_amd import pctree as P
from paper_2608_02123_amd.synth import CONFIGS, Workload, make_inputs
import compare as C

pytestmark = pytest.mark.gpu

MODES = {"shared": P.MODE_SHARED, "independent": P.MODE_INDEPENDENT}


def say(msg):
    print(msg, flush=True)


def run(inp, k, N, mode):
    w = inp["workload"]
    dev = P.device_inputs(inp)
    b = P.TreeBuilder(w.V, w.B, N, k, w.r, w.R, P.BF16 if w.dtype == "bf16" else P.F32,
                      trace=True, mode=MODES[mode])
    out = b.run(**dev)
    torch.cuda.synchronize()
    return {key: v.clone() for key, v in out.items()}


SHAPES = [
    # V, B, N, k, r, R, dtype
    (1024, 4, 16, 4, 32, 1, "f32"),
    (5, 3, 40, 8, 16, 2, "f32"),       # k > V, pool smaller than N
    (4099, 4, 64, 8, 64, 2, "bf16"),   # ragged tail
    (1000, 3, 40, 16, 32, 3, "bf16"),  # max k, three requests
    (3000, 6, 33, 1, 96, 4, "bf16"),   # k = 1: the chain itself
    (300, 63, 256, 2, 32, 1, "bf16"),  # max depth and budget
    (700, 3, 30, 5, 32, 20, "bf16"),   # 20 requests: every stage runs the wide form
]


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "V{}B{}N{}k{}r{}R{}{}".format(*s))
def test_mode_shape_parity(mode, shape):
    V, B, N, k, r, R, dt = shape
    say(f"[modes] {mode} {shape}")
    w = Workload("m", V=V, B=B, N=N, k=k, r=r, R=R, dtype=dt, peak="uniform", seed=5)
    inp = make_inputs(w)
    reps = C.compare_batch(run(inp, k, N, mode), inp, k, N, mode=mode)
    say(f"[modes] {mode} {shape}: {reps}")


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("name", ["qwen4b_b7", "qwen4b_b16"])
def test_mode_workload_parity(mode, name):
    w = CONFIGS[name]
    say(f"[modes] {mode} {name}")
    inp = make_inputs(w)
    reps = C.compare_batch(run(inp, w.k, w.N, mode), inp, w.k, w.N, mode=mode)
    say(f"[modes] {mode} {name}: {reps}")


_CACHE = {}


@pytest.mark.parametrize("req", range(CONFIGS["qwen14b_b16_r8"].R))
def test_shared_batched_serving(req):
    """Eight requests, k = 16, N = 128, r = 512, Shared-Markov scoring: one
    GPU call, every request replayed against the oracle."""
    w = CONFIGS["qwen14b_b16_r8"]
    if "shared" not in _CACHE:
        say(f"[modes] shared {w.name}")
        inp = make_inputs(w)
        _CACHE["shared"] = (inp, run(inp, w.k, w.N, "shared"))
    inp, out = _CACHE["shared"]
    reps = C.compare_batch(out, inp, w.k, w.N, requests=[req], mode="shared")
    say(f"[modes] shared {w.name} request {req}: {reps}")


@pytest.mark.parametrize("req", range(CONFIGS["qwen14b_b16_r8"].R))
def test_independent_batched_serving(req):
    """Eight requests, k = 16, N = 128, r = 512, parent-independent scoring
    (every stage in the wide form with one row per request): one GPU call,
    every request replayed against the oracle."""
    w = CONFIGS["qwen14b_b16_r8"]
    if "independent" not in _CACHE:
        say(f"[modes] independent {w.name}")
        inp = _CACHE["shared"][0] if "shared" in _CACHE else make_inputs(w)
        _CACHE["independent"] = (inp, run(inp, w.k, w.N, "independent"))
    inp, out = _CACHE["independent"]
    reps = C.compare_batch(out, inp, w.k, w.N, requests=[req], mode="independent")
    say(f"[modes] independent {w.name} request {req}: {reps}")


def test_modes_differ_under_conditioning():
    """sigma_E = 1: the three scorings give three different trees, and the
    GPU's tree of each control mode passes the comparator for that mode."""
    w = Workload("sc", V=4099, B=5, N=48, k=8, r=64, dtype="bf16", sigma_E=1.0, seed=2)
    say("[modes] conditioning")
    inp = make_inputs(w)
    toks = []
    for mode in ("shared", "independent"):
        out = run(inp, w.k, w.N, mode)
        C.compare_batch(out, inp, w.k, w.N, mode=mode)
        toks.append(out["token"][0].cpu().numpy())
    ref = O.build_tree_batch(inp, w.k, w.N)[0]["token"]
    assert not np.array_equal(toks[0], ref) and not np.array_equal(toks[1], ref)
    assert not np.array_equal(toks[0], toks[1])


@pytest.mark.parametrize("mode", list(MODES))
def test_chain_modes(mode):
    w = Workload("c", V=5000, B=9, N=1, k=1, r=64, R=3, dtype="bf16", peak="uniform", seed=4)
    say(f"[modes] chain {mode}")
    inp = make_inputs(w)
    d = P.device_inputs(inp)
    toks, lps = P.chain_decode(d["L"], d["E"], d["Wt"], d["h"], d["root"], mode=MODES[mode])
    torch.cuda.synchronize()
    W64 = inp["W"].astype(np.float64)
    for i in range(w.R):
        t, c = O.chain_decode(inp["L"][i], inp["E"], W64, inp["h"][i], int(inp["root"][i]),
                              w.dtype, mode=mode)
        assert np.array_equal(toks[i].cpu().numpy(), t), i
        assert np.abs(lps[i].cpu().numpy() - c).max() <= C.SCORE_TOL, i
