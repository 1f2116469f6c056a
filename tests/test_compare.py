"""CPU self-tests of the teacher-forced comparator (tests/compare.py).

The comparator must accept the oracle's own tree, reject corrupted trees
(wrong token, parent, score, mask bit, frontier member, count), and accept a
different but valid choice at a planted near-tie while reporting that the
round was not compared exactly.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import pctree_oracle as O
from paper_2608_02123_amd.synth import Workload, make_inputs
import compare as C


def oracle_as_gpu(res, k, B, V):
    """Format an oracle result like the library's outputs (float32 scores + trace)."""
    kk = min(k, V)
    pool = res["pool"]
    g = {key: np.array(res[key]) for key in ("token", "parent", "depth", "position")}
    g["logprob"] = res["logprob"].astype(np.float32)
    g["count"] = res["count"]
    g["mask"] = res["mask"].copy()
    tt = np.full((B, k), -1, np.int32)
    tp = np.full((B, k), -1, np.int32)
    ts = np.full((B, k), -np.inf, np.float32)
    for d, st in enumerate(res["stages"]):
        prev = res["stages"][d - 1]["frontier"] if d else None
        for s, i in enumerate(st["frontier"]):
            n = pool[i]
            tt[d, s] = n.token
            ts[d, s] = n.score
            tp[d, s] = -1 if d == 0 else prev.index(n.parent)
    assert all(len(st["frontier"]) <= kk for st in res["stages"])
    g["trace_token"], g["trace_parent_slot"], g["trace_score"] = tt, tp, ts
    return g


def _setup(seed=0, V=400, B=4, N=20, k=4):
    w = Workload("c", V=V, B=B, N=N, k=k, r=32, dtype="f32", seed=seed)
    inp = make_inputs(w)
    L, E, W, h = inp["L"][0], inp["E"], inp["W"].astype(np.float64), inp["h"][0]
    xt, pl = int(inp["root"][0]), int(inp["prefix_len"][0])
    res = O.build_tree(L, E, W, h, xt, pl, k, N, "f32")
    return (L, E, W, h, xt, pl, k, N), res


def _run(args, g):
    L, E, W, h, xt, pl, k, N = args
    return C.compare_request(g, L, E, W, h, xt, pl, k, N, "f32")


def test_accepts_oracle_tree():
    args, res = _setup()
    g = oracle_as_gpu(res, args[6], args[0].shape[0], args[0].shape[1])
    rep = _run(args, g)
    assert rep["exact"] and rep["count"] == args[7]


def _corrupt(name, g):
    g = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in g.items()}
    if name == "token":
        g["token"][3] = (g["token"][3] + 1) % 400
    elif name == "parent":
        i = int(np.nonzero(g["depth"] == 2)[0][0])
        others = [q for q in np.nonzero(g["depth"] == 1)[0] if q != g["parent"][i]]
        g["parent"][i] = others[0] if others else 0
    elif name == "score":
        g["logprob"][5] -= 0.01
    elif name == "mask":
        g["mask"][6, 0] ^= np.uint32(1 << 2)
    elif name == "frontier":
        g["trace_token"][2, 1] = (g["trace_token"][2, 1] + 7) % 400
    elif name == "count":
        g["count"] -= 1
        g["token"][g["count"]] = -1
    elif name == "position":
        g["position"][4] += 1
    elif name == "swap_order":
        g["token"][[1, 2]] = g["token"][[2, 1]]
    return g


@pytest.mark.parametrize("name", ["token", "parent", "score", "mask", "frontier", "count",
                                  "position", "swap_order"])
def test_rejects_corruption(name):
    args, res = _setup()
    g = _corrupt(name, oracle_as_gpu(res, args[6], args[0].shape[0], args[0].shape[1]))
    with pytest.raises(AssertionError):
        _run(args, g)


def test_near_tie_accepts_either_choice():
    """Plant a tie between the root's 4th and 5th child; the other choice is valid."""
    args, _ = _setup(seed=1, V=50, B=2, N=40, k=4)
    L, E, W, h, xt, pl, k, N = args
    W = np.zeros_like(W)  # every row is log_softmax(L_d): easy to plant ties
    L = L.copy()
    order = np.argsort(-L[0], kind="stable")
    a, b = order[3], order[4]
    L[0, b] = L[0, a]  # exact tie at the boundary: the oracle keeps the lower id
    lo, hi = min(a, b), max(a, b)
    args = (L, E, W, h, xt, pl, k, N)
    ref = O.build_tree(L, E, W, h, xt, pl, k, N, "f32")
    g_ref = oracle_as_gpu(ref, k, 2, 50)
    rep = _run(args, g_ref)
    assert not rep["exact"] and rep["min_gap"] < C.TIE
    # the alternative: the higher id wins the tie (as if rounding went the other way)
    L2 = L.copy()
    L2[0, hi] += np.float32(2e-6)
    alt = O.build_tree(L2, E, W, h, xt, pl, k, N, "f32")
    assert hi in alt["token"] and lo not in alt["token"][alt["depth"] == 1]
    g_alt = oracle_as_gpu(alt, k, 2, 50)
    rep = _run(args, g_alt)
    assert not rep["exact"]
