"""Stage-by-stage, teacher-forced comparison of a GPU round with the CPU oracle.

PCTree makes discrete choices (per-parent top-k, the frontier, the global
top-N) from floating-point scores, so two correct implementations can differ
where two candidates are closer than rounding.  The comparison therefore:

1. checks the GPU tree's structure exactly, as functions of its own parent
   array: root, canonical order, depths, positions (App. A) and the ancestor
   mask, bit for bit;
2. replays the GPU's frontier, stage by stage, through the oracle's rows
   (Eq. 2/3) and checks that every GPU choice is a valid selection under the
   oracle's float64 scores, where candidates closer than TIE count as tied;
   every GPU score must lie within SCORE_TOL of the oracle's score of the same
   path (Eq. 4);
3. when no selection boundary that can affect the emitted tree is closer than
   TIE, requires the GPU tree to equal the free-running oracle's tree exactly
   (token, parent, depth, position, mask) with log-probabilities within
   SCORE_TOL;
4. fails when any GPU score deviates from the oracle's by more than
   SCORE_GUARD: past it, two candidates more than TIE apart under the oracle
   could swap order on the GPU, and excluding ties closer than TIE would no
   longer make the exact comparison sound.

Every comparison appends a report row (label, request, exact, min_gap,
max_dev, count) to REPORTS; tests/conftest.py prints them at the end of the
session and writes them to a JSON file.
"""
from __future__ import annotations

import numpy as np

from oracle import pctree_oracle as O

TIE = 1e-4
SCORE_TOL = 1e-3
SCORE_GUARD = 5e-5

REPORTS: list = []  # one dict per compared request, in order


class Rows:
    """Oracle rows log pi_d(.|tok) of one request, cached by (depth, parent token)."""

    def __init__(self, L, E, W64, h, dtype):
        self.L, self.E, self.W, self.h, self.dtype = L, E, W64, h, dtype
        self.cache = {}

    def __call__(self, d, tok):
        key = (d, int(tok))
        if key not in self.cache:
            _, _, lp = O.child_logprobs(self.L[d], self.E, self.W, self.h[d], int(tok), self.dtype)
            self.cache[key] = lp
        return self.cache[key]


class ModeRows:
    """Oracle rows of the two control modes: one row per depth serves every
    parent (the Shared-Markov chain's rows, or log_softmax(L_d))."""

    def __init__(self, L, E, W64, h, x_t, dtype, mode):
        if mode == "shared":
            self.rows = O.shared_markov_rows(L, E, W64, h, int(x_t), dtype)
        elif mode == "independent":
            self.rows = [O.position_rows(L[d]) for d in range(L.shape[0])]
        else:
            raise ValueError(mode)

    def __call__(self, d, tok):
        return self.rows[d]


def _np(x):
    return x.detach().cpu().numpy() if hasattr(x, "detach") else np.asarray(x)


def check_structure(g, x_t, prefix, N, expect_count):
    """Exact checks of the emitted arrays as functions of the GPU's parent[]."""
    tok, par, dep, pos, lp, cnt = (g["token"], g["parent"], g["depth"], g["position"],
                                   g["logprob"], int(g["count"]))
    assert cnt == expect_count, f"count {cnt} != {expect_count}"
    if cnt:
        assert tok[0] == x_t and par[0] == -1 and dep[0] == 0 and lp[0] == 0.0, "root row"
    for i in range(1, cnt):
        assert 0 <= par[i] < i, f"parent[{i}]={par[i]}"
        assert dep[i] == dep[par[i]] + 1, f"depth[{i}]"
        assert (dep[i - 1], par[i - 1], tok[i - 1]) < (dep[i], par[i], tok[i]) or i == 1, \
            f"canonical order broken at {i}"
        assert lp[i] <= lp[par[i]], f"score increases along the edge into {i}"
    for i in range(cnt):
        assert pos[i] == prefix + dep[i], f"position[{i}]"
    assert (tok[cnt:] == -1).all() and (par[cnt:] == -1).all() and (dep[cnt:] == -1).all()
    assert (pos[cnt:] == -1).all() and np.isneginf(lp[cnt:]).all(), "padding rows"
    if "mask" in g:
        want = O.ancestor_mask(par, cnt, N)
        got = g["mask"].astype(np.uint32)
        assert np.array_equal(got, want), "ancestor mask differs"


def compare_request(g, L, E, W64, h, x_t, prefix, k, N, dtype, rows=None, oracle=None):
    """Compare one request.  ``g`` holds numpy arrays of the GPU outputs
    (token, parent, depth, position, logprob, count, mask, trace_*).

    Returns a report dict; raises AssertionError on a mismatch.
    """
    B, V = L.shape
    kk = min(k, V)
    pool_size = 1 + kk + (B - 1) * kk * kk
    rows = rows or Rows(L, E, W64, h, dtype)
    check_structure(g, x_t, prefix, N, min(N, pool_size))

    # --- 2. teacher-forced replay of the GPU frontiers -------------------
    tt, tp, ts = g["trace_token"], g["trace_parent_slot"], g["trace_score"]
    # frontier entering stage d: list of (path, oracle score, gpu score)
    front = [((int(x_t),), 0.0, float(ts[0, 0]))]
    assert tt[0, 0] == x_t and tp[0, 0] == -1, "stage-0 frontier must be the root"
    pool = {(int(x_t),): 0.0}  # path -> oracle score
    accept = {}  # path -> True if an acceptable child of a GPU frontier parent
    max_dev = 0.0
    margins = []  # (gap, score at the boundary, kind)
    for d in range(B):
        cands = []
        for j, (path, so, sg) in enumerate(front):
            max_dev = max(max_dev, abs(so - sg))
            assert abs(so - sg) <= SCORE_TOL, f"stage {d} slot {j}: score {sg} vs oracle {so}"
            lp = rows(d, path[-1])
            order = np.argsort(-lp, kind="stable")
            kth = lp[order[kk - 1]]
            if V > kk:
                margins.append((kth - lp[order[kk]], so + kth, "child"))
            for v in order[:kk]:
                cands.append((path + (int(v),), so + float(lp[v])))
            # children within TIE of the k'-th are acceptable alternatives
            for v in np.nonzero(lp >= kth - TIE)[0]:
                accept[path + (int(v),)] = so + float(lp[v])
        for p_, s_ in cands:
            pool[p_] = s_
        if d + 1 < B:
            cs = sorted((s for _, s in cands), reverse=True)
            cut = cs[kk - 1]
            if len(cs) > kk:
                margins.append((cut - cs[kk], cut, "frontier"))
            nxt = []
            for s in range(kk):
                ps, tk, sc = int(tp[d + 1, s]), int(tt[d + 1, s]), float(ts[d + 1, s])
                assert 0 <= ps < len(front), f"stage {d + 1} slot {s}: parent slot {ps}"
                path = front[ps][0] + (tk,)
                assert path in accept, f"stage {d + 1} slot {s}: {path} is not a top-k child"
                so = accept[path]
                assert so >= cut - TIE, f"stage {d + 1}: frontier member {so} below cut {cut}"
                nxt.append((path, so, sc))
            paths = {p for p, _, _ in nxt}
            assert len(paths) == kk, "duplicate frontier members"
            lo = min(s for _, s, _ in nxt)
            for p_, s_ in cands:
                if p_ not in paths:
                    assert s_ <= lo + TIE, f"stage {d + 1}: rejected candidate {s_} > {lo}"
            front = nxt
            assert (tt[d + 1, kk:] == -1).all() if tt.shape[1] > kk else True

    # --- global top-N -------------------------------------------------------
    cnt = int(g["count"])
    tok, par, lpg = g["token"], g["parent"], g["logprob"]
    paths = []
    for i in range(cnt):
        p_ = (int(tok[i]),) if i == 0 else paths[par[i]] + (int(tok[i]),)
        paths.append(p_)
    sel = {}
    for i, p_ in enumerate(paths):
        so = pool.get(p_, accept.get(p_))
        assert so is not None, f"node {i} {p_} was never generated"
        max_dev = max(max_dev, abs(so - float(lpg[i])))
        assert abs(so - float(lpg[i])) <= SCORE_TOL, f"node {i}: {lpg[i]} vs oracle {so}"
        sel[p_] = so
    allscores = sorted(pool.values(), reverse=True)
    if cnt < len(pool):
        gcut = allscores[cnt - 1]
        margins.append((gcut - allscores[cnt], gcut, "global"))
        lo = min(sel.values())
        assert lo >= gcut - TIE, f"selected node {lo} below the N-th score {gcut}"
        for p_, s_ in pool.items():
            if p_ not in sel:
                assert s_ <= lo + TIE, f"unselected node {p_} ({s_}) beats selected {lo}"

    assert max_dev <= SCORE_GUARD, (
        f"max |score deviation| {max_dev:.3g} exceeds {SCORE_GUARD}: the {TIE} tie exclusion "
        "is not sound at this deviation")

    # --- 3. exact equality when no relevant boundary is a near-tie ------------
    gcut = allscores[min(cnt, len(allscores)) - 1]
    relevant = [m for m in margins if m[2] == "global" or m[1] >= gcut - TIE]
    min_gap = min((m[0] for m in relevant), default=np.inf)
    exact = min_gap >= TIE
    ref = oracle if oracle is not None else O.build_tree(L, E, W64, h, x_t, prefix, k, N, dtype)
    same = all(np.array_equal(g[key], ref[key]) for key in ("token", "parent", "depth", "position"))
    if exact:
        for key in ("token", "parent", "depth", "position"):
            assert np.array_equal(g[key], ref[key]), f"{key} differs from the oracle"
        if "mask" in g:
            assert np.array_equal(g["mask"].astype(np.uint32), ref["mask"]), "mask differs"
        c = ref["count"]
        assert np.abs(g["logprob"][:c] - ref["logprob"][:c]).max(initial=0) <= SCORE_TOL
    # exact: the tree had to equal the oracle's and does; identical: it does
    # (also where a near tie let it differ)
    return {"exact": bool(exact), "identical": bool(same), "min_gap": float(min_gap),
            "max_dev": float(max_dev), "count": int(cnt)}


def gpu_to_numpy(out, req):
    g = {k: _np(v[req]) for k, v in out.items()}
    g["count"] = int(g["count"])
    if "mask" in g:
        g["mask"] = g["mask"].view(np.uint32)
    return g


def compare_batch(out, inp, k, N, requests=None, mode="parent", label=None):
    """Compare every request (or the listed ones) of a GPU batch output.

    Each request's report is also appended to REPORTS under ``label`` (the
    workload's name, the mode and k / N by default)."""
    w = inp["workload"]
    if label is None:
        label = f"{w.name}/{mode}/k{k}/N{N}"
    W64 = inp["W"].astype(np.float64)
    reports = []
    for req in (range(inp["L"].shape[0]) if requests is None else requests):
        g = gpu_to_numpy(out, req)
        L, h, x_t, pl = inp["L"][req], inp["h"][req], int(inp["root"][req]), \
            int(inp["prefix_len"][req])
        rows = oracle = None
        if mode != "parent":
            rows = ModeRows(L, inp["E"], W64, h, x_t, w.dtype, mode)
            oracle = O.build_tree(L, inp["E"], W64, h, x_t, pl, k, N, w.dtype, mode=mode)
        rep = compare_request(g, L, inp["E"], W64, h, x_t, pl, k, N, w.dtype,
                              rows=rows, oracle=oracle)
        reports.append(rep)
        REPORTS.append({"label": label, "request": int(req), **rep})
    return reports
