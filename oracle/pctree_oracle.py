"""Plain CPU oracle of the PCTree per-round draft-tree builder.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the bench's
CPU-baseline leg may import or run this module.  The product path (the HIP
library and its Python binding) never touches it, and this module shares no
code, tables or helpers with that path.

What it computes (paper Sec. 4, Alg. 1), for each request independently and in
float64 throughout, materialising every row of child logits:

1. frontier <- {x_t} with joint score 0; pool <- {x_t}            (Alg. 1 init)
2. for stage d = 0..B-1 (stage d builds tree level d+1, Sec. 4.1):
   a. every frontier parent p gets z_d(p) = L_d + Markov(p)        (Eq. 2/3)
      and log pi_d(.|p) = log_softmax(z_d(p))                      (Eq. 2)
   b. the local top-k children of p under log pi_d(.|p) join the pool with
      score s(child) = s(p) + log pi_d(child|p)                    (Eq. 4)
   c. the k highest-scoring candidates of this layer become the next
      frontier                                                     (Sec. 4.1)
3. S <- global top-N of the pool by (score desc, depth asc, stable id), the
   root included and always kept                                   (Sec. 4.2)
4. S is emitted as a flat token tensor with parent indices, position ids
   (tree depth + verified-prefix length) and the ancestor-only tree
   attention mask                                                  (App. A)

The Markov head.  The paper states only that the head is low-rank and adds a
bias determined by the preceding token (Sec. 3.2).  This oracle uses the form
``Markov_d(p) = W^T . SiLU(E[p] + h_d)`` with ``E[V][r]``, ``W[r][V]`` and a
per-depth feature ``h_d[r]``.

Readings where the paper is silent (each is also listed in the design notes):

* activation rounding: ``u = SiLU(x)`` is evaluated in float64 from
  ``x = E[p] + h_d`` and rounded to nearest-even onto float32, and then, for a
  bf16 drafter, onto bfloat16 -- the precision in which a bf16 head feeds its
  projection.  Everything after that is float64 here.
* per-parent child order: (log pi desc, token asc).
* layer order for the frontier: (score desc, token asc, parent slot asc),
  where the slot of a frontier node is its rank in that order.
* global order: (score desc, depth asc, token asc, parent slot asc); the
  "stable node identifier" is taken to be (token, parent slot).
* k' = min(k, V); the frontier after the last stage is not formed (it is
  never used); a pool smaller than N is emitted whole.
* emission order: depth ascending, then the root-to-node token path in
  lexicographic order (equivalently: parent's emitted index, then token).
* the mask covers the N x N tree block only (prefix columns are all ones
  for the consumer), packed 32 nodes per uint32 word, bit j%32 of word j//32.

Parity pins (tests/test_oracle_pins.py): brute-force enumeration of all
V^d paths, an exact best-first top-N search, the greedy chain of Eq. 1 for
k = 1, the Shared-Markov control for a parent-independent head, the
parent-independent scoring as the tree of a zero head, the W = 0 closed form, a hand-derived V = 4 example, and structural invariants.
Parity unpinned by the paper: emission order, padding values and the
activation rounding points above (choices of this library, not of the paper).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

__all__ = [
    "activation",
    "child_logprobs",
    "local_topk",
    "build_tree",
    "build_tree_batch",
    "chain_decode",
    "shared_markov_rows",
    "position_rows",
    "ancestor_mask",
    "Node",
]


# ---------------------------------------------------------------------------
# The Markov head and one row of child log-probabilities (Eq. 2 / Eq. 3)
# ---------------------------------------------------------------------------

def _to_bf16_rne(x32: np.ndarray) -> np.ndarray:
    """Round float32 values to nearest-even on the bfloat16 grid (finite inputs)."""
    b = np.asarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    rounded = ((b + 0x7FFF + lsb) >> 16) << 16
    return rounded.astype(np.uint32).view(np.float32)


def activation(E_row: np.ndarray, h_row: np.ndarray, dtype: str) -> np.ndarray:
    """u = SiLU(E[p] + h_d) at the drafter's input precision (float64 result).

    SiLU(x) = x * sigmoid(x) = x / (1 + exp(-x)), evaluated in float64, then
    rounded to float32 and, for a bf16 drafter, to bfloat16.
    """
    x = E_row.astype(np.float64) + h_row.astype(np.float64)
    with np.errstate(over="ignore"):
        silu = x / (1.0 + np.exp(-x))
    u32 = silu.astype(np.float32)
    if dtype == "bf16":
        u32 = _to_bf16_rne(u32)
    elif dtype != "f32":
        raise ValueError(dtype)
    return u32.astype(np.float64)


def child_logprobs(L_d, E, W, h_d, parent_token: int, dtype: str):
    """z_d(p) = L_d + Markov(p) and log pi_d(.|p) = log_softmax(z_d(p)).

    Returns (z, lse, logpi) as float64; ``W`` is the mathematical [r][V] matrix.
    """
    u = activation(E[parent_token], h_d, dtype)
    z = L_d.astype(np.float64) + u @ W  # Eq. 3 for one parent: the shared L_d plus its own bias
    m = z.max()
    lse = m + np.log(np.sum(np.exp(z - m)))
    logpi = z - lse  # Eq. 2
    return z, lse, logpi


def local_topk(logpi: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k best children: stable sort by (log pi desc, token asc)."""
    order = np.argsort(-logpi, kind="stable")
    return order[:k]


# ---------------------------------------------------------------------------
# Tree construction (Alg. 1)
# ---------------------------------------------------------------------------

@dataclass
class Node:
    token: int
    parent: int  # pool index of the parent, -1 for the root
    depth: int
    score: float  # joint path score s(c), Eq. 4
    slot: int  # frontier slot of the parent (0 for the root)
    path: tuple  # root-to-node token path, root excluded


def _glob_key(n: Node):
    return (-n.score, n.depth, n.token, n.slot)


def _layer_key(n: Node):
    return (-n.score, n.token, n.slot)


def position_rows(L_d):
    """Parent-independent row of one depth: log_softmax(L_d) in float64 (Eq. 2
    with no Markov term)."""
    z = L_d.astype(np.float64)
    m = z.max()
    return z - (m + np.log(np.sum(np.exp(z - m))))


def shared_markov_rows(L, E, W, h, x_t: int, dtype: str):
    """Shared-Markov control (Sec. 5.3): the greedy chain's refined rows q_d.

    The DSpark chain of Eq. 1 is built first; at depth d its row
    log pi_d(.|y_{d-1}) is reused for every parent of that depth.
    """
    rows = []
    prev = x_t
    for d in range(L.shape[0]):
        _, _, logpi = child_logprobs(L[d], E, W, h[d], prev, dtype)
        rows.append(logpi)
        prev = int(local_topk(logpi, 1)[0])
    return rows


def build_tree(L, E, W, h, x_t: int, prefix_len: int, k: int, N: int, dtype: str,
               mode: str = "parent"):
    """One request's round.  ``L [B][V]``, ``E [V][r]``, ``W [r][V]``, ``h [B][r]``.

    ``mode="parent"`` is PCTree (every parent conditions its own row);
    ``mode="shared"`` is the Shared-Markov control; ``mode="independent"`` is
    parent-independent per-position scoring (Sec. 4: every parent of depth d
    is expanded with the backbone's own distribution, log_softmax(L_d)).
    Returns a dict with the emitted tree and the per-stage record
    (candidates, frontiers).
    """
    B, V = L.shape
    kk = min(k, V)
    if mode == "shared":
        shared = shared_markov_rows(L, E, W, h, x_t, dtype)
    elif mode == "independent":
        shared = [position_rows(L[d]) for d in range(B)]
    elif mode == "parent":
        shared = None
    else:
        raise ValueError(mode)

    pool = [Node(token=int(x_t), parent=-1, depth=0, score=0.0, slot=0, path=())]
    frontier = [0]
    stages = []
    for d in range(B):
        cands = []
        rows = []
        for j, p in enumerate(frontier):
            par = pool[p]
            if shared is None:
                _, _, logpi = child_logprobs(L[d], E, W, h[d], par.token, dtype)
            else:
                logpi = shared[d]
            rows.append(logpi)
            for v in local_topk(logpi, kk):
                v = int(v)
                cands.append(Node(token=v, parent=p, depth=d + 1,
                                  score=par.score + float(logpi[v]), slot=j,
                                  path=par.path + (v,)))
        first = len(pool)
        pool.extend(cands)  # every child joins the pool before pruning
        cand_ids = list(range(first, len(pool)))
        stage = {"frontier": list(frontier), "candidates": cand_ids, "rows": rows}
        if d < B - 1:
            ranked = sorted(cand_ids, key=lambda i: _layer_key(pool[i]))
            frontier = ranked[:kk]
            stage["next_frontier"] = list(frontier)
            stage["layer_ranked"] = ranked
        stages.append(stage)

    ranked_all = sorted(range(len(pool)), key=lambda i: _glob_key(pool[i]))
    count = min(N, len(pool))
    S = ranked_all[:count]
    assert S[0] == 0, "the root (score 0) must be selected first"
    in_S = set(S)
    assert all(pool[i].parent in in_S for i in S[1:]), "selected set is not prefix-closed"

    # Emission: depth ascending, then (parent's emitted index, token).
    emit_of = {}
    order = []
    for lev in range(B + 1):
        level = [i for i in S if pool[i].depth == lev]
        level.sort(key=lambda i: (emit_of.get(pool[i].parent, -1), pool[i].token))
        for i in level:
            emit_of[i] = len(order)
            order.append(i)
    assert len(order) == count

    token = np.full(N, -1, np.int32)
    parent = np.full(N, -1, np.int32)
    depth = np.full(N, -1, np.int32)
    position = np.full(N, -1, np.int32)
    logprob = np.full(N, -np.inf, np.float64)
    for e, i in enumerate(order):
        n = pool[i]
        token[e] = n.token
        parent[e] = emit_of[n.parent] if n.parent >= 0 else -1
        depth[e] = n.depth
        position[e] = prefix_len + n.depth  # App. A: tree depth + verified prefix length
        logprob[e] = n.score
    mask = ancestor_mask(parent, count, N)
    return {
        "token": token, "parent": parent, "depth": depth, "position": position,
        "logprob": logprob, "count": count, "mask": mask,
        "pool": pool, "stages": stages, "selected": S, "ranked_all": ranked_all,
        "order": order,
    }


def ancestor_mask(parent: np.ndarray, count: int, N: int) -> np.ndarray:
    """Ancestor-only tree mask (App. A): row i admits i itself and its ancestors.

    Packed as uint32 words [N][ceil(N/32)], bit j%32 of word j//32; rows at or
    beyond ``count`` are zero.
    """
    nw = (N + 31) // 32
    dense = np.zeros((N, N), dtype=bool)
    for i in range(count):
        j = i
        while j >= 0:
            dense[i, j] = True
            j = int(parent[j])
    words = np.zeros((N, nw), dtype=np.uint32)
    for i in range(N):
        for j in np.nonzero(dense[i])[0]:
            words[i, j // 32] |= np.uint32(1) << np.uint32(j % 32)
    return words


def chain_decode(L, E, W, h, x_t: int, dtype: str, mode: str = "parent"):
    """The DSpark chain of Eq. 1: y_d = argmax_v z_d(y_{d-1}), y_{-1} = x_t.

    Ties go to the lowest token id.  Returns tokens [B+1] (x_t first) and the
    cumulative log-probabilities [B+1] (0 for x_t).  A chain has one parent
    per depth, so ``mode="shared"`` gives the same chain; ``mode="independent"``
    takes each y_d from log_softmax(L_d) alone.
    """
    B = L.shape[0]
    toks = [int(x_t)]
    cum = [0.0]
    for d in range(B):
        if mode == "independent":
            logpi = position_rows(L[d])
        else:
            _, _, logpi = child_logprobs(L[d], E, W, h[d], toks[-1], dtype)
        y = int(np.flatnonzero(logpi == logpi.max())[0])
        toks.append(y)
        cum.append(cum[-1] + float(logpi[y]))
    return np.array(toks, np.int32), np.array(cum, np.float64)


def build_tree_batch(inp: dict, k: int, N: int, mode: str = "parent"):
    """Run :func:`build_tree` for every request of a synthetic batch."""
    w = inp["workload"]
    dtype = w.dtype
    E = inp["E"]
    W = inp["W"].astype(np.float64)
    out = []
    for i in range(inp["L"].shape[0]):
        out.append(build_tree(inp["L"][i], E, W, inp["h"][i], int(inp["root"][i]),
                              int(inp["prefix_len"][i]), k, N, dtype, mode))
    return out
