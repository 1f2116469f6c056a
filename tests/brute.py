"""Exhaustive and best-first reference searches used to pin the oracle.

These are written independently of ``oracle/``: they score every root-to-node
path directly from the definitions (Eq. 2 row log-softmax, Eq. 4 path score)
and select the global top-N with no frontier pruning at all.  Under the width
condition "k' >= |S* ∩ level d| for every depth d" PCTree's layer-wise
pruning cannot lose a node of the exact top-N S*, so the oracle must return
exactly S*; below that width only validity can be asserted (Sec. 6, item 2).
"""
from __future__ import annotations

import heapq
import itertools

import numpy as np
from scipy.special import expit, log_softmax


def head_row(L_d, E, W, h_d, u_tok, dtype):
    """log pi_d(.|u) straight from the definitions, float64."""
    x = E[u_tok].astype(np.float64) + h_d.astype(np.float64)
    a = (x * expit(x)).astype(np.float32)  # SiLU, rounded to the f32 head input
    if dtype == "bf16":
        b = a.view(np.uint32).astype(np.uint64)
        b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
        a = b.astype(np.uint32).view(np.float32)
    z = L_d.astype(np.float64) + a.astype(np.float64) @ W.astype(np.float64)
    return log_softmax(z)


def brute_force_topn(L, E, W, h, x_t, N, dtype):
    """Exact top-N over all sum_{d<=B} V^d prefixes (root included).

    Returns a list of (path, score) sorted by (score desc, depth asc, path asc)
    and the gap between the N-th and (N+1)-th score.
    """
    B, V = L.shape
    table = np.array([[head_row(L[d], E, W, h[d], u, dtype) for u in range(V)]
                      for d in range(B)])  # [B][V(parent)][V(child)]
    nodes = [((), 0.0)]
    for depth in range(1, B + 1):
        for path in itertools.product(range(V), repeat=depth):
            s = 0.0
            prev = x_t
            for d, v in enumerate(path):
                s += table[d, prev, v]
                prev = v
            nodes.append((path, s))
    nodes.sort(key=lambda t: (-t[1], len(t[0]), t[0]))
    gap = nodes[N - 1][1] - nodes[N][1] if len(nodes) > N else np.inf
    return nodes[:N], gap


def best_first_topn(L, E, W, h, x_t, N, dtype):
    """Exact top-N by best-first search.

    Path scores never increase along a path (every log-probability is <= 0), so
    popping the best open node from a max-heap yields nodes in non-increasing
    score order; the first N pops are the exact top-N.
    """
    B, V = L.shape
    heap = [(0.0, 0, (), int(x_t))]
    out = []
    while heap and len(out) < N + 1:
        negs, depth, path, tok = heapq.heappop(heap)
        out.append((path, -negs))
        if depth < B:
            row = head_row(L[depth], E, W, h[depth], tok, dtype)
            for v in range(V):
                heapq.heappush(heap, (negs - float(row[v]), depth + 1, path + (v,), v))
    gap = out[N - 1][1] - out[N][1] if len(out) > N else np.inf
    return out[:N], gap
