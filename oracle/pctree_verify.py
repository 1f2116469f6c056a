"""Plain CPU oracle of the tree-verification bookkeeping that follows a round.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the bench's
CPU-baseline leg may import or run this module.  The product path never
touches it, and it shares no code with that path.

What it computes (paper Sec. 4.2 and App. A, "Tensor implementation"):

* retrieve indices: the selected tree induces padded root-to-leaf rows, one
  per leaf, used to compare each proposed child with the target's prediction
  at the node before it;
* greedy tree acceptance: the standard greedy tree rule of speculative
  decoding (the rule of SpecInfer and EAGLE-2 that the paper uses): along a
  row, a proposed node is accepted when its token equals the target's greedy
  next token at the preceding node of the row, and every earlier node of the
  row was accepted; the longest accepted row wins, and the target's
  prediction at its last accepted node is the bonus token;
* compaction: after the longest accepted row is chosen, the per-node KV
  entries (and target hidden states) along that row are gathered and written
  right after the verified prefix.

Readings where the paper is silent (each is also listed in the design notes):

* a leaf is a selected node that is no selected node's parent; rows are in
  ascending leaf index (with the canonical emission order of the tree
  builder this is the root-to-leaf token paths in depth-then-lexicographic
  order of their leaves);
* each row lists node indices from the root to its leaf and is padded with -1
  to ``max_depth + 1`` entries;
* the accepted length counts accepted draft nodes, the root excluded; rows
  that accept equally long prefixes accept the same nodes (siblings carry
  distinct tokens), and the lowest row index is reported;
* malformed trees: a parent index outside ``[0, i)`` for node ``i`` is no
  edge (the upward walk from a leaf stops there, and that node heads the
  row); a path longer than ``max_depth + 1`` keeps its first
  ``max_depth + 1`` nodes from the head; row entries outside ``[0, N)`` end
  a row;
* an empty tree (count 0) has no rows: accepted length 0, row -1, bonus -1.

Parity pins (tests/test_verify_pins.py): a node-by-node walk down the tree,
exhaustive checking of every node's ancestor chain, the chain case (k = 1,
where the rule is the plain longest matching prefix), row invariants and a
hand-derived example in tests/golden/verify_hand.json.  Parity unpinned by
the paper: the row order, the padding values and the malformed-input rules
above (choices of this library, not of the paper).
"""
from __future__ import annotations

import numpy as np

__all__ = ["retrieve_rows", "accept_greedy", "compact_rows"]


def _edge(parent: np.ndarray, i: int) -> int:
    """The parent of node i if it is a valid edge (in [0, i)), else -1."""
    p = int(parent[i])
    return p if 0 <= p < i else -1


def retrieve_rows(parent: np.ndarray, count: int, max_depth: int):
    """Padded root-to-leaf rows of one request's tree (App. A).

    ``parent[N]`` as emitted by the tree builder, ``count`` selected nodes.
    Returns ``(rows [N][max_depth+1] int32, nrows)``; rows past ``nrows`` are
    all -1.
    """
    N = len(parent)
    count = max(0, min(int(count), N))
    has_child = np.zeros(N, dtype=bool)
    for j in range(count):
        p = _edge(parent, j)
        if p >= 0:
            has_child[p] = True
    width = max_depth + 1
    rows = np.full((N, width), -1, np.int32)
    nrows = 0
    for i in range(count):
        if has_child[i]:
            continue
        path = [i]
        while _edge(parent, path[-1]) >= 0:
            path.append(_edge(parent, path[-1]))
        path.reverse()  # head (the root of a well-formed tree) first
        path = path[:width]
        rows[nrows, : len(path)] = path
        nrows += 1
    return rows, nrows


def accept_greedy(token: np.ndarray, rows: np.ndarray, nrows: int, target_next: np.ndarray):
    """Greedy tree acceptance over the retrieve rows (Sec. 4.2, App. A).

    ``token[N]`` are the draft tokens, ``target_next[N]`` the target's greedy
    next token after each node (from the one verification forward).  Returns
    ``(accept_len, best_row, accepted_nodes [max_depth+1], bonus)``.
    """
    N = len(token)
    width = rows.shape[1]
    nodes = np.full(width, -1, np.int32)
    best_len, best_row = -1, -1
    for j in range(int(nrows)):
        row = rows[j]
        if not (0 <= row[0] < N):
            continue
        a = 0
        # position l is accepted if its token equals the target's prediction
        # at position l - 1 and every earlier position was accepted
        for l in range(1, width):
            if not (0 <= row[l] < N):
                break
            if int(token[row[l]]) != int(target_next[row[l - 1]]):
                break
            a = l
        if a > best_len:  # strict: ties keep the lowest row
            best_len, best_row = a, j
    if best_row < 0:
        return 0, -1, nodes, -1
    nodes[: best_len + 1] = rows[best_row, : best_len + 1]
    bonus = int(target_next[rows[best_row, best_len]])
    return best_len, best_row, nodes, bonus


def compact_rows(cache: np.ndarray, prefix_len: int, accepted_nodes: np.ndarray,
                 accept_len: int) -> np.ndarray:
    """KV compaction after acceptance (App. A).

    ``cache[T][...]`` holds the verified prefix at ``[0, prefix_len)`` and the
    tree's entries at ``[prefix_len, prefix_len + N)`` (tree node i at slot
    ``prefix_len + i``).  The entries of the accepted nodes, root first, move
    to slots ``prefix_len .. prefix_len + accept_len``; every other slot keeps
    its value.  Returns the new cache (the input is not modified).
    """
    out = cache.copy()
    for m in range(int(accept_len) + 1):
        out[prefix_len + m] = cache[prefix_len + int(accepted_nodes[m])]
    return out
