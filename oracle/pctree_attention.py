"""Plain CPU oracle of tree-masked verification attention (one target layer).

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the bench's
CPU-baseline leg may import or run this module.  The product path never
touches it, and it shares no code with that path.

What it computes (paper Sec. 4.2 and App. A, "Tensor implementation"): the
emitted tree is checked in one forward of the target model, in which the
query of tree node i may look at the verified prefix, at node i itself and at
the nodes on its path up to the root, and at nothing else.  For one attention
layer with grouped-query heads (``g = Hq / Hkv`` query heads share a key/value
head, query head h reading key/value head ``h // g``) this is

    out[r, i, h] = sum_{s in A(r, i)} softmax_s(scale * q[r, i, h] . K[r, h//g, s])
                                      * V[r, h//g, s]

with ``A(r, i) = {0 .. P-1} U {P + j : bit j of mask row i is set, j < count}``,
``P = prefix_len[r]``: cache slot ``P + j`` holds tree node j (the layout the
compaction step assumes).  Everything is evaluated in float64 from the
stored (bf16) operands, by the plain definition: a full score row, its
maximum, exponentials, their sum, and the weighted sum of value rows.

Readings where the paper is silent (each is also listed in the design notes):

* the mask rows are the builder's packed ancestor words (bit j % 32 of word
  j // 32); a bit at or past ``count`` is ignored;
* a query row at or past ``count`` has no output: it is all zeros;
* a row that admits no slot at all (empty prefix and an empty mask row) is
  all zeros;
* ``scale`` is the caller's (usually ``1 / sqrt(D)``); the oracle uses its
  float64 value.

Parity pins (tests/test_attention_pins.py): torch's scaled dot-product
attention in float64 with an explicit boolean mask (a library routine), a
single admitted slot (the output is that slot's value row), equal keys (the
output is the mean of the admitted value rows), invariance of the output
under a permutation of the prefix slots, the chain tree (k = 1) as causal
attention, and planted mistakes in a copy of this module, each caught by a
pin.
"""
from __future__ import annotations

import numpy as np

__all__ = ["admitted_slots", "tree_attention"]


def admitted_slots(mask_row: np.ndarray, count: int, prefix_len: int) -> np.ndarray:
    """Cache slots one tree query may read: the prefix, then its tree nodes."""
    tree = [prefix_len + j for j in range(count)
            if (int(mask_row[j // 32]) >> (j % 32)) & 1]
    return np.concatenate([np.arange(prefix_len, dtype=np.int64),
                           np.asarray(tree, dtype=np.int64)])


def tree_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, mask: np.ndarray,
                   count: np.ndarray, prefix_len: np.ndarray, scale: float) -> np.ndarray:
    """Tree-masked attention of every request, node and query head.

    q [R][N][Hq][D], k and v [R][Hkv][C][D] (any float dtype; read as float64),
    mask [R][N][ceil(N/32)] uint32, count [R], prefix_len [R].
    Returns out [R][N][Hq][D] float64.
    """
    R, N, Hq, D = q.shape
    Hkv = k.shape[1]
    g = Hq // Hkv
    out = np.zeros((R, N, Hq, D), dtype=np.float64)
    for r in range(R):
        c = int(count[r])
        P = int(prefix_len[r])
        for i in range(min(c, N)):
            slots = admitted_slots(mask[r, i], c, P)
            if slots.size == 0:
                continue
            for h in range(Hq):
                kv = h // g
                keys = k[r, kv, slots].astype(np.float64)
                vals = v[r, kv, slots].astype(np.float64)
                s = float(scale) * (keys @ q[r, i, h].astype(np.float64))
                e = np.exp(s - s.max())
                out[r, i, h] = (e @ vals) / e.sum()
    return out
