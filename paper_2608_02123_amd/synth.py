"""Seeded synthetic inputs for one draft-tree round.

This module draws the tensors a tree-build round consumes: shared base logits
``L[R][B][V]`` (standing in for one parallel-backbone forward, Sec. 3.2), the
Markov-head parameters ``E[V][r]``, ``W[r][V]`` and per-depth features
``h[R][B][r]``, the root token ``x_t`` and the verified-prefix length of each
request.  It performs none of the method's arithmetic: it only draws numbers
and rounds them once to the storage precision, so both the CPU oracle and the
GPU path receive bit-identical operands.

Recipe (the paper measured Qwen3-4B/8B/14B with DSpark drafts on nine public
suites; none of those checkpoints or datasets are used, these seeded tensors
stand in for them):

* ``L_d[v] ~ N(0, 3^2)`` plus a peak added to 3 distinct tokens per depth whose
  rank follows a Zipf(1.1) law truncated to ``[1, V]`` (token = rank - 1).
  Peak height: +8 (``"const8"``), ``U(4, 12)`` per depth (``"uniform"``), or
  ``12 - 9 d / (B - 1)`` (``"decay"``: confidence falling with depth).
* ``E ~ N(0, 0.02)``, ``W ~ N(0, 0.05)`` (standard deviations), ``h ~ N(0, 1)``.
* root token uniform over the vocabulary; prefix length uniform in [1, 1024].
* Values are drawn in float64 and rounded once, round-to-nearest-even, to the
  storage dtype (``"f32"`` or ``"bf16"``).  ``h`` is always float32.

Streams: request ``i`` of a batch draws ``root, prefix_len, L, h`` from
``default_rng((seed + i, 1))``; the shared head ``E, W`` comes from
``default_rng((seed, 2))`` (one drafter serves every request).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = ["Workload", "CONFIGS", "make_inputs", "round_to_bf16", "bf16_bits",
           "random_tree", "target_next", "make_kv_cache", "ATTN_SHAPES",
           "make_attention_inputs"]


@dataclass(frozen=True)
class Workload:
    """Shape of one tree-build round (symbols as in the paper's Sec. 4.1)."""

    name: str
    V: int  # vocabulary size
    B: int  # block size = number of sequential Markov stages
    N: int  # verification node budget (root included)
    k: int  # local branching factor
    r: int  # Markov-head rank
    R: int = 1  # independent requests built in one call
    dtype: str = "bf16"  # storage dtype of L, E, W
    peak: str = "const8"  # peak-height schedule of the base logits
    seed: int = 0
    sigma_L: float = 3.0
    sigma_E: float = 0.02
    sigma_W: float = 0.05
    extra: dict = field(default_factory=dict)


# The five workloads of the headline table plus the brute-force shape.
CONFIGS = {
    "tiny": Workload("tiny", V=1024, B=4, N=16, k=4, r=32, dtype="f32", peak="const8"),
    "brute": Workload("brute", V=8, B=4, N=10, k=8, r=32, dtype="f32", peak="const8"),
    "qwen4b_b7": Workload("qwen4b_b7", V=151936, B=7, N=32, k=8, r=256, peak="const8"),
    "qwen8b_b7": Workload("qwen8b_b7", V=151936, B=7, N=48, k=8, r=384, peak="uniform"),
    "qwen4b_b16": Workload("qwen4b_b16", V=151936, B=16, N=64, k=8, r=256, peak="decay"),
    "qwen14b_b16_r8": Workload(
        "qwen14b_b16_r8", V=151936, B=16, N=128, k=16, r=512, R=8, peak="decay"
    ),
}


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values once, to nearest-even, onto the bfloat16 grid.

    Works on the float64 bit pattern: bfloat16 keeps 7 of the 52 stored
    mantissa bits, so the low 45 bits are rounded away (ties to even).
    Returns float32 values that are exactly representable in bfloat16.
    (Finite inputs within the float32 normal range, or zero.)
    """
    b = np.ascontiguousarray(x, dtype=np.float64).view(np.uint64)
    lsb = (b >> np.uint64(45)) & np.uint64(1)
    b = (b + (np.uint64((1 << 44) - 1) + lsb)) & ~np.uint64((1 << 45) - 1)
    return b.view(np.float64).astype(np.float32)


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that already lie on the bf16 grid."""
    b = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    if np.any(b & 0xFFFF):
        raise ValueError("values are not bfloat16-representable")
    return (b >> 16).astype(np.uint16)


def _round(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return x.astype(np.float32)
    if dtype == "bf16":
        return round_to_bf16(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def _zipf_tokens(rng: np.random.Generator, V: int, count: int, a: float = 1.1) -> np.ndarray:
    """``count`` distinct tokens whose rank follows Zipf(a) truncated to [1, V]."""
    count = min(count, V)
    w = np.arange(1, V + 1, dtype=np.float64) ** (-a)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    out: list[int] = []
    while len(out) < count:
        t = int(np.searchsorted(cdf, rng.random(), side="right"))
        t = min(t, V - 1)
        if t not in out:
            out.append(t)
    return np.array(out, dtype=np.int64)


def _peak_height(w: Workload, d: int, rng: np.random.Generator) -> float:
    if w.peak == "const8":
        return 8.0
    if w.peak == "uniform":
        return float(rng.uniform(4.0, 12.0))
    if w.peak == "decay":
        return 12.0 - 9.0 * d / max(w.B - 1, 1)
    if w.peak == "none":
        return 0.0
    raise ValueError(f"unknown peak schedule {w.peak!r}")


def make_inputs(w: Workload) -> dict:
    """Draw one round's inputs.

    Returns a dict of numpy arrays: ``L [R][B][V]``, ``E [V][r]``, ``W [r][V]``
    (float32 holding values of the storage dtype), ``h [R][B][r]`` float32,
    ``root [R]`` and ``prefix_len [R]`` int32, and ``workload``.
    """
    R, B, V, r = w.R, w.B, w.V, w.r
    L = np.empty((R, B, V), dtype=np.float32)
    h = np.empty((R, B, r), dtype=np.float32)
    root = np.empty(R, dtype=np.int32)
    prefix_len = np.empty(R, dtype=np.int32)
    for i in range(R):
        rng = np.random.default_rng((w.seed + i, 1))
        root[i] = rng.integers(0, V)
        prefix_len[i] = rng.integers(1, 1025)
        Li = rng.standard_normal((B, V)) * w.sigma_L
        for d in range(B):
            toks = _zipf_tokens(rng, V, 3)
            Li[d, toks] += _peak_height(w, d, rng)
        L[i] = _round(Li, w.dtype)
        h[i] = rng.standard_normal((B, r)).astype(np.float32)
    rs = np.random.default_rng((w.seed, 2))
    E = _round(rs.standard_normal((V, r)) * w.sigma_E, w.dtype)
    W = _round(rs.standard_normal((r, V)) * w.sigma_W, w.dtype)
    return {
        "L": L,
        "E": E,
        "W": W,
        "h": h,
        "root": root,
        "prefix_len": prefix_len,
        "workload": w,
    }


# ---------------------------------------------------------------------------
# Inputs of the verification bookkeeping after a round
# ---------------------------------------------------------------------------

def random_tree(rng: np.random.Generator, N: int, count: int, max_depth: int, V: int):
    """A random tree of ``count`` nodes in ``N`` slots, shaped like an emitted one.

    Node 0 is the root; node i > 0 hangs below a uniformly drawn earlier node
    of depth < ``max_depth`` (so ``parent[i] < i``), with a token drawn
    uniformly from the vocabulary and distinct from its siblings' tokens.
    Slots past ``count`` hold -1.  Returns ``(token, parent, depth)`` int32.
    """
    token = np.full(N, -1, np.int32)
    parent = np.full(N, -1, np.int32)
    depth = np.full(N, -1, np.int32)
    if count <= 0:
        return token, parent, depth
    token[0] = rng.integers(0, V)
    depth[0] = 0
    kids: dict[int, set] = {0: set()}
    for i in range(1, count):
        open_nodes = [j for j in range(i) if depth[j] < max_depth and len(kids[j]) < V]
        p = int(open_nodes[rng.integers(0, len(open_nodes))])
        t = int(rng.integers(0, V))
        while t in kids[p]:
            t = int(rng.integers(0, V))
        kids[p].add(t)
        kids[i] = set()
        token[i], parent[i], depth[i] = t, p, depth[p] + 1
    return token, parent, depth


def target_next(rng: np.random.Generator, token: np.ndarray, parent: np.ndarray, count: int,
                V: int, accept_p: float) -> np.ndarray:
    """Synthetic greedy predictions of the target at each tree node.

    Stands in for the argmax of the verification forward's logits: at a node
    with children, with probability ``accept_p`` the prediction is the token
    of one of its children (drawn uniformly), otherwise a uniform token.
    """
    N = len(token)
    out = rng.integers(0, V, size=N).astype(np.int32)
    children: dict[int, list] = {}
    for i in range(1, max(0, min(count, N))):
        children.setdefault(int(parent[i]), []).append(int(token[i]))
    for i in range(max(0, min(count, N))):
        kids = children.get(i)
        if kids and rng.random() < accept_p:
            out[i] = kids[int(rng.integers(0, len(kids)))]
    return out


def make_kv_cache(rng: np.random.Generator, groups: int, capacity: int, width: int) -> np.ndarray:
    """A synthetic bf16 KV cache ``[groups][capacity][width]`` (as uint16 bits).

    ``groups`` stands for (layer, K or V) pairs of a target model; every slot
    holds ``width`` bf16 values (heads x head dimension).  Random bit patterns
    of finite values: the compaction only moves them.
    """
    bits = rng.integers(0, 1 << 16, size=(groups, capacity, width), dtype=np.uint32)
    bits &= ~np.uint32(0x4000)  # exponent below all ones: finite values
    return bits.astype(np.uint16)


# ---------------------------------------------------------------------------
# Inputs of one tree-masked verification attention layer
# ---------------------------------------------------------------------------

# (query heads, key/value heads, head dimension) of the Qwen3 targets'
# attention layers (grouped-query attention).
ATTN_SHAPES = {
    "qwen3_4b": (32, 8, 128),
    "qwen3_8b": (32, 8, 128),
    "qwen3_14b": (40, 8, 128),
}


def make_attention_inputs(rng: np.random.Generator, R: int, N: int, Hq: int, Hkv: int, D: int,
                          prefix_len: np.ndarray, count: np.ndarray, capacity: int,
                          q_scale: float = 1.0) -> dict:
    """Synthetic operands of one attention layer of the verification forward.

    ``q [R][N][Hq][D]`` (``N(0, q_scale^2)``), ``k`` and ``v [R][Hkv][capacity][D]``
    (``N(0, 1)``), all rounded once to bf16 (float32 arrays on the bf16 grid).
    Slots ``prefix_len[r] + count[r]`` and beyond, which no query may read,
    hold NaN, so that a read past the admitted slots cannot go unnoticed.
    Query rows at or past ``count[r]`` are drawn like the others.
    A larger ``q_scale`` sharpens the attention rows.
    """
    q = round_to_bf16(rng.normal(0.0, q_scale, size=(R, N, Hq, D)))
    k = round_to_bf16(rng.normal(0.0, 1.0, size=(R, Hkv, capacity, D)))
    v = round_to_bf16(rng.normal(0.0, 1.0, size=(R, Hkv, capacity, D)))
    for r in range(R):
        end = int(prefix_len[r]) + int(count[r])
        k[r, :, end:] = np.nan
        v[r, :, end:] = np.nan
    return {"q": q, "k": k, "v": v}
