"""C ABI checks that need no GPU: the library loads, exports every function that
include/pctree.h declares, and rejects bad arguments on the host before any
device work (so every error status is reachable without a device)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

from paper_2608_02123_amd import pctree as P

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include")
HEADERS = sorted(os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h"))
A = 0x100000  # fake, suitably aligned device addresses (validation never dereferences)


def declared_functions():
    names = set()
    for h in HEADERS:
        text = open(h).read()
        names |= set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(pctree_\w+)\s*\(", text, re.M))
    return sorted(names)


def test_exports_every_declared_symbol():
    """Every function that include/*.h declares, in the default library and
    in its stage-timeline build."""
    names = declared_functions()
    assert {"pctree_build_tree", "pctree_build_mask", "pctree_chain_decode",
            "pctree_workspace_bytes", "pctree_status_string", "pctree_abi_version",
            "pctree_profile_enable", "pctree_debug_set", "pctree_timeline_read"} <= set(names)
    for path in (P.LIB_PATH, P.TIMELINE_LIB_PATH):
        lib = ctypes.CDLL(path)
        for n in names:
            assert hasattr(lib, n), (path, n)
    assert P.lib().pctree_abi_version() == 1


def test_status_strings():
    for code, name in enumerate(["PCTREE_OK", "PCTREE_ERR_INVALID_ARGUMENT",
                                 "PCTREE_ERR_UNSUPPORTED", "PCTREE_ERR_WORKSPACE",
                                 "PCTREE_ERR_HIP"]):
        assert P.status_string(code) == name
    assert P.status_string(99) == "PCTREE_ERR_UNKNOWN"


def shape(**kw):
    base = dict(vocab=151936, block=16, budget=64, topk=8, rank=256, requests=1, dtype=P.BF16,
                mode=0)
    base.update(kw)
    return P.Shape(*(base[n] for n, _ in P.Shape._fields_))


def inputs(**kw):
    base = {n: A + 0x1000 * i for i, (n, _) in enumerate(P._Inputs._fields_)}
    base.update(kw)
    return P._Inputs(*(base[n] for n, _ in P._Inputs._fields_))


def tree(**kw):
    base = {n: A + 0x100000 + 0x1000 * i for i, (n, _) in enumerate(P._Tree._fields_)}
    base.update(kw)
    return P._Tree(*(base[n] for n, _ in P._Tree._fields_))


def build(s=None, i=None, t=None, tr=None, ws=A * 16, nbytes=None):
    s = s if s is not None else shape()
    if nbytes is None:
        nbytes = P.lib().pctree_workspace_bytes(ctypes.byref(s)) if s else 0
    return P.lib().pctree_build_tree(
        ctypes.byref(s) if s is not None else None,
        ctypes.byref(i) if i is not None else None,
        ctypes.byref(t) if t is not None else None,
        ctypes.byref(tr) if tr is not None else None,
        ctypes.c_void_p(ws) if ws else None, nbytes, None)


@pytest.mark.parametrize("field", ["vocab", "block", "budget", "topk", "rank", "requests"])
def test_nonpositive_sizes_are_invalid(field):
    assert build(shape(**{field: 0}), inputs(), tree()) == P.ERR_INVALID_ARGUMENT
    assert build(shape(**{field: -3}), inputs(), tree()) == P.ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), P.ERR_INVALID_ARGUMENT),
    (dict(mode=3), P.ERR_UNSUPPORTED),
    (dict(mode=-1), P.ERR_UNSUPPORTED),
    (dict(vocab=(1 << 20) + 1), P.ERR_UNSUPPORTED),
    (dict(block=64), P.ERR_UNSUPPORTED),
    (dict(topk=17), P.ERR_UNSUPPORTED),
    (dict(budget=257), P.ERR_UNSUPPORTED),
    (dict(requests=257), P.ERR_UNSUPPORTED),
    (dict(rank=48), P.ERR_UNSUPPORTED),
    (dict(rank=544), P.ERR_UNSUPPORTED),
    (dict(dtype=P.F32, rank=40), P.ERR_UNSUPPORTED),
    (dict(dtype=P.F32, rank=144), P.ERR_UNSUPPORTED),
])
def test_shape_limits(kw, code):
    assert build(shape(**kw), inputs(), tree()) == code
    assert P.lib().pctree_workspace_bytes(ctypes.byref(shape(**kw))) == 0


def test_null_and_misaligned_pointers():
    assert P.lib().pctree_build_tree(None, None, None, None, None, 0, None) == \
        P.ERR_INVALID_ARGUMENT
    assert build(i=None, t=tree()) == P.ERR_INVALID_ARGUMENT
    for n, _ in P._Inputs._fields_:
        assert build(i=inputs(**{n: 0}), t=tree()) == P.ERR_INVALID_ARGUMENT, n
    assert build(i=inputs(proj_t=A + 8), t=tree()) == P.ERR_INVALID_ARGUMENT
    assert build(i=inputs(root_token=A + 2), t=tree()) == P.ERR_INVALID_ARGUMENT
    assert build(i=inputs(), t=None) == P.ERR_INVALID_ARGUMENT
    for n, _ in P._Tree._fields_:
        if n != "mask":
            assert build(i=inputs(), t=tree(**{n: 0})) == P.ERR_INVALID_ARGUMENT, n
    assert build(i=inputs(), t=tree(logprob=A + 2)) == P.ERR_INVALID_ARGUMENT
    bad_trace = P._Trace(A, 0, A)
    assert build(i=inputs(), t=tree(), tr=bad_trace) == P.ERR_INVALID_ARGUMENT


def test_workspace_errors():
    s = shape()
    need = P.lib().pctree_workspace_bytes(ctypes.byref(s))
    assert need > 0
    assert build(s, inputs(), tree(), ws=0) == P.ERR_WORKSPACE
    assert build(s, inputs(), tree(), ws=A * 16 + 128) == P.ERR_WORKSPACE
    assert build(s, inputs(), tree(), nbytes=need - 1) == P.ERR_WORKSPACE


def test_workspace_size_grows_with_the_problem():
    ws = lambda **kw: P.lib().pctree_workspace_bytes(ctypes.byref(shape(**kw)))  # noqa: E731
    assert ws(budget=128) >= ws(budget=64)
    assert ws(topk=16) > ws(topk=8)
    # within one form: the persistent one (R * k' <= 16) keeps every stage's
    # partials, the multi-launch one (R * k' > 16) reuses a single set
    assert ws(requests=2) > ws(requests=1)
    assert ws(requests=16) > ws(requests=8)
    assert ws(block=32) > ws(block=16)
    assert ws() % 256 == 0


def test_build_mask_validation():
    f = P.lib().pctree_build_mask
    assert f(None, A, 1, 8, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 0, 8, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 1, 0, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A + 1, A, 1, 8, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 1, 1025, A, None) == P.ERR_UNSUPPORTED


def test_chain_decode_validation():
    f = P.lib().pctree_chain_decode
    s = shape(topk=0, budget=0)  # ignored by the chain
    vp = ctypes.c_void_p
    assert f(ctypes.byref(shape(mode=3)), ctypes.byref(inputs()), vp(A), vp(A), vp(A * 16),
             1 << 30, None) == P.ERR_UNSUPPORTED
    assert f(ctypes.byref(s), ctypes.byref(inputs()), None, vp(A), vp(A * 16), 1 << 30,
             None) == P.ERR_INVALID_ARGUMENT
    assert f(ctypes.byref(s), ctypes.byref(inputs()), vp(A), vp(A), vp(A * 16), 64,
             None) == P.ERR_WORKSPACE
    assert f(ctypes.byref(s), None, vp(A), vp(A), vp(A * 16), 1 << 30,
             None) == P.ERR_INVALID_ARGUMENT


def test_build_retrieve_validation():
    f = P.lib().pctree_build_retrieve
    assert f(None, A, 1, 8, 4, A, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 0, 8, 4, A, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 1, 0, 4, A, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 1, 8, -1, A, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 1, 8, 4, None, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A + 2, 1, 8, 4, A, A, None) == P.ERR_INVALID_ARGUMENT
    assert f(A, A, 1, 1025, 4, A, A, None) == P.ERR_UNSUPPORTED
    assert f(A, A, 1, 8, 64, A, A, None) == P.ERR_UNSUPPORTED


def test_accept_greedy_validation():
    f = P.lib().pctree_accept_greedy
    ok = [A, A, A, A, 1, 8, 4, A, A, A, A]
    for i in (0, 1, 2, 3, 7, 8, 9, 10):
        args = list(ok)
        args[i] = None
        assert f(*args, None) == P.ERR_INVALID_ARGUMENT, i
        args[i] = A + 2
        assert f(*args, None) == P.ERR_INVALID_ARGUMENT, i
    for i, bad in ((4, 0), (5, 0), (6, -1)):
        args = list(ok)
        args[i] = bad
        assert f(*args, None) == P.ERR_INVALID_ARGUMENT, i
    for i, big in ((5, 1025), (6, 64)):
        args = list(ok)
        args[i] = big
        assert f(*args, None) == P.ERR_UNSUPPORTED, i


def test_compact_kv_validation():
    f = P.lib().pctree_compact_kv
    ok = [A, 1 << 20, 1 << 16, 4, 256, 256, A, A, A, 1, 64, 16]
    args = list(ok)
    args[0] = None
    assert f(*args, None) == P.ERR_INVALID_ARGUMENT
    for i, bad in ((0, A + 8), (1, 8), (2, 24), (5, 24), (5, 8), (3, 0), (4, 0), (9, 0),
                   (10, 0), (11, -1), (6, None), (7, A + 2), (8, None)):
        args = list(ok)
        args[i] = bad
        assert f(*args, None) == P.ERR_INVALID_ARGUMENT, (i, bad)
    for i, big in ((11, 64), (10, 1025)):
        args = list(ok)
        args[i] = big
        assert f(*args, None) == P.ERR_UNSUPPORTED, i


def _attn_shape(R=1, N=64, Hq=32, Hkv=8, D=128, C=1088, scale=None):
    return P.AttnShape(R, N, Hq, Hkv, D, C, 0.125 if scale is None else scale)


def test_tree_attention_workspace():
    ws = lambda **kw: P.lib().pctree_attention_workspace_bytes(ctypes.byref(_attn_shape(**kw)))  # noqa: E731,E501
    # few workgroups (one request, 8 kv heads, 2 query blocks): the 1088 slots are
    # split into 6 runs of 192, each leaving D + 2 floats per (node, head)
    assert ws() == 6 * 64 * 32 * (128 + 2) * 4 + 256
    # enough workgroups without a split: no workspace
    assert ws(R=8, N=128, Hq=40) == 0
    assert ws(C=64) == 0  # a single 64-slot chunk is not split
    for bad in (dict(R=0), dict(N=0), dict(Hq=0), dict(Hkv=0), dict(D=0), dict(C=0),
                dict(Hq=30), dict(D=96), dict(N=1025), dict(scale=float("nan")),
                dict(scale=float("inf"))):
        assert ws(**bad) == 0, bad


def test_tree_attention_validation():
    f = P.lib().pctree_tree_attention
    need = P.lib().pctree_attention_workspace_bytes(ctypes.byref(_attn_shape()))

    def call(shape=None, ptrs=None, ws=A, nb=None):
        p = [A, A, A, A, A, A, A] if ptrs is None else ptrs
        return f(ctypes.byref(shape or _attn_shape()), *p, ws, need if nb is None else nb, None)

    assert f(None, A, A, A, A, A, A, A, A, need, None) == P.ERR_INVALID_ARGUMENT
    for i in range(7):
        p = [A] * 7
        p[i] = None
        assert call(ptrs=p) == P.ERR_INVALID_ARGUMENT, i
        p[i] = A + (8 if i in (0, 1, 2, 6) else 2)
        assert call(ptrs=p) == P.ERR_INVALID_ARGUMENT, i
    for kw in (dict(R=0), dict(Hq=12, Hkv=8), dict(scale=float("nan")), dict(C=-1),
               dict(scale=0.0), dict(scale=-0.125)):
        assert call(shape=_attn_shape(**kw)) == P.ERR_INVALID_ARGUMENT, kw
    for kw in (dict(D=96), dict(N=1025), dict(R=70000)):
        assert call(shape=_attn_shape(**kw)) == P.ERR_UNSUPPORTED, kw
    assert call(ws=None) == P.ERR_WORKSPACE
    assert call(ws=A + 64) == P.ERR_WORKSPACE
    assert call(nb=need - 1) == P.ERR_WORKSPACE
