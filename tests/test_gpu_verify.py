"""GPU parity of the verification bookkeeping (retrieve rows, greedy acceptance,
KV compaction) against the CPU oracle, through the C ABI.  All of it is
integer or byte work, so every output must match bit for bit."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import pctree_oracle as O
from oracle import pctree_verify as VO
from paper_2608_02123_amd.synth import (CONFIGS, make_inputs, make_kv_cache, random_tree,
                                        target_next)

pytestmark = pytest.mark.gpu


def _lib():
    from paper_2608_02123_amd import pctree as P
    return P


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def _batch(seed, R, N, max_depth, V, counts=None, accept_p=0.8):
    rng = np.random.default_rng((seed, 11))
    tok = np.full((R, N), -1, np.int32)
    par = np.full((R, N), -1, np.int32)
    tn = np.zeros((R, N), np.int32)
    cnt = np.zeros(R, np.int32)
    for i in range(R):
        room = sum(V ** d for d in range(max_depth + 1))
        c = int(rng.integers(0, N + 1)) if counts is None else counts[i]
        c = min(c, room)
        tok[i], par[i], _ = random_tree(rng, N, c, max_depth, V)
        tn[i] = target_next(rng, tok[i], par[i], c, V, accept_p)
        cnt[i] = c
    return tok, par, cnt, tn


def _check(tok, par, cnt, tn, max_depth):
    P = _lib()
    R, N = par.shape
    rows, nrows = P.build_retrieve(_dev(par), _dev(cnt), max_depth)
    acc = P.accept_greedy(_dev(tok), rows, nrows, _dev(tn))
    torch.cuda.synchronize()
    rows, nrows = rows.cpu().numpy(), nrows.cpu().numpy()
    acc = {k: v.cpu().numpy() for k, v in acc.items()}
    for i in range(R):
        want_rows, want_n = VO.retrieve_rows(par[i], int(cnt[i]), max_depth)
        assert nrows[i] == want_n, i
        assert np.array_equal(rows[i], want_rows), i
        a, j, nodes, b = VO.accept_greedy(tok[i], want_rows, want_n, tn[i])
        assert (acc["accept_len"][i], acc["accept_row"][i], acc["bonus"][i]) == (a, j, b), i
        assert np.array_equal(acc["accept_node"][i], nodes), i


@pytest.mark.parametrize("seed,R,N,max_depth,V,p", [
    (0, 8, 64, 16, 151936, 0.9),      # bench shape, high acceptance
    (1, 16, 128, 16, 50, 0.7),        # batched serving shape, small vocab
    (2, 3, 1024, 63, 7, 0.95),        # largest budget and depth
    (3, 5, 33, 4, 3, 0.5),            # ragged, shallow
    (4, 4, 1, 0, 10, 0.9),            # root only
])
def test_retrieve_accept_random(seed, R, N, max_depth, V, p):
    _check(*_batch(seed, R, N, max_depth, V, accept_p=p), max_depth)


def test_retrieve_accept_empty_and_full():
    tok, par, cnt, tn = _batch(5, 4, 40, 6, 9, counts=[0, 1, 40, 17])
    _check(tok, par, cnt, tn, 6)


def test_retrieve_accept_malformed():
    rng = np.random.default_rng(9)
    R, N, md = 6, 50, 5
    tok, par, cnt, tn = _batch(6, R, N, 12, 20, counts=[50, 50, 30, 50, 20, 50])
    par[0, 10] = 10          # self loop: not an edge
    par[1, 7] = 40           # forward index
    par[2, 3] = -5           # negative
    par[3, :] = np.clip(np.arange(N) - 1, -1, None)  # one path of 50 > max_depth + 1
    cnt[4] = 77              # count beyond N: clamped
    cnt[5] = -3              # negative count: empty
    tn[:] = np.where(rng.random((R, N)) < 0.5, tn, rng.integers(0, 20, (R, N)))
    _check(tok, par, cnt, tn, md)


def test_accept_rows_out_of_range():
    P = _lib()
    R, N, W = 2, 8, 4
    tok = np.arange(R * N, dtype=np.int32).reshape(R, N) % 5
    tn = np.roll(tok, -1, axis=1).astype(np.int32)
    rows = np.full((R, N, W), -1, np.int32)
    rows[0, 0] = [0, 1, 99, 3]     # 99 ends the row
    rows[0, 1] = [0, 1, 2, 3]
    rows[1, 0] = [-7, 1, 2, 3]     # bad head: row skipped
    rows[1, 1] = [0, 1, 2, -1]
    nrows = np.array([2, 5], np.int32)  # request 1 reads three all -1 rows
    acc = P.accept_greedy(_dev(tok), _dev(rows), _dev(nrows), _dev(tn))
    torch.cuda.synchronize()
    for i in range(R):
        a, j, nodes, b = VO.accept_greedy(tok[i], rows[i], int(nrows[i]), tn[i])
        assert acc["accept_len"][i].item() == a and acc["accept_row"][i].item() == j
        assert acc["bonus"][i].item() == b
        assert np.array_equal(acc["accept_node"][i].cpu().numpy(), nodes)


def test_end_to_end_tiny_round():
    """Tree from the builder, rows and acceptance on the device, against the
    oracle's own tree run through the verification oracle."""
    P = _lib()
    w = CONFIGS["tiny"]
    inp = make_inputs(w)
    d = P.device_inputs(inp)
    out = P.build_tree(d["L"], d["E"], d["Wt"], d["h"], d["root"], d["prefix_len"], w.k, w.N)
    ref = O.build_tree_batch(inp, w.k, w.N)[0]
    torch.cuda.synchronize()
    assert np.array_equal(out["token"][0].cpu().numpy(), ref["token"])
    assert np.array_equal(out["parent"][0].cpu().numpy(), ref["parent"])
    rng = np.random.default_rng(2)
    tn = target_next(rng, ref["token"], ref["parent"], ref["count"], w.V, 0.9)[None]
    rows, nrows = P.build_retrieve(out["parent"], out["count"], w.B)
    acc = P.accept_greedy(out["token"], rows, nrows, _dev(tn))
    torch.cuda.synchronize()
    want_rows, want_n = VO.retrieve_rows(ref["parent"], ref["count"], w.B)
    assert nrows[0].item() == want_n
    assert np.array_equal(rows[0].cpu().numpy(), want_rows)
    a, j, nodes, b = VO.accept_greedy(ref["token"], want_rows, want_n, tn[0])
    assert (acc["accept_len"][0].item(), acc["accept_row"][0].item(), acc["bonus"][0].item()) \
        == (a, j, b)
    assert np.array_equal(acc["accept_node"][0].cpu().numpy(), nodes)


@pytest.mark.parametrize("groups,width,R", [(72, 1024, 2), (3, 8, 5), (1, 2560, 3)])
def test_compact_kv(groups, width, R):
    """Qwen3-4B-like KV (36 layers x K/V, 8 heads x 128 dims, bf16), a tiny
    one, and a hidden-state-like single group."""
    P = _lib()
    rng = np.random.default_rng((groups, width))
    N, md = 64, 16
    tok, par, cnt, tn = _batch(7, R, N, md, 30, accept_p=0.95)
    rows = np.full((R, N, md + 1), -1, np.int32)
    nrows = np.zeros(R, np.int32)
    acc_len = np.zeros(R, np.int32)
    acc_node = np.full((R, md + 1), -1, np.int32)
    for i in range(R):
        rows[i], nrows[i] = VO.retrieve_rows(par[i], int(cnt[i]), md)
        acc_len[i], _, acc_node[i], _ = VO.accept_greedy(tok[i], rows[i], int(nrows[i]), tn[i])
    prefix = rng.integers(0, 100, R).astype(np.int32)
    cap = int(prefix.max()) + N + 3
    if R >= 3:
        acc_node[R - 1, 1] = acc_node[R - 1, 0]  # not increasing: left untouched
        acc_len[R - 1] = max(acc_len[R - 1], 1)
    cache = np.stack([make_kv_cache(rng, groups, cap, width) for _ in range(R)])
    d = _dev(cache.view(np.int16))
    P.compact_kv(d, _dev(prefix), _dev(acc_node), _dev(acc_len), N)
    torch.cuda.synchronize()
    got = d.cpu().numpy().view(np.uint16)
    for i in range(R):
        ok = all(acc_node[i, m] > (acc_node[i, m - 1] if m else -1)
                 for m in range(acc_len[i] + 1))
        for g in range(groups):
            want = (VO.compact_rows(cache[i, g], int(prefix[i]), acc_node[i], int(acc_len[i]))
                    if ok else cache[i, g])
            assert np.array_equal(got[i, g], want), (i, g)
