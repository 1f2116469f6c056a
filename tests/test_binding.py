"""CPU checks of the Python binding's argument checking (no GPU needed): every
input must have exactly the layout the shape describes before a launch, since
the kernels index the inputs by the shape alone."""
from __future__ import annotations

import ctypes

import pytest
import torch

from paper_2608_02123_amd import pctree as P

V, B, N, k, r, R = 300, 4, 16, 4, 32, 2


def tensors(dtype=torch.bfloat16):
    return {
        "L": torch.zeros(R, B, V, dtype=dtype),
        "E": torch.zeros(V, r, dtype=dtype),
        "Wt": torch.zeros(V, r, dtype=dtype),
        "h": torch.zeros(R, B, r, dtype=torch.float32),
        "root": torch.zeros(R, dtype=torch.int32),
        "prefix_len": torch.zeros(R, dtype=torch.int32),
    }


def check(shape_dtype=P.BF16, **override):
    t = tensors()
    t.update(override)
    P.check_inputs(P.make_shape(V, B, N, k, r, R, shape_dtype), **t, device=False)


def test_matching_inputs_pass():
    check()
    t = tensors(torch.float32)
    P.check_inputs(P.make_shape(V, B, N, k, r, R, P.F32), **t, device=False)


@pytest.mark.parametrize("name,bad", [
    ("L", torch.zeros(R, B, V - 1, dtype=torch.bfloat16)),      # shorter vocabulary
    ("L", torch.zeros(R - 1, B, V, dtype=torch.bfloat16)),      # fewer requests
    ("E", torch.zeros(V, r // 2, dtype=torch.bfloat16)),        # smaller rank
    ("Wt", torch.zeros(r, V, dtype=torch.bfloat16)),            # W not transposed
    ("h", torch.zeros(R, B - 1, r, dtype=torch.float32)),       # fewer depths
    ("root", torch.zeros(R + 1, dtype=torch.int32)),
    ("prefix_len", torch.zeros(1, dtype=torch.int32)),
])
def test_wrong_shapes_are_rejected(name, bad):
    with pytest.raises(ValueError, match=name):
        check(**{name: bad})


@pytest.mark.parametrize("name,bad", [
    ("L", torch.zeros(R, B, V, dtype=torch.float32)),           # f32 logits, bf16 builder
    ("E", torch.zeros(V, r, dtype=torch.float16)),
    ("h", torch.zeros(R, B, r, dtype=torch.bfloat16)),
    ("root", torch.zeros(R, dtype=torch.int64)),
    ("prefix_len", torch.zeros(R, dtype=torch.float32)),
])
def test_wrong_dtypes_are_rejected(name, bad):
    with pytest.raises(TypeError, match=name):
        check(**{name: bad})


def test_bf16_tensors_for_an_f32_builder_are_rejected():
    with pytest.raises(TypeError, match="L"):
        check(shape_dtype=P.F32)


def test_non_contiguous_and_host_tensors_are_rejected():
    with pytest.raises(ValueError, match="contiguous"):
        check(Wt=torch.zeros(r, V, dtype=torch.bfloat16).t())
    t = tensors()
    with pytest.raises(ValueError, match="device"):
        P.check_inputs(P.make_shape(V, B, N, k, r, R, P.BF16), **t, device=True)


def test_abandoned_counts_raise():
    P.check_counts(torch.tensor([3, 0, 16], dtype=torch.int32))
    with pytest.raises(P.RoundAborted) as e:
        P.check_counts(torch.tensor([3, -1, -1], dtype=torch.int32))
    assert e.value.requests == [1, 2]


def test_debug_set_validates_and_restores():
    bad = P.DebugConfig(-1, 0, -5, 0)
    assert P.lib().pctree_debug_set(ctypes.byref(bad)) == P.ERR_INVALID_ARGUMENT
    P.debug_set(wait_ticks=0, force_multilaunch=True, round_slices=7, wide_unbounded=True)
    assert P.lib().pctree_debug_set(None) == P.OK
    P.debug_set()
