"""pctree_build_tree_noalloc (the entry point for callers that cannot
allocate) against pctree_build_tree, through the C ABI.

Both run the same kernels; only the workspace differs (the library's fixed
per-device array instead of the caller's buffer), so the outputs must be
identical bit for bit.  Calls in a row share the array: the second and third
calls use smaller inputs than the one before, so that whatever the previous
call left in the array is still there when the next one starts.
"""
from __future__ import annotations

import ctypes

import pytest
import torch

from paper_2608_02123_amd import pctree as P
from paper_2608_02123_amd.synth import CONFIGS, make_inputs


def say(msg):
    print(msg, flush=True)


KEYS = ("token", "parent", "depth", "position", "logprob", "count", "mask",
        "trace_token", "trace_parent_slot", "trace_score")


@pytest.mark.gpu
def test_noalloc_matches_the_workspace_entry_point():
    # largest workspace first: the 8-request Qwen3-14B round (per-stage
    # launches, 10.6 MiB), then the Qwen3-4B block of 16 (one persistent
    # launch, 6 MiB), then the small fp32 workload
    for name in ("qwen14b_b16_r8", "qwen4b_b16", "tiny"):
        w = CONFIGS[name]
        dt = P.BF16 if w.dtype == "bf16" else P.F32
        need = P.workspace_bytes(w.V, w.B, w.N, w.k, w.r, w.R, dt)
        assert 0 < need <= P.NOALLOC_SCRATCH_BYTES
        say(f"[noalloc] {name}: workspace {need / 2**20:.1f} MiB")
        dev = P.device_inputs(make_inputs(w))
        b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, dt, mask=True, trace=True,
                          workspace=False)
        for call in range(2):  # twice: the second finds the first's scratch contents
            got = {k: v.clone() for k, v in b.run_noalloc(**dev, check=True).items()}
            torch.cuda.synchronize()
            ref_b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, dt, mask=True, trace=True)
            ref_b.workspace.fill_(0xA5)
            ref = ref_b.run(**dev, check=True)
            torch.cuda.synchronize()
            for key in KEYS:
                assert torch.equal(got[key], ref[key]), f"{name} call {call}: {key} differs"
            say(f"[noalloc] {name} call {call}: identical to pctree_build_tree")


def test_noalloc_rejects_shapes_past_its_array():
    """Host-side check, before any device work: a workspace need larger than
    PCTREE_NOALLOC_SCRATCH_BYTES is PCTREE_ERR_WORKSPACE."""
    big = P.make_shape(1 << 20, 63, 256, 16, 512, 256, P.BF16)
    assert P.lib().pctree_workspace_bytes(ctypes.byref(big)) > P.NOALLOC_SCRATCH_BYTES
    fake = 0x100000
    inp = P._Inputs(*(fake + 0x1000 * i for i in range(6)))
    tree = P._Tree(*(fake + 0x100000 + 0x1000 * i for i in range(7)))
    st = P.lib().pctree_build_tree_noalloc(ctypes.byref(big), ctypes.byref(inp),
                                           ctypes.byref(tree), None, None)
    assert st == P.ERR_WORKSPACE
    bad = P.make_shape(0, 4, 16, 4, 32, 1, P.BF16)
    st = P.lib().pctree_build_tree_noalloc(ctypes.byref(bad), ctypes.byref(inp),
                                           ctypes.byref(tree), None, None)
    assert st == P.ERR_INVALID_ARGUMENT
