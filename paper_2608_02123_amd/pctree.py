"""Python binding of ``libpctree.so`` (the C ABI declared in include/pctree.h).

Argument marshalling only: every step of a round runs in the library's HIP
kernels.  torch supplies device memory and the current HIP stream.  If the
library has not been built this module raises; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "PCTreeError",
    "RoundAborted",
    "lib",
    "Shape",
    "workspace_bytes",
    "build_tree",
    "build_mask",
    "chain_decode",
    "build_retrieve",
    "accept_greedy",
    "compact_kv",
    "AttnShape",
    "attention_workspace_bytes",
    "tree_attention",
    "TreeAttention",
    "TreeBuilder",
    "timeline_available",
    "timeline_read",
    "status_string",
    "DebugConfig",
    "debug_set",
    "F32",
    "BF16",
    "MODE_PARENT",
    "MODE_SHARED",
    "MODE_INDEPENDENT",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
# (PCTREE_LIB: another build of the same library, e.g. the host-sanitizer one)
LIB_PATH = os.environ.get("PCTREE_LIB") or os.path.join(_HERE, "libpctree.so")
# the stage-timeline build of the same library (include/pctree_profile.h)
TIMELINE_LIB_PATH = os.path.join(_HERE, "libpctree_timeline.so")
TIMELINE_WHO, TIMELINE_STAGES, TIMELINE_EVENTS = 5, 65, 8

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
F32, BF16 = 0, 1
NOALLOC_SCRATCH_BYTES = 32 << 20  # PCTREE_NOALLOC_SCRATCH_BYTES
MODE_PARENT, MODE_SHARED, MODE_INDEPENDENT = 0, 1, 2  # pctree_mode


class PCTreeError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)}")
        self.status = status


class RoundAborted(RuntimeError):
    """A round was abandoned on the device (count = -1, every row padded)."""

    def __init__(self, requests):
        super().__init__(f"round abandoned for requests {list(requests)} (count = -1): a "
                         "workgroup of the single-launch round did not start in time")
        self.requests = list(requests)


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("vocab", "block", "budget", "topk", "rank", "requests", "dtype", "mode")]


class AttnShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("requests", "budget", "q_heads", "kv_heads", "head_dim", "capacity")] + \
               [("scale", ctypes.c_float)]


class _Inputs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("base_logits", "emb", "proj_t", "depth_feat", "root_token", "prefix_len")]


class _Tree(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("token", "parent", "depth", "position", "logprob", "count", "mask")]


class _Trace(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("token", "parent_slot", "score")]


class DebugConfig(ctypes.Structure):
    """pctree_debug_config of include/pctree_profile.h (test-only launch overrides)."""
    _fields_ = [("wait_ticks", ctypes.c_int64), ("force_multilaunch", ctypes.c_int32),
                ("round_slices", ctypes.c_int32), ("wide_unbounded", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; "
                "g.build()'` (the HIP library is required; there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz = ctypes.c_void_p, ctypes.c_size_t
        L.pctree_workspace_bytes.argtypes = [ctypes.POINTER(Shape)]
        L.pctree_workspace_bytes.restype = sz
        L.pctree_build_tree.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(_Inputs),
                                        ctypes.POINTER(_Tree), ctypes.POINTER(_Trace), vp, sz, vp]
        L.pctree_build_tree.restype = ctypes.c_int
        L.pctree_build_tree_noalloc.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(_Inputs),
                                                ctypes.POINTER(_Tree), ctypes.POINTER(_Trace), vp]
        L.pctree_build_tree_noalloc.restype = ctypes.c_int
        L.pctree_build_mask.argtypes = [vp, vp, ctypes.c_int32, ctypes.c_int32, vp, vp]
        L.pctree_build_mask.restype = ctypes.c_int
        L.pctree_chain_decode.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(_Inputs), vp, vp,
                                          vp, sz, vp]
        L.pctree_chain_decode.restype = ctypes.c_int
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        L.pctree_build_retrieve.argtypes = [vp, vp, i32, i32, i32, vp, vp, vp]
        L.pctree_build_retrieve.restype = ctypes.c_int
        L.pctree_accept_greedy.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp, vp]
        L.pctree_accept_greedy.restype = ctypes.c_int
        L.pctree_compact_kv.argtypes = [vp, i64, i64, i32, i32, i32, vp, vp, vp, i32, i32, i32,
                                        vp]
        L.pctree_compact_kv.restype = ctypes.c_int
        L.pctree_attention_workspace_bytes.argtypes = [ctypes.POINTER(AttnShape)]
        L.pctree_attention_workspace_bytes.restype = sz
        L.pctree_tree_attention.argtypes = [ctypes.POINTER(AttnShape), vp, vp, vp, vp, vp, vp, vp,
                                            vp, sz, vp]
        L.pctree_tree_attention.restype = ctypes.c_int
        L.pctree_status_string.argtypes = [ctypes.c_int]
        L.pctree_status_string.restype = ctypes.c_char_p
        L.pctree_abi_version.argtypes = []
        L.pctree_abi_version.restype = ctypes.c_int32
        L.pctree_profile_enable.argtypes = [ctypes.c_int32]
        L.pctree_profile_enable.restype = ctypes.c_int
        L.pctree_profile_read.argtypes = [ctypes.POINTER(ctypes.c_double),
                                          ctypes.POINTER(ctypes.c_int64),
                                          ctypes.POINTER(ctypes.c_char_p)]
        L.pctree_profile_read.restype = ctypes.c_int
        L.pctree_debug_set.argtypes = [ctypes.POINTER(DebugConfig)]
        L.pctree_debug_set.restype = ctypes.c_int
        L.pctree_timeline_available.argtypes = []
        L.pctree_timeline_available.restype = ctypes.c_int32
        L.pctree_timeline_read.argtypes = [vp, ctypes.POINTER(ctypes.c_double)]
        L.pctree_timeline_read.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().pctree_status_string(status).decode()


def _check(status: int, what: str) -> None:
    if status != OK:
        raise PCTreeError(status, what)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}: float32 or bfloat16 expected")


def make_shape(V, B, N, k, r, R, dtype, mode=0) -> Shape:
    return Shape(V, B, N, k, r, R, dtype, mode)


def workspace_bytes(V, B, N, k, r, R=1, dtype=BF16) -> int:
    return int(lib().pctree_workspace_bytes(ctypes.byref(make_shape(V, B, N, k, r, R, dtype))))


_TORCH_DTYPE = {F32: torch.float32, BF16: torch.bfloat16}


def check_inputs(shape: Shape, L, E, Wt, h, root, prefix_len, *, device=True) -> None:
    """Raise unless every input has exactly the layout ``shape`` describes:
    ``L [R][B][V]``, ``E [V][r]`` and ``Wt [V][r]`` in the shape's dtype,
    ``h [R][B][r]`` float32, ``root [R]`` and ``prefix_len [R]`` int32, all
    contiguous (and on a GPU when ``device``).  The kernels index these
    tensors by the shape alone, so a smaller tensor would be read past its end.
    """
    V, B, r, R = shape.vocab, shape.block, shape.rank, shape.requests
    want = {
        "L": (L, (R, B, V), _TORCH_DTYPE.get(shape.dtype)),
        "E": (E, (V, r), _TORCH_DTYPE.get(shape.dtype)),
        "Wt": (Wt, (V, r), _TORCH_DTYPE.get(shape.dtype)),
        "h": (h, (R, B, r), torch.float32),
        "root": (root, (R,), torch.int32),
        "prefix_len": (prefix_len, (R,), torch.int32),
    }
    for name, (t, shp, dt) in want.items():
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
        if dt is None or t.dtype != dt:
            raise TypeError(f"{name} must be {dt}, got {t.dtype}")
        if tuple(t.shape) != shp:
            raise ValueError(f"{name} must have shape {shp}, got {tuple(t.shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if device and not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")


def _inputs(shape, L, E, Wt, h, root, prefix_len):
    check_inputs(shape, L, E, Wt, h, root, prefix_len)
    return _Inputs(*(t.data_ptr() for t in (L, E, Wt, h, root, prefix_len)))


def check_counts(count) -> None:
    """Raise RoundAborted if a request's count is -1 (waits for the stream)."""
    c = count.cpu()
    bad = (c == -1).nonzero().flatten().tolist()
    if bad:
        raise RoundAborted(bad)


class TreeBuilder:
    """Pre-allocated outputs and workspace for repeated rounds of one shape.

    ``run(L, E, Wt, h, root, prefix_len)`` enqueues one round on the current
    stream and returns the output tensors (overwritten by the next call).
    With ``check=True`` it then waits for the round and raises
    :class:`RoundAborted` if the device abandoned it (count = -1).
    """

    def __init__(self, V, B, N, k, r, R=1, dtype=BF16, device="cuda", mask=True, trace=False,
                 mode=MODE_PARENT, workspace=True):
        self.shape = make_shape(V, B, N, k, r, R, dtype, mode)
        nbytes = int(lib().pctree_workspace_bytes(ctypes.byref(self.shape)))
        if nbytes == 0:
            _check(lib().pctree_build_tree(ctypes.byref(self.shape), None, None, None, None, 0,
                                           None), "shape")
        # workspace=False: only run_noalloc() (the library's own scratch array)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device) if workspace \
            else None
        i32 = dict(dtype=torch.int32, device=device)
        self.out = {
            "token": torch.empty(R, N, **i32),
            "parent": torch.empty(R, N, **i32),
            "depth": torch.empty(R, N, **i32),
            "position": torch.empty(R, N, **i32),
            "logprob": torch.empty(R, N, dtype=torch.float32, device=device),
            "count": torch.empty(R, **i32),
        }
        if mask:
            self.out["mask"] = torch.empty(R, N, (N + 31) // 32, **i32)
        self._tree = _Tree(*(self.out[n].data_ptr() for n in
                             ("token", "parent", "depth", "position", "logprob", "count")),
                           self.out["mask"].data_ptr() if mask else None)
        self._trace = None
        if trace:
            self.out["trace_token"] = torch.empty(R, B, k, **i32)
            self.out["trace_parent_slot"] = torch.empty(R, B, k, **i32)
            self.out["trace_score"] = torch.empty(R, B, k, dtype=torch.float32, device=device)
            self._trace = _Trace(self.out["trace_token"].data_ptr(),
                                 self.out["trace_parent_slot"].data_ptr(),
                                 self.out["trace_score"].data_ptr())

    def run(self, L, E, Wt, h, root, prefix_len, stream=None, check=False):
        self.bind(L, E, Wt, h, root, prefix_len)
        return self.launch(stream, check=check)

    def bind(self, L, E, Wt, h, root, prefix_len):
        """Check and remember the inputs once; ``launch()`` then only enqueues."""
        self._inp = _inputs(self.shape, L, E, Wt, h, root, prefix_len)
        self._keep = (L, E, Wt, h, root, prefix_len)
        self._args = (ctypes.byref(self.shape), ctypes.byref(self._inp), ctypes.byref(self._tree),
                      ctypes.byref(self._trace) if self._trace is not None else None)

    def launch(self, stream=None, check=False):
        if self.workspace is None:
            raise RuntimeError("this builder has no workspace: use run_noalloc()")
        st = lib().pctree_build_tree(*self._args, ctypes.c_void_p(self.workspace.data_ptr()),
                                     self.workspace.numel(), _stream(stream))
        _check(st, "pctree_build_tree")
        if check:
            check_counts(self.out["count"])
        return self.out

    def run_noalloc(self, L, E, Wt, h, root, prefix_len, stream=None, check=False):
        """The same round through pctree_build_tree_noalloc: no workspace
        argument, the library's fixed per-device scratch array instead."""
        self.bind(L, E, Wt, h, root, prefix_len)
        st = lib().pctree_build_tree_noalloc(*self._args, _stream(stream))
        _check(st, "pctree_build_tree_noalloc")
        if check:
            check_counts(self.out["count"])
        return self.out


def build_tree(L, E, Wt, h, root, prefix_len, k, N, *, mask=True, trace=False, stream=None,
               mode=MODE_PARENT, check=True):
    """One round for tensors ``L [R][B][V]``, ``E [V][r]``, ``Wt [V][r]``, ``h [R][B][r]``.

    Returns a dict of freshly allocated output tensors (see include/pctree.h).
    With ``check`` (the default) it waits for the round and raises
    :class:`RoundAborted` if the device abandoned it.
    """
    R, B, V = L.shape
    r = E.shape[1]
    b = TreeBuilder(V, B, N, k, r, R, _dtype_code(L), device=L.device, mask=mask, trace=trace,
                    mode=mode)
    return b.run(L, E, Wt, h, root, prefix_len, stream=stream, check=check)


def debug_set(wait_ticks: int = -1, force_multilaunch: bool = False,
              round_slices: int = 0, wide_unbounded: bool = False) -> None:
    """Test-only launch overrides (pctree_debug_set); no arguments restores the defaults."""
    cfg = DebugConfig(int(wait_ticks), 1 if force_multilaunch else 0, int(round_slices),
                      1 if wide_unbounded else 0)
    _check(lib().pctree_debug_set(ctypes.byref(cfg)), "pctree_debug_set")


def profile_enable(on: bool = True) -> None:
    """Bracket the dominant kernel's launches with hipEvents (include/pctree_profile.h)."""
    _check(lib().pctree_profile_enable(1 if on else 0), "pctree_profile_enable")


def profile_read():
    """(total milliseconds, launches, kernel name) recorded since enabling; clears them."""
    ms, n, name = ctypes.c_double(), ctypes.c_int64(), ctypes.c_char_p()
    _check(lib().pctree_profile_read(ctypes.byref(ms), ctypes.byref(n), ctypes.byref(name)),
           "pctree_profile_read")
    return ms.value, n.value, name.value.decode()


def timeline_available() -> bool:
    """Whether the loaded library is the stage-timeline build."""
    return bool(lib().pctree_timeline_available())


def timeline_read():
    """The stage timeline's stamps in microseconds, as a float64 array
    [who][stage][event] (NaN where not stamped), zeroing them
    (pctree_timeline_read; waits for the current device first)."""
    import numpy as np

    torch.cuda.synchronize()
    n = TIMELINE_WHO * TIMELINE_STAGES * TIMELINE_EVENTS
    buf = (ctypes.c_int64 * n)()
    rate = ctypes.c_double()
    _check(lib().pctree_timeline_read(ctypes.cast(buf, ctypes.c_void_p), ctypes.byref(rate)),
           "pctree_timeline_read")
    ticks = np.frombuffer(buf, dtype=np.int64).reshape(TIMELINE_WHO, TIMELINE_STAGES,
                                                       TIMELINE_EVENTS)
    return np.where(ticks > 0, ticks / rate.value, np.nan)


def build_mask(parent, count, stream=None):
    """Ancestor mask ``[R][N][ceil(N/32)]`` (int32 view of uint32 words)."""
    if parent.dtype != torch.int32 or count.dtype != torch.int32:
        raise TypeError("parent and count must be int32")
    if not (parent.is_cuda and count.is_cuda and parent.is_contiguous()):
        raise ValueError("parent and count must be contiguous device tensors")
    R, N = parent.shape
    mask = torch.empty(R, N, (N + 31) // 32, dtype=torch.int32, device=parent.device)
    st = lib().pctree_build_mask(_ptr(parent), _ptr(count), R, N, _ptr(mask), _stream(stream))
    _check(st, "pctree_build_mask")
    return mask


def chain_decode(L, E, Wt, h, root, prefix_len=None, stream=None, mode=MODE_PARENT):
    """The greedy chain of Eq. 1: returns (tokens [R][B+1], cumulative logprobs [R][B+1])."""
    R, B, V = L.shape
    r = E.shape[1]
    if prefix_len is None:
        prefix_len = torch.zeros(R, dtype=torch.int32, device=L.device)
    shape = make_shape(V, B, 1, 1, r, R, _dtype_code(L), mode)
    nbytes = int(lib().pctree_workspace_bytes(ctypes.byref(shape)))
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=L.device)
    toks = torch.empty(R, B + 1, dtype=torch.int32, device=L.device)
    lps = torch.empty(R, B + 1, dtype=torch.float32, device=L.device)
    inp = _inputs(shape, L, E, Wt, h, root, prefix_len)
    st = lib().pctree_chain_decode(ctypes.byref(shape), ctypes.byref(inp), _ptr(toks), _ptr(lps),
                                   ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(stream))
    _check(st, "pctree_chain_decode")
    return toks, lps


def _int32_dev(name, t):
    if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous int32 device tensor")


def build_retrieve(parent, count, max_depth, stream=None):
    """Retrieve rows of emitted trees: (rows [R][N][max_depth+1], nrows [R]) int32."""
    _int32_dev("parent", parent)
    _int32_dev("count", count)
    R, N = parent.shape
    rows = torch.empty(R, N, max_depth + 1, dtype=torch.int32, device=parent.device)
    nrows = torch.empty(R, dtype=torch.int32, device=parent.device)
    st = lib().pctree_build_retrieve(_ptr(parent), _ptr(count), R, N, max_depth, _ptr(rows),
                                     _ptr(nrows), _stream(stream))
    _check(st, "pctree_build_retrieve")
    return rows, nrows


def accept_greedy(token, rows, nrows, target_next, stream=None):
    """Greedy tree acceptance over retrieve rows; returns a dict of int32 tensors
    ``accept_len [R]``, ``accept_row [R]``, ``accept_node [R][W]``, ``bonus [R]``."""
    for name, t in (("token", token), ("rows", rows), ("nrows", nrows),
                    ("target_next", target_next)):
        _int32_dev(name, t)
    R, N, W = rows.shape
    if tuple(token.shape) != (R, N) or tuple(target_next.shape) != (R, N):
        raise ValueError("token and target_next must be [R][N] like the rows")
    i32 = dict(dtype=torch.int32, device=rows.device)
    out = {"accept_len": torch.empty(R, **i32), "accept_row": torch.empty(R, **i32),
           "accept_node": torch.empty(R, W, **i32), "bonus": torch.empty(R, **i32)}
    st = lib().pctree_accept_greedy(_ptr(token), _ptr(rows), _ptr(nrows), _ptr(target_next), R, N,
                                    W - 1, _ptr(out["accept_len"]), _ptr(out["accept_row"]),
                                    _ptr(out["accept_node"]), _ptr(out["bonus"]), _stream(stream))
    _check(st, "pctree_accept_greedy")
    return out


def compact_kv(cache, prefix_len, accept_node, accept_len, budget, stream=None):
    """Move each request's accepted cache slots right after its prefix, in place.

    ``cache [R][groups][capacity][...]`` is any contiguous device tensor whose
    trailing dimensions form one slot (a multiple of 16 bytes).
    """
    if not cache.is_cuda or not cache.is_contiguous() or cache.dim() < 3:
        raise ValueError("cache must be a contiguous [R][groups][capacity][...] device tensor")
    for name, t in (("prefix_len", prefix_len), ("accept_node", accept_node),
                    ("accept_len", accept_len)):
        _int32_dev(name, t)
    R, G, T = cache.shape[:3]
    es = cache.element_size()
    slot = cache[0, 0, 0].numel() * es
    st = lib().pctree_compact_kv(_ptr(cache), cache.stride(0) * es, cache.stride(1) * es, G, T,
                                 slot, _ptr(prefix_len), _ptr(accept_node), _ptr(accept_len), R,
                                 budget, accept_node.shape[1] - 1, _stream(stream))
    _check(st, "pctree_compact_kv")
    return cache


def attention_workspace_bytes(R, N, Hq, Hkv, D, C, scale=None) -> int:
    sc = float(scale) if scale is not None else D ** -0.5
    return int(lib().pctree_attention_workspace_bytes(ctypes.byref(
        AttnShape(R, N, Hq, Hkv, D, C, sc))))


class TreeAttention:
    """One tree-attention layer shape with its workspace, for repeated calls."""

    def __init__(self, R, N, Hq, Hkv, D, C, scale=None, device="cuda"):
        self.shape = AttnShape(R, N, Hq, Hkv, D, C,
                               float(scale) if scale is not None else D ** -0.5)
        nb = int(lib().pctree_attention_workspace_bytes(ctypes.byref(self.shape)))
        self.workspace = torch.empty(max(nb, 1), dtype=torch.uint8, device=device)
        self.ws_bytes = nb
        self.device = device

    def __call__(self, q, k, v, mask, count, prefix_len, out=None, stream=None):
        s = self.shape
        R, N, Hq, Hkv, D, C = s.requests, s.budget, s.q_heads, s.kv_heads, s.head_dim, s.capacity
        for name, t, shp in (("q", q, (R, N, Hq, D)), ("k", k, (R, Hkv, C, D)),
                             ("v", v, (R, Hkv, C, D))):
            if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() \
                    or tuple(t.shape) != shp:
                raise ValueError(f"{name} must be a contiguous bf16 device tensor {shp}")
        if mask.dtype != torch.int32 and mask.dtype != torch.uint32:
            raise TypeError("mask must be the [R][N][(N+31)/32] words of build_mask")
        if tuple(mask.shape) != (R, N, (N + 31) // 32) or not mask.is_contiguous() \
                or not mask.is_cuda:
            raise ValueError("mask must be [R][N][(N+31)/32] and contiguous")
        _int32_dev("count", count)
        _int32_dev("prefix_len", prefix_len)
        if out is None:
            out = torch.empty(R, N, Hq, D, dtype=torch.bfloat16, device=q.device)
        st = lib().pctree_tree_attention(ctypes.byref(s), _ptr(q), _ptr(k), _ptr(v), _ptr(mask),
                                         _ptr(count), _ptr(prefix_len), _ptr(out),
                                         _ptr(self.workspace), self.ws_bytes, _stream(stream))
        _check(st, "pctree_tree_attention")
        return out


def tree_attention(q, k, v, mask, count, prefix_len, scale=None, stream=None):
    """Tree-masked attention of one target layer: q [R][N][Hq][D], k and v
    [R][Hkv][C][D] bf16, mask from ``build_mask``; returns out [R][N][Hq][D] bf16."""
    R, N, Hq, D = q.shape
    Hkv, C = k.shape[1], k.shape[2]
    return TreeAttention(R, N, Hq, Hkv, D, C, scale, device=q.device)(
        q, k, v, mask, count, prefix_len, stream=stream)


def device_inputs(inp: dict, device="cuda") -> dict:
    """Upload one round's host inputs (the dict returned by ``synth.make_inputs``).

    The head matrix is stored transposed, ``Wt [V][r]`` (each token's rank
    vector contiguous, the same layout as ``E``); this packing is done once,
    when the drafter's weights are loaded, not per round.
    """
    import numpy as np

    dt = torch.bfloat16 if inp["workload"].dtype == "bf16" else torch.float32

    def up(a, dtype):
        return torch.from_numpy(np.ascontiguousarray(a)).to(device=device).to(dtype)

    return {
        "L": up(inp["L"], dt),
        "E": up(inp["E"], dt),
        "Wt": up(inp["W"].T, dt),
        "h": up(inp["h"], torch.float32),
        "root": up(inp["root"], torch.int32),
        "prefix_len": up(inp["prefix_len"], torch.int32),
    }
