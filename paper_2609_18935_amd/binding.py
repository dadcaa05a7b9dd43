"""Python binding of libtailupdate.so (argument marshalling only).

Every step of the update runs in the HIP library; this module only turns torch
device tensors into pointers, keeps the host metadata of each context in the
C structs the library reads and writes, and raises on non-zero status. PyTorch
is used for device memory and streams.

If the shared library is missing the import fails loudly: there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# TU_LIBRARY may name another build of the same library (e.g. one with host-side
# sanitizers for the host tests)
LIB_PATH = os.environ.get("TU_LIBRARY") or os.path.join(_HERE, "libtailupdate.so")

TU_OK = 0
TU_ERR_ARG = -1
TU_ERR_RANGE = -2
TU_ERR_CAPACITY = -3
TU_ERR_WORKSPACE = -4
TU_ERR_HIP = -5
TU_LAYER_ATTN = 0
TU_LAYER_DELTA = 1
TU_MAX_RANGES = 128
TU_MAX_PLACE_RUNS = 32
TU_PLACE_TAIL = 0
TU_PLACE_SLOT = 1
TU_PLACE_RELOCATE = 2
_PLACEMENTS = {"tail": TU_PLACE_TAIL, "slot": TU_PLACE_SLOT, "relocate": TU_PLACE_RELOCATE}

_i32, _i64, _f32, _f64, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double, ctypes.c_void_p


class tu_interval(ctypes.Structure):
    _fields_ = [("begin", _i64), ("end", _i64)]


class tu_seq(ctypes.Structure):
    _fields_ = [("len", _i64), ("capacity", _i64), ("next_pos", _i64),
                ("live", ctypes.POINTER(tu_interval)), ("n_live", _i32), ("live_cap", _i32),
                ("d_pos", _vp), ("vt_rows", _i64)]


class tu_attn_params(ctypes.Structure):
    _fields_ = [("n_q_heads", _i32), ("n_kv_heads", _i32), ("head_dim", _i32), ("rotary_dim", _i32),
                ("rope_theta", _f64), ("softmax_scale", _f32), ("kv_splits", _i32)]


class tu_delta_params(ctypes.Structure):
    _fields_ = [("n_k_heads", _i32), ("n_v_heads", _i32), ("d_k", _i32), ("d_v", _i32), ("chunk", _i32),
                ("scale", _f32)]


class tu_seq_update(ctypes.Structure):
    _fields_ = [("seq", ctypes.POINTER(tu_seq)), ("ranges", ctypes.POINTER(_i64)), ("n_ranges", _i32),
                ("T", _i64), ("src_index", _vp), ("post_ranges", ctypes.POINTER(_i64)), ("n_post_ranges", _i32),
                ("placement", _i32), ("place_runs", ctypes.POINTER(_i64)), ("n_place_runs", _i32)]


class tu_layer_io(ctypes.Structure):
    _fields_ = [("kind", _i32), ("k_cache", ctypes.POINTER(_vp)), ("v_cache", ctypes.POINTER(_vp)),
                ("vt_cache", ctypes.POINTER(_vp)), ("state", ctypes.POINTER(_vp)), ("q", _vp), ("k", _vp), ("v", _vp), ("beta", _vp), ("g", _vp),
                ("out", _vp)]


class tu_conv_tensor(ctypes.Structure):
    _fields_ = [("state", _vp), ("x", _vp), ("weight", _vp), ("out", _vp), ("T", _i64), ("channels", _i32),
                ("reserved", _i32)]


class tu_update(ctypes.Structure):
    _fields_ = [("n_seq", _i32), ("seqs", ctypes.POINTER(tu_seq_update)), ("n_layers", _i32),
                ("layers", ctypes.POINTER(tu_layer_io)), ("attn", tu_attn_params), ("delta", tu_delta_params)]


# exported symbols and their signatures (mirrors include/tailupdate.h)
_SIGNATURES = {
    "tu_abi_version": (_i32, []),
    "tu_last_error": (ctypes.c_char_p, []),
    "tu_validate_ranges": (_i32, [ctypes.POINTER(tu_seq), ctypes.POINTER(_i64), _i32, ctypes.POINTER(_i64)]),
    "compact_kv_workspace_size": (ctypes.c_size_t, [_i64, _i32, _i32, _i32]),
    "compact_kv": (_i32, [ctypes.POINTER(tu_seq), ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _i32, _i32,
                          ctypes.POINTER(_i64), _i32, _vp, _vp, ctypes.c_size_t, _vp]),
    "compact_kv_noalloc": (_i32, [ctypes.POINTER(tu_seq), ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _i32, _i32,
                                  ctypes.POINTER(_i64), _i32, _vp, _vp, _vp]),
    "tail_prefill_attention_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(tu_attn_params), _i64, _i64]),
    "tu_vt_cache_bytes": (ctypes.c_size_t, [_i64, _i32, _i32]),
    "refresh_vt_cache": (_i32, [ctypes.POINTER(tu_seq), ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _i32, _i32,
                                _vp, ctypes.c_size_t, _vp]),
    "tail_prefill_attention": (_i32, [ctypes.POINTER(tu_seq), _vp, _vp, _vp, ctypes.POINTER(tu_attn_params), _vp,
                                      _vp, _vp, _i64, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "commit_tail": (_i32, [ctypes.POINTER(tu_seq), _i64]),
    "delta_rule_continue_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(tu_delta_params), _i64]),
    "delta_rule_continue": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i64, ctypes.POINTER(tu_delta_params), _vp, _vp,
                                   ctypes.c_size_t, _vp]),
    "short_conv_continue": (_i32, [_vp, _vp, _vp, _i64, _i32, _i32, _i32, _vp, _vp]),
    "short_conv_continue_batch": (_i32, [ctypes.POINTER(tu_conv_tensor), _i32, _i32, _i32, _vp]),
    "update_layer_stack_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(tu_update)]),
    "tu_validate_update": (_i32, [ctypes.POINTER(tu_update)]),
    "update_layer_stack": (_i32, [ctypes.POINTER(tu_update), _vp, ctypes.c_size_t, _vp]),
    "relocate_keys": (_i32, [ctypes.POINTER(tu_seq), ctypes.POINTER(_vp), _i32, ctypes.POINTER(tu_attn_params),
                             ctypes.POINTER(_i64), _i32, _vp]),
    "attention_probe_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(tu_attn_params), _i64, _i32]),
    "attention_probe": (_i32, [ctypes.POINTER(tu_seq), _vp, ctypes.POINTER(tu_attn_params), _vp, _i32, _f32, _vp,
                               _vp, ctypes.c_size_t, _vp]),
    "attention_group_mass_workspace_size": (ctypes.c_size_t, [_i64, _i32]),
    "attention_group_mass": (_i32, [ctypes.POINTER(tu_seq), _vp, ctypes.POINTER(_i64), _i32, _i32, _vp, _vp, _vp,
                                    _vp, ctypes.c_size_t, _vp]),
    "attention_tv_workspace_size": (ctypes.c_size_t, [_i64]),
    "attention_tv_distance": (_i32, [_vp, _vp, _vp, _i64, _vp, _vp, ctypes.c_size_t, _vp]),
    "tu_workspace_faults": (_i32, [_vp, ctypes.POINTER(_i32), _vp]),
    "tu_profile_enable": (_i32, [_i32]),
    "tu_profile_collect": (_i32, [ctypes.c_char_p, _i32, ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_double),
                                  _i32]),
}

_lib_handle = None
ABI_VERSION = 5   # TU_ABI_VERSION of include/tailupdate.h that these structures follow


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_18935_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        if h.tu_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {h.tu_abi_version()}, this binding expects {ABI_VERSION}:"
                               " rebuild it")
        _lib_handle = h
    return _lib_handle


class TailUpdateError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[{code}] {message}")
        self.code = code


def _check(code: int):
    if code != TU_OK:
        raise TailUpdateError(code, lib().tu_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        # NULL is the default stream; torch's current stream when a GPU is present
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _torch_stream(stream, device):
    """The torch stream object a call runs on (None: the current stream)."""
    if stream is None:
        return None
    if isinstance(stream, torch.cuda.Stream):
        return stream
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    return torch.cuda.ExternalStream(handle, device=device)


def _workspace(nbytes: int, device, workspace: Optional[torch.Tensor], stream=None) -> torch.Tensor:
    """The caller's workspace, or a new one. A new one is freed when the call returns,
    while its kernels may still run on `stream`: when that is not the current stream,
    the allocation is recorded on it, so that the caching allocator does not hand the
    memory to another tensor before those kernels are done."""
    if workspace is not None:
        return workspace
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    ts = _torch_stream(stream, device)
    if ts is not None and ts != torch.cuda.current_stream(device):
        ws.record_stream(ts)
    return ws


def _ranges_array(ranges, width: int = 2) -> tuple:
    import numpy as np
    r = np.ascontiguousarray(np.asarray(ranges, dtype=np.int64).reshape(-1, width))
    arr = (_i64 * max(1, r.size))(*r.reshape(-1).tolist())
    return arr, int(r.shape[0])


# ----------------------------------------------------------------------------- parameters

def attn_params(n_q_heads: int, n_kv_heads: int, head_dim: int, rotary_dim: Optional[int] = None,
                rope_theta: float = 1.0e7, softmax_scale: Optional[float] = None, kv_splits: int = 0):
    return tu_attn_params(n_q_heads, n_kv_heads, head_dim, head_dim if rotary_dim is None else rotary_dim,
                          float(rope_theta), float(head_dim ** -0.5 if softmax_scale is None else softmax_scale),
                          int(kv_splits))


def delta_params(n_k_heads: int, n_v_heads: int, d_k: int, d_v: int, chunk: int, scale: Optional[float] = None):
    return tu_delta_params(n_k_heads, n_v_heads, d_k, d_v, chunk, float(d_k ** -0.5 if scale is None else scale))


# ----------------------------------------------------------------------------- contexts

class Context:
    """A character context: host metadata (tu_seq) plus the device position array.

    The caller owns the K/V caches of every attention layer ([capacity][Hkv][D]
    bf16) and the fp32 states of every delta layer.
    """

    def __init__(self, capacity: int, device="cuda", live_cap: int = 4096):
        self.pos = torch.zeros(max(1, capacity), dtype=torch.int32, device=device)
        self._live = (tu_interval * live_cap)()
        self.c = tu_seq(0, int(capacity), 0, self._live, 0, int(live_cap), self.pos.data_ptr(), 0)

    @property
    def len(self) -> int:
        return int(self.c.len)

    @property
    def capacity(self) -> int:
        return int(self.c.capacity)

    @property
    def next_pos(self) -> int:
        return int(self.c.next_pos)

    @property
    def vt_rows(self) -> int:
        return int(self.c.vt_rows)

    def intervals(self) -> List[tuple]:
        return [(int(self._live[i].begin), int(self._live[i].end)) for i in range(self.c.n_live)]

    def set_metadata(self, intervals: Sequence[tuple], next_pos: int, vt_rows: int = 0):
        """Declare the live positions of a cache the caller filled (pos must match);
        vt_rows: rows of the layers' V^T copies that hold those rows (0: none)."""
        if len(intervals) > self.c.live_cap:
            raise ValueError("too many intervals")
        n = 0
        for i, (a, b) in enumerate(intervals):
            self._live[i] = tu_interval(int(a), int(b))
            n += int(b) - int(a)
        self.c.n_live = len(intervals)
        self.c.len = n
        self.c.next_pos = int(next_pos)
        self.c.vt_rows = int(vt_rows)

    def snapshot(self):
        """The context's metadata and positions (Section 4.1 state apart from the caches
        and recurrent states, which the caller owns and copies itself)."""
        return (self.intervals(), self.next_pos, self.pos.clone(), self.vt_rows)

    def restore(self, snap):
        iv, nxt, pos, vt_rows = snap
        self.pos.copy_(pos)
        self.set_metadata(iv, nxt, vt_rows)

    def validate_ranges(self, ranges) -> int:
        arr, n = _ranges_array(ranges)
        removed = _i64(0)
        _check(lib().tu_validate_ranges(ctypes.byref(self.c), arr, n, ctypes.byref(removed)))
        return int(removed.value)


# ----------------------------------------------------------------------------- entry points

def compact_kv(ctx: Context, k_layers: Sequence[torch.Tensor], v_layers: Sequence[torch.Tensor], ranges,
               src_index: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None, stream=None):
    n = len(k_layers)
    Hkv, D = int(k_layers[0].shape[1]), int(k_layers[0].shape[2])
    ks = (_vp * max(1, n))(*[_ptr(t) for t in k_layers])
    vs = (_vp * max(1, n))(*[_ptr(t) for t in v_layers])
    arr, nr = _ranges_array(ranges)
    nbytes = lib().compact_kv_workspace_size(ctx.len, n, Hkv, D)
    ws = _workspace(nbytes, ctx.pos.device, workspace, stream)
    _check(lib().compact_kv(ctypes.byref(ctx.c), ks, vs, n, Hkv, D, arr, nr, _ptr(src_index), _ptr(ws),
                            ws.numel(), _stream(stream)))
    return ws


TU_NOALLOC_SCRATCH_BYTES = 8 << 20


def compact_kv_noalloc(ctx: Context, k_layers: Sequence[torch.Tensor], v_layers: Sequence[torch.Tensor], ranges,
                       src_index: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None, stream=None):
    """compact_kv with its scratch in the library's fixed per-GPU array (no allocation);
    `status` (256 bytes on the device, optional) receives the call's device checks."""
    n = len(k_layers)
    Hkv, D = int(k_layers[0].shape[1]), int(k_layers[0].shape[2])
    ks = (_vp * max(1, n))(*[_ptr(t) for t in k_layers])
    vs = (_vp * max(1, n))(*[_ptr(t) for t in v_layers])
    arr, nr = _ranges_array(ranges)
    _check(lib().compact_kv_noalloc(ctypes.byref(ctx.c), ks, vs, n, Hkv, D, arr, nr, _ptr(src_index), _ptr(status),
                                    _stream(stream)))


def vt_cache_bytes(capacity: int, n_kv_heads: int, head_dim: int) -> int:
    return int(lib().tu_vt_cache_bytes(int(capacity), int(n_kv_heads), int(head_dim)))


def new_vt_cache(capacity: int, n_kv_heads: int, head_dim: int, device="cuda") -> torch.Tensor:
    """A V^T copy for one attention layer of a context of `capacity` rows (its contents
    start stale: the context's vt_rows says how many rows are current)."""
    return torch.empty(vt_cache_bytes(capacity, n_kv_heads, head_dim), dtype=torch.uint8, device=device)


def refresh_vt_cache(ctx: Context, v_layers: Sequence[torch.Tensor], vt_layers: Sequence[torch.Tensor],
                     workspace: Optional[torch.Tensor] = None, stream=None):
    """Pack rows [ctx.vt_rows, ctx.len) of each value cache into its V^T copy; then
    ctx.vt_rows == ctx.len. Returns the (status) workspace."""
    n = len(v_layers)
    Hkv, D = int(v_layers[0].shape[1]), int(v_layers[0].shape[2])
    vs = (_vp * max(1, n))(*[_ptr(t) for t in v_layers])
    ts = (_vp * max(1, n))(*[_ptr(t) for t in vt_layers])
    ws = _workspace(256, ctx.pos.device, workspace, stream)
    _check(lib().refresh_vt_cache(ctypes.byref(ctx.c), vs, ts, n, Hkv, D, _ptr(ws), ws.numel(), _stream(stream)))
    return ws


def tail_prefill_attention(ctx: Context, k_cache: torch.Tensor, v_cache: torch.Tensor, params: tu_attn_params,
                           q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, out: torch.Tensor,
                           q_hat: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                           stream=None, vt_cache: Optional[torch.Tensor] = None):
    T = int(q.shape[0])
    nbytes = lib().tail_prefill_attention_workspace_size(ctypes.byref(params), T, ctx.len)
    ws = _workspace(nbytes, q.device, workspace, stream)
    _check(lib().tail_prefill_attention(ctypes.byref(ctx.c), _ptr(k_cache), _ptr(v_cache), _ptr(vt_cache),
                                        ctypes.byref(params), _ptr(q), _ptr(k), _ptr(v), T, _ptr(out), _ptr(q_hat),
                                        _ptr(ws), ws.numel(), _stream(stream)))
    return ws


def commit_tail(ctx: Context, T: int):
    _check(lib().commit_tail(ctypes.byref(ctx.c), int(T)))


def delta_rule_continue(state: torch.Tensor, q, k, v, beta, g, params: tu_delta_params, out: torch.Tensor,
                        workspace: Optional[torch.Tensor] = None, stream=None):
    T = int(q.shape[0])
    nbytes = lib().delta_rule_continue_workspace_size(ctypes.byref(params), T)
    ws = _workspace(nbytes, state.device, workspace, stream)
    _check(lib().delta_rule_continue(_ptr(state), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(g), T,
                                     ctypes.byref(params), _ptr(out), _ptr(ws), ws.numel(), _stream(stream)))
    return ws


def relocate_keys(ctx: Context, k_layers: Sequence[torch.Tensor], params: Optional[tu_attn_params], moves,
                  stream=None):
    """Rotate the stored keys of the rows holding each move's source positions
    [src_begin, src_end) to dst_begin + offset and relabel them; moves: [n][3]."""
    n = len(k_layers)
    ks = (_vp * max(1, n))(*[_ptr(t) for t in k_layers])
    arr, nm = _ranges_array(moves, 3)
    p = params if params is not None else tu_attn_params()
    _check(lib().relocate_keys(ctypes.byref(ctx.c), ks, n, ctypes.byref(p), arr, nm, _stream(stream)))


def attention_probe(ctx: Context, k_cache: torch.Tensor, params: tu_attn_params, q: torch.Tensor,
                    probs: torch.Tensor, weight: float = 1.0, workspace: Optional[torch.Tensor] = None, stream=None):
    """probs[:len] += weight * the fp32 reference-softmax distribution of the last
    q.shape[0] rows' queries (raw q [n][Hq][D]) over the rows they see, averaged over
    those queries and all heads."""
    n = int(q.shape[0])
    nbytes = lib().attention_probe_workspace_size(ctypes.byref(params), ctx.len, n)
    ws = _workspace(nbytes, q.device, workspace, stream)
    _check(lib().attention_probe(ctypes.byref(ctx.c), _ptr(k_cache), ctypes.byref(params), _ptr(q), n, float(weight),
                                 _ptr(probs), _ptr(ws), ws.numel(), _stream(stream)))


def attention_group_mass(ctx: Context, probs: torch.Tensor, groups, window: int = 8,
                         workspace: Optional[torch.Tensor] = None, stream=None):
    """Memory-group masses of a token distribution: returns device tensors (mass [m],
    window mass [m], summary [3] = memory mass, effective group count, window share)."""
    arr, m = _ranges_array(groups)
    mass = torch.empty(max(1, m), dtype=torch.float32, device=probs.device)
    win = torch.empty_like(mass)
    summary = torch.empty(3, dtype=torch.float32, device=probs.device)
    ws = _workspace(lib().attention_group_mass_workspace_size(ctx.len, m), probs.device, workspace, stream)
    _check(lib().attention_group_mass(ctypes.byref(ctx.c), _ptr(probs), arr, m, int(window), _ptr(mass), _ptr(win),
                                      _ptr(summary), _ptr(ws), ws.numel(), _stream(stream)))
    return mass[:m], win[:m], summary


def attention_tv_distance(p: torch.Tensor, q: torch.Tensor, q_row_of_p: Optional[torch.Tensor] = None,
                          workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """0.5 * sum |p - q[map]| as a device fp32 tensor [1]."""
    n = int(p.numel())
    tv = torch.empty(1, dtype=torch.float32, device=p.device)
    ws = _workspace(lib().attention_tv_workspace_size(n), p.device, workspace, stream)
    _check(lib().attention_tv_distance(_ptr(p), _ptr(q), _ptr(q_row_of_p), n, _ptr(tv), _ptr(ws), ws.numel(),
                                       _stream(stream)))
    return tv


TU_CONV_IDENTITY = 0
TU_CONV_SILU = 1


def short_conv_continue(state: Optional[torch.Tensor], x: torch.Tensor, weight: torch.Tensor, out: torch.Tensor,
                        activation: str = "silu", stream=None):
    """Short causal convolution of x [T][C] continued from state [W-1][C] (updated in
    place); weight [C][W]; out [T][C]; all bf16 on the device."""
    T, C = int(x.shape[0]), int(x.shape[1])
    W = int(weight.shape[1])
    act = {"silu": TU_CONV_SILU, "none": TU_CONV_IDENTITY}[activation]
    _check(lib().short_conv_continue(_ptr(state), _ptr(x), _ptr(weight), T, C, W, act, _ptr(out), _stream(stream)))


def short_conv_continue_batch(items, activation: str = "silu", stream=None):
    """items: sequence of (state, x, weight, out) tensors sharing one width (see
    short_conv_continue); all are continued in as few launches as possible."""
    arr = (tu_conv_tensor * max(1, len(items)))()
    W = None
    for i, (st, x, w, out) in enumerate(items):
        if W is not None and int(w.shape[1]) != W:
            raise ValueError("all tensors of a batch share one width")
        W = int(w.shape[1])
        arr[i] = tu_conv_tensor(_ptr(st), _ptr(x), _ptr(w), _ptr(out), int(x.shape[0]), int(x.shape[1]), 0)
    act = {"silu": TU_CONV_SILU, "none": TU_CONV_IDENTITY}[activation]
    _check(lib().short_conv_continue_batch(arr, len(items), W or 1, act, _stream(stream)))


class LayerIO:
    """Inputs and outputs of one layer of a stack update (tail rows packed over contexts)."""

    def __init__(self, kind: int, q, k, v, out, k_cache=None, v_cache=None, state=None, beta=None, g=None,
                 vt_cache=None):
        self.kind = kind
        self.q, self.k, self.v, self.out = q, k, v, out
        self.k_cache, self.v_cache, self.state = k_cache, v_cache, state
        self.vt_cache = vt_cache   # per context: a V^T copy (new_vt_cache) or None
        self.beta, self.g = beta, g


class StackUpdate:
    """A prepared update_layer_stack call (ctypes structs built once, reusable)."""

    def __init__(self, contexts: Sequence[Context], ranges: Sequence, tails: Sequence[int], layers: Sequence[LayerIO],
                 attn: Optional[tu_attn_params] = None, delta: Optional[tu_delta_params] = None,
                 src_index: Optional[Sequence[Optional[torch.Tensor]]] = None, post_ranges: Optional[Sequence] = None,
                 placement: Optional[Sequence[str]] = None, place_runs: Optional[Sequence] = None):
        """post_ranges[s]: position ranges made of context s's tail positions whose rows
        are removed once the tail is prefilled (maintenance delimiters), or None.
        placement[s]: "tail" (default), "slot" or "relocate"; place_runs[s]: the [n][2]
        position runs the tail takes for "slot" and "relocate"."""
        n = len(contexts)
        self.contexts = list(contexts)
        self._keep = []
        self._seq_arr = (tu_seq_update * max(1, n))()
        for s, ctx in enumerate(contexts):
            arr, nr = _ranges_array(ranges[s])
            self._keep.append(arr)
            si = None if src_index is None else src_index[s]
            pr = None if post_ranges is None or post_ranges[s] is None else post_ranges[s]
            parr, npr = _ranges_array(pr if pr is not None else [])
            self._keep.append(parr)
            pl = "tail" if placement is None or placement[s] is None else placement[s]
            runs = None if place_runs is None or place_runs[s] is None else place_runs[s]
            rarr, nrr = _ranges_array(runs if runs is not None else [])
            self._keep.append(rarr)
            self._seq_arr[s] = tu_seq_update(ctypes.pointer(ctx.c), arr, nr, int(tails[s]), _ptr(si), parr, npr,
                                             _PLACEMENTS[pl], rarr, nrr)
        self._layer_arr = (tu_layer_io * max(1, len(layers)))()
        for l, L in enumerate(layers):
            def plist(ts):
                if ts is None:
                    return None
                a = (_vp * max(1, n))(*[_ptr(t) for t in ts])
                self._keep.append(a)
                return a
            self._layer_arr[l] = tu_layer_io(L.kind, plist(L.k_cache), plist(L.v_cache),
                                             plist(getattr(L, "vt_cache", None)), plist(L.state), _ptr(L.q),
                                             _ptr(L.k), _ptr(L.v), _ptr(L.beta), _ptr(L.g), _ptr(L.out))
        self.u = tu_update(n, self._seq_arr, len(layers), self._layer_arr,
                           attn if attn is not None else tu_attn_params(),
                           delta if delta is not None else tu_delta_params())

    def validate(self):
        _check(lib().tu_validate_update(ctypes.byref(self.u)))

    def workspace_size(self) -> int:
        n = lib().update_layer_stack_workspace_size(ctypes.byref(self.u))
        if n == 0:
            self.validate()
        return int(n)

    def run(self, workspace: torch.Tensor, stream=None):
        _check(lib().update_layer_stack(ctypes.byref(self.u), _ptr(workspace), workspace.numel(), _stream(stream)))


TU_FAULT_POSITIONS = 1   # device positions disagreed with the host's live runs
TU_FAULT_WAIT = 2        # a bounded wait of the in-place move expired
TU_FAULT_RANGE = 4       # a value rounded to f16 overflowed


def workspace_faults(workspace: torch.Tensor, stream=None) -> int:
    """The device-check bits (TU_FAULT_*) of the last call that ran with `workspace`
    (on `stream`); synchronises `stream`."""
    out = ctypes.c_int32(0)
    _check(lib().tu_workspace_faults(_ptr(workspace), ctypes.byref(out), _stream(stream)))
    return int(out.value)


def profile_enable(on: bool = True):
    """Bracket every library kernel launch of this thread with HIP events on its stream."""
    _check(lib().tu_profile_enable(1 if on else 0))


def profile_collect(max_entries: int = 32) -> dict:
    """{kernel name: (launch count, summed milliseconds)} since the last collect."""
    stride = 64
    names = ctypes.create_string_buffer(stride * max_entries)
    counts = (_i32 * max_entries)()
    totals = (ctypes.c_double * max_entries)()
    n = lib().tu_profile_collect(names, stride, counts, totals, max_entries)
    if n < 0:
        _check(n)
    raw = names.raw
    out = {}
    for i in range(n):
        name = raw[i * stride:(i + 1) * stride].split(b"\0", 1)[0].decode()
        out[name] = (int(counts[i]), float(totals[i]))
    return out


def update_layer_stack(contexts, ranges, tails, layers, attn=None, delta=None, workspace=None, stream=None,
                       src_index=None, post_ranges=None, placement=None, place_runs=None):
    up = StackUpdate(contexts, ranges, tails, layers, attn, delta, src_index, post_ranges, placement, place_runs)
    nbytes = up.workspace_size()
    dev = contexts[0].pos.device if contexts else "cuda"
    ws = _workspace(nbytes, dev, workspace, stream)
    up.run(ws, stream)
    up.workspace = ws
    return up
