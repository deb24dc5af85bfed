"""Thin ctypes binding of libstarkv.so (argument marshalling only).

Every function mirrors the C entry point of the same name in
include/starkv.h.  Tensors are PyTorch tensors that live on the GPU; the
binding passes their data pointers and the current HIP stream.  It checks
that buffers are large enough so that a wrong Python call fails here rather
than inside a kernel.  All compute happens in the library's HIP kernels; if
the library is not built, every call raises.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int32, c_int64, c_size_t, c_void_p, c_char_p

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libstarkv.so")

F32 = 0
BF16 = 1
TEM_DECAY = {"exp": 0, "linear": 1, "gamma": 2}     # starkv_tem_decay
AEB_MODE = {"entropy": 0, "confidence": 1}          # starkv_aeb_mode
MAX_SPANS = 64

STATUS = {
    0: "OK", 1: "E_NULL", 2: "E_SHAPE", 3: "E_BUDGET", 4: "E_SPANS",
    5: "E_PARAM", 6: "E_DTYPE", 7: "E_ALIGN", 8: "E_WORKSPACE", 9: "E_STATE",
    10: "E_HIP",
}


class Dims(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("H", c_int32), ("G", c_int32),
                ("d", c_int32), ("L", c_int32), ("W", c_int32),
                ("dtype", c_int32), ("per_head", c_int32)]

    @property
    def Lp(self) -> int:
        return self.L - self.W

    @property
    def Ns(self) -> int:
        """Scoring subspaces: one per KV group, or one per head."""
        return self.H if self.per_head else self.G


class KVLayout(ctypes.Structure):
    _fields_ = [("layer_stride", c_int64), ("group_stride", c_int64),
                ("token_stride", c_int64)]


class Params(ctypes.Structure):
    _fields_ = [("lam", c_float), ("n_warmup", c_int32), ("n_ramp", c_int32),
                ("rho_mi", c_float), ("tau", c_float), ("rho_t", c_float),
                ("delta", c_float), ("d_min", c_float), ("t_min", c_float),
                ("t_max", c_float), ("n_bins", c_int32), ("grid", c_int32),
                ("pool_kernel", c_int32), ("eps", c_float), ("tem_decay", c_int32),
                ("aeb_mode", c_int32)]


class Span(ctypes.Structure):
    _fields_ = [("start", c_int32), ("rows", c_int32), ("cols", c_int32),
                ("frame", c_int32)]


class StarKVError(RuntimeError):
    def __init__(self, fn: str, code: int):
        self.code = code
        self.name = STATUS.get(code, str(code))
        super().__init__(f"{fn} failed: STARKV_{self.name}")


_lib = None

# name -> (restype, argtypes)
SIGNATURES = {
    "starkv_abi_version": (c_int32, []),
    "starkv_status_str": (c_char_p, [c_int32]),
    "starkv_params_default": (None, [POINTER(Params)]),
    "starkv_workspace_bytes": (c_size_t, [POINTER(Dims)]),
    "starkv_scalars_count": (c_size_t, [POINTER(Dims)]),
    "starkv_state_bytes": (c_size_t, [POINTER(Dims), c_int32]),
    "starkv_state_init": (c_int32, [POINTER(Dims), c_void_p, c_int32, c_void_p]),
    "starkv_score": (c_int32, [POINTER(Dims), POINTER(Params), c_void_p, c_void_p,
                               POINTER(KVLayout), c_void_p, c_void_p, c_void_p,
                               c_void_p, c_size_t, c_void_p]),
    "starkv_score_noalloc": (c_int32, [POINTER(Dims), POINTER(Params), c_void_p, c_void_p,
                                       POINTER(KVLayout), c_void_p, c_void_p, c_void_p,
                                       c_void_p]),
    "starkv_update_state": (c_int32, [POINTER(Dims), POINTER(Params), c_void_p,
                                      c_void_p, POINTER(Span), c_int32, c_int32,
                                      c_void_p, c_int32, c_void_p, c_void_p,
                                      c_size_t, c_void_p]),
    "starkv_select": (c_int32, [POINTER(Dims), POINTER(Params), c_void_p, c_void_p,
                                c_void_p, POINTER(Span), c_int32, c_int32, c_int32,
                                c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "starkv_update_state_select": (c_int32, [POINTER(Dims), POINTER(Params), c_void_p,
                                             c_void_p, c_void_p, POINTER(Span), c_int32,
                                             c_int32, c_void_p, c_int32, c_void_p, c_int32,
                                             c_void_p, c_void_p, c_void_p, c_size_t,
                                             c_void_p]),
    "starkv_compact": (c_int32, [POINTER(Dims), c_void_p, c_void_p,
                                 POINTER(KVLayout), c_void_p, c_int32, c_void_p,
                                 c_void_p, c_void_p]),
    "starkv_decode_workspace_bytes": (c_size_t, [POINTER(Dims), c_int32]),
    "starkv_decode": (c_int32, [POINTER(Dims), c_void_p, c_void_p, c_void_p,
                                POINTER(KVLayout), c_int32, c_void_p, c_void_p, c_size_t,
                                c_void_p]),
}


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                "(there is no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(fn: str, code: int):
    if code != 0:
        raise StarKVError(fn, code)


# ------------------------------------------------------------------ helpers

def make_dims(n_layers, H, G, d, L, W, dtype, per_head=False) -> Dims:
    return Dims(n_layers, H, G, d, L, W, dtype, 1 if per_head else 0)


def params_default() -> Params:
    p = Params()
    lib().starkv_params_default(ctypes.byref(p))
    return p


def workspace_bytes(dims: Dims) -> int:
    return int(lib().starkv_workspace_bytes(ctypes.byref(dims)))


def scalars_count(dims: Dims) -> int:
    return int(lib().starkv_scalars_count(ctypes.byref(dims)))


def state_bytes(dims: Dims, frame_cap: int) -> int:
    return int(lib().starkv_state_bytes(ctypes.byref(dims), frame_cap))


def spans_array(spans):
    """[(start, rows, cols, frame), ...] -> ctypes array (or None)."""
    if not spans:
        return None, 0
    arr = (Span * len(spans))(*[Span(*map(int, s)) for s in spans])
    return arr, len(spans)


def contiguous_layout(t, dims: Dims) -> KVLayout:
    """Layout of a cache tensor shaped [n_layers, G, L_cap, d] (any strides
    with a unit last stride)."""
    assert t.dim() == 4 and t.stride(3) == 1
    return KVLayout(t.stride(0), t.stride(1), t.stride(2))


def _stream(stream):
    """A hipStream_t handle: a torch stream, a raw handle, or None for the
    current torch stream."""
    if stream is not None:
        return c_void_p(getattr(stream, "cuda_stream", stream))
    import torch
    return c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return c_void_p(t.data_ptr()) if t is not None else c_void_p(0)


def _need(t, nbytes, what):
    if t is None:
        return
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{what}: {have} bytes < {nbytes} required")
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")


def _esz(dims):
    return 4 if dims.dtype == F32 else 2


def _need_cache(t, dims, lay, what):
    """The strided cache view must lie inside the tensor's storage."""
    if t is None:
        return
    last = ((dims.n_layers - 1) * lay.layer_stride + (dims.G - 1) * lay.group_stride
            + (dims.L - 1) * lay.token_stride + dims.d)
    _need(t, last * _esz(dims), what)


# ------------------------------------------------------------------ entry points

def state_init(dims: Dims, state, frame_cap: int, stream=None):
    _need(state, state_bytes(dims, frame_cap), "state")
    _check("starkv_state_init", lib().starkv_state_init(
        ctypes.byref(dims), _ptr(state), frame_cap, _stream(stream)))


def score(dims: Dims, params: Params, q, k, k_layout: KVLayout, S, sbar, gstar,
          ws, stream=None):
    nl, Lp = dims.n_layers, dims.Lp
    _need(q, nl * dims.H * dims.W * dims.d * _esz(dims), "q")
    _need_cache(k, dims, k_layout, "k")
    _need(S, nl * dims.Ns * Lp * 4, "S")
    _need(sbar, nl * Lp * 4, "sbar")
    _need(gstar, nl * Lp, "gstar")
    _need(ws, workspace_bytes(dims), "ws")
    _check("starkv_score", lib().starkv_score(
        ctypes.byref(dims), ctypes.byref(params), _ptr(q), _ptr(k),
        ctypes.byref(k_layout), _ptr(S), _ptr(sbar), _ptr(gstar), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def score_noalloc(dims: Dims, params: Params, q, k, k_layout: KVLayout, S, sbar, gstar,
                  stream=None):
    """starkv_score with the library's own device workspace (no ws)."""
    nl, Lp = dims.n_layers, dims.Lp
    _need(q, nl * dims.H * dims.W * dims.d * _esz(dims), "q")
    _need_cache(k, dims, k_layout, "k")
    _need(S, nl * dims.Ns * Lp * 4, "S")
    _need(sbar, nl * Lp * 4, "sbar")
    _need(gstar, nl * Lp, "gstar")
    _check("starkv_score_noalloc", lib().starkv_score_noalloc(
        ctypes.byref(dims), ctypes.byref(params), _ptr(q), _ptr(k),
        ctypes.byref(k_layout), _ptr(S), _ptr(sbar), _ptr(gstar), _stream(stream)))


def update_state(dims: Dims, params: Params, S, sbar, spans, frame: int, state,
                 frame_cap: int, scalars, ws=None, stream=None):
    arr, n = spans_array(spans)
    _need(S, dims.n_layers * dims.Ns * dims.Lp * 4, "S")
    _need(sbar, dims.n_layers * dims.Lp * 4, "sbar")
    _need(scalars, dims.n_layers * scalars_count(dims) * 4, "scalars")
    _need(state, state_bytes(dims, frame_cap), "state")
    _check("starkv_update_state", lib().starkv_update_state(
        ctypes.byref(dims), ctypes.byref(params), _ptr(S), _ptr(sbar), arr, n,
        frame, _ptr(state), frame_cap, _ptr(scalars), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def select(dims: Dims, params: Params, sbar, gstar, scalars, spans, frame: int,
           B: int, s, idx, ws=None, stream=None):
    arr, n = spans_array(spans)
    _need(sbar, dims.n_layers * dims.Lp * 4, "sbar")
    _need(gstar, dims.n_layers * dims.Lp, "gstar")
    _need(scalars, dims.n_layers * scalars_count(dims) * 4, "scalars")
    _need(s, dims.n_layers * dims.Lp * 4, "s")
    if B > 0:
        _need(idx, dims.n_layers * B * 4, "idx")
    _check("starkv_select", lib().starkv_select(
        ctypes.byref(dims), ctypes.byref(params), _ptr(sbar), _ptr(gstar),
        _ptr(scalars), arr, n, frame, B, _ptr(s), _ptr(idx), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def update_state_select(dims: Dims, params: Params, S, sbar, gstar, spans, frame: int,
                        state, frame_cap: int, scalars, B: int, s, idx, ws=None,
                        stream=None):
    arr, n = spans_array(spans)
    _need(S, dims.n_layers * dims.Ns * dims.Lp * 4, "S")
    _need(sbar, dims.n_layers * dims.Lp * 4, "sbar")
    _need(gstar, dims.n_layers * dims.Lp, "gstar")
    _need(scalars, dims.n_layers * scalars_count(dims) * 4, "scalars")
    _need(state, state_bytes(dims, frame_cap), "state")
    _need(s, dims.n_layers * dims.Lp * 4, "s")
    if B > 0:
        _need(idx, dims.n_layers * B * 4, "idx")
    _check("starkv_update_state_select", lib().starkv_update_state_select(
        ctypes.byref(dims), ctypes.byref(params), _ptr(S), _ptr(sbar), _ptr(gstar), arr, n,
        frame, _ptr(state), frame_cap, _ptr(scalars), B, _ptr(s), _ptr(idx), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def compact(dims: Dims, k, v, kv_layout: KVLayout, idx, B: int, k_out, v_out,
            stream=None):
    nbytes = dims.n_layers * dims.G * (B + dims.W) * dims.d * _esz(dims)
    _need_cache(k, dims, kv_layout, "k")
    _need_cache(v, dims, kv_layout, "v")
    if B > 0:
        _need(idx, dims.n_layers * B * 4, "idx")
    _need(k_out, nbytes, "k_out")
    _need(v_out, nbytes, "v_out")
    _check("starkv_compact", lib().starkv_compact(
        ctypes.byref(dims), _ptr(k), _ptr(v), ctypes.byref(kv_layout), _ptr(idx),
        B, _ptr(k_out), _ptr(v_out), _stream(stream)))


def decode_workspace_bytes(dims: Dims, n_tokens: int) -> int:
    return int(lib().starkv_decode_workspace_bytes(ctypes.byref(dims), n_tokens))


def decode(dims: Dims, q, k, v, kv_layout: KVLayout, n_tokens: int, out, ws, stream=None):
    """Decode attention of one token per head over n_tokens cached tokens."""
    nl = dims.n_layers
    _need(q, nl * dims.H * dims.d * _esz(dims), "q")
    last = ((nl - 1) * kv_layout.layer_stride + (dims.G - 1) * kv_layout.group_stride
            + (n_tokens - 1) * kv_layout.token_stride + dims.d)
    _need(k, last * _esz(dims), "k")
    _need(v, last * _esz(dims), "v")
    _need(out, nl * dims.H * dims.d * 4, "out")
    _need(ws, decode_workspace_bytes(dims, n_tokens), "ws")
    _check("starkv_decode", lib().starkv_decode(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), ctypes.byref(kv_layout), n_tokens,
        _ptr(out), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
