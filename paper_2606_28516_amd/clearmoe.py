"""Python binding of the CLEAR-MoE C ABI (``include/clearmoe.h``).

Argument marshalling only: every step of the layer runs in the HIP library
``libclearmoe.so``.  PyTorch supplies device memory and the current stream.
There is no fallback: if the library is missing or a call fails, an
exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

__all__ = ["ClearMoEError", "Shape", "lib", "version", "workspace_bytes", "alloc_workspace",
           "route", "dispatch", "combine", "ffn_forward", "from_stored", "to_stored",
           "DISPATCH_HIST_IN_WS", "F32", "BF16", "SYMBOLS", "N_STAGES", "stage_names",
           "timing_start", "timing_stop", "make_shape", "dense_ffn_forward",
           "padded_workspace_bytes", "ffn_forward_padded", "ffn_forward_noalloc",
           "StackLayer", "make_stack_layer", "stack_shape", "stack_workspace_bytes",
           "stack_forward", "Router", "make_router", "route_ex",
           "ffn_forward_ex"]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libclearmoe.so")
F32, BF16 = 0, 1
DISPATCH_HIST_IN_WS = 1
SYMBOLS = ("clearmoe_version", "clearmoe_source_digest", "clearmoe_status_string", "clearmoe_workspace_bytes",
           "clearmoe_route", "clearmoe_dispatch", "clearmoe_combine", "clearmoe_ffn_forward",
           "clearmoe_dense_ffn_forward", "clearmoe_stage_name", "clearmoe_timing_start",
           "clearmoe_timing_start_sampled", "clearmoe_timing_stop", "clearmoe_padded_workspace_bytes",
           "clearmoe_ffn_forward_padded", "clearmoe_route_ex", "clearmoe_ffn_forward_ex",
           "clearmoe_ffn_forward_noalloc", "clearmoe_stack_workspace_bytes",
           "clearmoe_stack_forward")
NOALLOC_SCRATCH_BYTES = 64 << 20
ERR_TOO_LARGE = 5
N_STAGES = 20


class ClearMoEError(RuntimeError):
    pass


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("T", "D", "H", "E", "k", "r", "q", "dtype", "renorm")]


class Router(ctypes.Structure):
    """clearmoe_router: scores (linear, or an MLP with `hidden` units) and the
    selection rule (top-k, or adaptive top-1 / top-2 at threshold tau)."""
    _fields_ = [("Wg", ctypes.c_void_p), ("bg", ctypes.c_void_p), ("Wh", ctypes.c_void_p),
                ("bh", ctypes.c_void_p), ("W2", ctypes.c_void_p), ("hidden", ctypes.c_int32),
                ("adaptive", ctypes.c_int32), ("dense_stride", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("tau", ctypes.c_double)]


class StackLayer(ctypes.Structure):
    """clearmoe_stack_layer: a dense FFN (moe = 0) or a CLEAR-MoE layer
    (moe = 1, k experts per token, with its router)."""
    _fields_ = [("moe", ctypes.c_int32), ("k", ctypes.c_int32), ("W1", ctypes.c_void_p),
                ("b1", ctypes.c_void_p), ("US", ctypes.c_void_p), ("Vt", ctypes.c_void_p),
                ("b2", ctypes.c_void_p), ("P", ctypes.c_void_p), ("Q", ctypes.c_void_p),
                ("W2", ctypes.c_void_p), ("router", Router)]


_lib = None


def lib():
    """Load the in-tree library.  It is built first when it is missing or was
    built from other sources than the ones in the tree (the library carries
    the digest of its sources)."""
    global _lib
    if _lib is None:
        from . import build as _build
        want = _build.source_digest()
        have = _build.built_digest(LIB_PATH)
        if have != want:
            import sys
            print(f"clearmoe: library {'missing' if not have else 'stale (' + have + ')'}, "
                  f"building for sources {want}", file=sys.stderr)
            _build.build()
            if _build.built_digest(LIB_PATH) != want:
                raise ClearMoEError("the rebuilt library does not carry the source digest")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz, u32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_uint
        sp = ctypes.POINTER(Shape)
        L.clearmoe_version.restype = ctypes.c_int
        L.clearmoe_source_digest.restype = ctypes.c_char_p
        L.clearmoe_status_string.restype = ctypes.c_char_p
        L.clearmoe_status_string.argtypes = [ctypes.c_int]
        L.clearmoe_workspace_bytes.restype = sz
        L.clearmoe_workspace_bytes.argtypes = [sp]
        L.clearmoe_route.restype = ctypes.c_int
        L.clearmoe_route.argtypes = [sp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.clearmoe_dispatch.restype = ctypes.c_int
        L.clearmoe_dispatch.argtypes = [sp, vp, vp, sz, vp, vp, vp, vp, vp, vp, u32, vp]
        L.clearmoe_combine.restype = ctypes.c_int
        L.clearmoe_combine.argtypes = [sp, vp, vp, vp, vp, vp]
        L.clearmoe_ffn_forward.restype = ctypes.c_int
        L.clearmoe_ffn_forward.argtypes = [sp] + [vp] * 13 + [vp, sz, vp]
        rp = ctypes.POINTER(Router)
        L.clearmoe_route_ex.restype = ctypes.c_int
        L.clearmoe_route_ex.argtypes = [sp, rp, vp, vp, vp, vp, sz, vp]
        L.clearmoe_ffn_forward_ex.restype = ctypes.c_int
        L.clearmoe_ffn_forward_ex.argtypes = [sp, rp] + [vp] * 11 + [vp, sz, vp]
        L.clearmoe_padded_workspace_bytes.restype = sz
        L.clearmoe_padded_workspace_bytes.argtypes = [sp]
        L.clearmoe_ffn_forward_padded.restype = ctypes.c_int
        L.clearmoe_ffn_forward_padded.argtypes = [sp] + [vp] * 13 + [vp, sz, vp]
        L.clearmoe_ffn_forward_noalloc.restype = ctypes.c_int
        L.clearmoe_ffn_forward_noalloc.argtypes = [sp] + [vp] * 13 + [vp]
        lp = ctypes.POINTER(StackLayer)
        L.clearmoe_stack_workspace_bytes.restype = sz
        L.clearmoe_stack_workspace_bytes.argtypes = [sp, lp, ctypes.c_int32]
        L.clearmoe_stack_forward.restype = ctypes.c_int
        L.clearmoe_stack_forward.argtypes = [sp, lp, ctypes.c_int32, ctypes.c_int32, vp, vp, vp, sz,
                                             vp]
        L.clearmoe_dense_ffn_forward.restype = ctypes.c_int
        L.clearmoe_dense_ffn_forward.argtypes = [sp] + [vp] * 6 + [vp, sz, vp]
        L.clearmoe_stage_name.restype = ctypes.c_char_p
        L.clearmoe_stage_name.argtypes = [ctypes.c_int]
        L.clearmoe_timing_start.restype = ctypes.c_int
        L.clearmoe_timing_start.argtypes = [u32, ctypes.c_int]
        L.clearmoe_timing_start_sampled.restype = ctypes.c_int
        L.clearmoe_timing_start_sampled.argtypes = [u32, ctypes.c_int, ctypes.c_int]
        L.clearmoe_timing_stop.restype = ctypes.c_int
        L.clearmoe_timing_stop.argtypes = [ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_int32)]
        _lib = L
    return _lib


def version() -> int:
    return lib().clearmoe_version()


def _check(rc: int, what: str) -> None:
    if rc != 0:
        msg = lib().clearmoe_status_string(rc).decode()
        raise ClearMoEError(f"{what}: {msg} (status {rc})")


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise ClearMoEError(f"unsupported dtype {t.dtype}")


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ClearMoEError("tensor is not on the GPU")
    if not t.is_contiguous():
        raise ClearMoEError("tensor is not contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def make_shape(T, D, E, k, dtype, H=0, r=0, q=0, renorm=1) -> Shape:
    """renorm = 1: the top-k gates renormalised over the selected experts;
    0: their probabilities under the softmax over all E."""
    return Shape(int(T), int(D), int(H), int(E), int(k), int(r), int(q), int(dtype), int(renorm))


def workspace_bytes(shape: Shape) -> int:
    return int(lib().clearmoe_workspace_bytes(ctypes.byref(shape)))


def alloc_workspace(shape: Shape, device="cuda") -> torch.Tensor:
    n = workspace_bytes(shape)
    if n == 0:
        raise ClearMoEError("invalid shape")
    return torch.empty(n, dtype=torch.uint8, device=device)


def route(x, Wg, bg, k: int, ws: Optional[torch.Tensor] = None, stream=None, renorm: int = 1):
    """clearmoe_route: returns (idx [T,k] int32, gate [T,k] float32)."""
    T, D = x.shape
    E = Wg.shape[0]
    s = make_shape(T, D, E, k, _dt(x), renorm=renorm)
    ws = alloc_workspace(s, x.device) if ws is None else ws
    idx = torch.empty((T, k), dtype=torch.int32, device=x.device)
    gate = torch.empty((T, k), dtype=torch.float32, device=x.device)
    rc = lib().clearmoe_route(ctypes.byref(s), _p(x), _p(Wg), _p(bg), _p(idx), _p(gate), _p(ws),
                              ws.numel(), _stream(stream))
    _check(rc, "clearmoe_route")
    return idx, gate


def make_router(Wg, bg=None, Wh=None, bh=None, adaptive: bool = False, tau: float = 0.0,
                dense_stride: int = 0, W2=None):
    """A Router over device tensors (keep the tensors alive while it is used):
    linear when Wh is None, else an MLP with Wh.shape[0] hidden units; with
    dense_stride > 0, token t with t % dense_stride == 0 is a class token
    (dense path, fc2 weight W2)."""
    p = lambda t: None if t is None else _p(t).value  # noqa: E731
    return Router(p(Wg), p(bg), p(Wh), p(bh), p(W2), 0 if Wh is None else int(Wh.shape[0]),
                  1 if adaptive else 0, int(dense_stride), 0, float(tau))


def route_ex(x, router: Router, E: int, k: int, ws: Optional[torch.Tensor] = None, stream=None,
             renorm: int = 1):
    """clearmoe_route_ex: returns (idx [T,k] int32, -1 = empty slot; gate [T,k])."""
    T, D = x.shape
    s = make_shape(T, D, E, k, _dt(x), renorm=renorm)
    ws = alloc_workspace(s, x.device) if ws is None else ws
    idx = torch.empty((T, k), dtype=torch.int32, device=x.device)
    gate = torch.empty((T, k), dtype=torch.float32, device=x.device)
    rc = lib().clearmoe_route_ex(ctypes.byref(s), ctypes.byref(router), _p(x), _p(idx), _p(gate),
                                 _p(ws), ws.numel(), _stream(stream))
    _check(rc, "clearmoe_route_ex")
    return idx, gate


def dispatch(idx, E: int, ws: Optional[torch.Tensor] = None, x=None, D: Optional[int] = None,
             hist_in_ws: bool = False, stream=None):
    """clearmoe_dispatch: returns (counts, offsets, perm, inv, xperm or None)."""
    T, k = idx.shape
    if x is not None:
        D, dtype = x.shape[1], _dt(x)
    else:
        D, dtype = 8, BF16          # no rows to copy: D only has to be valid
    s = make_shape(T, D, E, k, dtype)
    ws = alloc_workspace(s, idx.device) if ws is None else ws
    dev = idx.device
    counts = torch.empty(E, dtype=torch.int32, device=dev)
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
    perm = torch.empty(T * k, dtype=torch.int32, device=dev)
    inv = torch.empty(T * k, dtype=torch.int32, device=dev)
    xperm = None if x is None else torch.empty((T * k, D), dtype=x.dtype, device=dev)
    rc = lib().clearmoe_dispatch(ctypes.byref(s), _p(idx), _p(ws), ws.numel(), _p(counts),
                                 _p(offsets), _p(perm), _p(inv), _p(x), _p(xperm),
                                 DISPATCH_HIST_IN_WS if hist_in_ws else 0, _stream(stream))
    _check(rc, "clearmoe_dispatch")
    return counts, offsets, perm, inv, xperm


def combine(ye, inv, gate, out: Optional[torch.Tensor] = None, stream=None):
    """clearmoe_combine: y[t] = sum_j gate[t,j] * ye[inv[t*k+j]]."""
    T, k = gate.shape
    D = ye.shape[1]
    E = max(k, 1)
    s = make_shape(T, D, E, k, _dt(ye))
    y = torch.empty((T, D), dtype=ye.dtype, device=ye.device) if out is None else out
    rc = lib().clearmoe_combine(ctypes.byref(s), _p(ye), _p(inv), _p(gate), _p(y),
                                _stream(stream))
    _check(rc, "clearmoe_combine")
    return y


def padded_workspace_bytes(shape: Shape) -> int:
    return int(lib().clearmoe_padded_workspace_bytes(ctypes.byref(shape)))


def _layer_call(name, ws_bytes, x, W1, b1, US, Vt, b2, P, Q, Wg, bg, k, ws, out, idx_out,
                gate_out, stream, renorm=1):
    T, D = x.shape
    H = W1.shape[0]
    r = US.shape[1]
    E, _, q = P.shape
    s = make_shape(T, D, E, k, _dt(x), H=H, r=r, q=q, renorm=renorm)
    if ws is None:
        n = ws_bytes(s)
        if n == 0:
            raise ClearMoEError("invalid shape")
        ws = torch.empty(n, dtype=torch.uint8, device=x.device)
    y = torch.empty((T, D), dtype=x.dtype, device=x.device) if out is None else out
    rc = getattr(lib(), name)(ctypes.byref(s), _p(x), _p(W1), _p(b1), _p(US), _p(Vt), _p(b2),
                              _p(P), _p(Q), _p(Wg), _p(bg), _p(y), _p(idx_out), _p(gate_out),
                              _p(ws), ws.numel(), _stream(stream))
    _check(rc, name)
    return y


def ffn_forward(x, W1, b1, US, Vt, b2, P, Q, Wg, bg, k: int, ws: Optional[torch.Tensor] = None,
                out: Optional[torch.Tensor] = None, idx_out=None, gate_out=None, stream=None,
                renorm: int = 1):
    """clearmoe_ffn_forward: the whole layer.  Returns y [T, D]."""
    return _layer_call("clearmoe_ffn_forward", workspace_bytes, x, W1, b1, US, Vt, b2, P, Q, Wg,
                       bg, k, ws, out, idx_out, gate_out, stream, renorm)


def ffn_forward_noalloc(x, W1, b1, US, Vt, b2, P, Q, Wg, bg, k: int,
                        out: Optional[torch.Tensor] = None, idx_out=None, gate_out=None,
                        stream=None, renorm: int = 1):
    """clearmoe_ffn_forward_noalloc: the whole layer with the library's own
    fixed scratch (no workspace).  Returns y [T, D]."""
    T, D = x.shape
    H = W1.shape[0]
    r = US.shape[1]
    E, _, q = P.shape
    s = make_shape(T, D, E, k, _dt(x), H=H, r=r, q=q, renorm=renorm)
    y = torch.empty((T, D), dtype=x.dtype, device=x.device) if out is None else out
    rc = lib().clearmoe_ffn_forward_noalloc(ctypes.byref(s), _p(x), _p(W1), _p(b1), _p(US), _p(Vt),
                                            _p(b2), _p(P), _p(Q), _p(Wg), _p(bg), _p(y),
                                            _p(idx_out), _p(gate_out), _stream(stream))
    _check(rc, "clearmoe_ffn_forward_noalloc")
    return y


def ffn_forward_padded(x, W1, b1, US, Vt, b2, P, Q, Wg, bg, k: int,
                       ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                       idx_out=None, gate_out=None, stream=None, renorm: int = 1):
    """clearmoe_ffn_forward_padded: the whole layer through the padded batched
    backend (blocks the host until dispatch is done).  Returns y [T, D]."""
    return _layer_call("clearmoe_ffn_forward_padded", padded_workspace_bytes, x, W1, b1, US, Vt,
                       b2, P, Q, Wg, bg, k, ws, out, idx_out, gate_out, stream, renorm)


def ffn_forward_ex(x, W1, b1, US, Vt, b2, P, Q, router: Router, k: int,
                   ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                   idx_out=None, gate_out=None, stream=None, renorm: int = 1):
    """clearmoe_ffn_forward_ex: the whole layer with any router.  Returns y."""
    T, D = x.shape
    H = W1.shape[0]
    r = US.shape[1]
    E, _, q = P.shape
    s = make_shape(T, D, E, k, _dt(x), H=H, r=r, q=q, renorm=renorm)
    ws = alloc_workspace(s, x.device) if ws is None else ws
    y = torch.empty((T, D), dtype=x.dtype, device=x.device) if out is None else out
    rc = lib().clearmoe_ffn_forward_ex(ctypes.byref(s), ctypes.byref(router), _p(x), _p(W1),
                                       _p(b1), _p(US), _p(Vt), _p(b2), _p(P), _p(Q), _p(y),
                                       _p(idx_out), _p(gate_out), _p(ws), ws.numel(),
                                       _stream(stream))
    _check(rc, "clearmoe_ffn_forward_ex")
    return y


def dense_ffn_forward(x, W1, b1, W2, b2, ws: Optional[torch.Tensor] = None,
                      out: Optional[torch.Tensor] = None, stream=None):
    """clearmoe_dense_ffn_forward: y = GELU(x W1^T + b1) W2^T + b2."""
    T, D = x.shape
    H = W1.shape[0]
    s = make_shape(T, D, 1, 1, _dt(x), H=H)
    ws = alloc_workspace(s, x.device) if ws is None else ws
    y = torch.empty((T, D), dtype=x.dtype, device=x.device) if out is None else out
    rc = lib().clearmoe_dense_ffn_forward(ctypes.byref(s), _p(x), _p(W1), _p(b1), _p(W2), _p(b2),
                                          _p(y), _p(ws), ws.numel(), _stream(stream))
    _check(rc, "clearmoe_dense_ffn_forward")
    return y


def make_stack_layer(W1, b1, b2, US=None, Vt=None, P=None, Q=None, router: Optional[Router] = None,
                     k: int = 1, W2=None) -> StackLayer:
    """A stack layer over device tensors (keep them alive while it is used):
    dense when router is None (W1, b1, W2, b2), else a CLEAR-MoE layer."""
    p = lambda t: None if t is None else _p(t).value  # noqa: E731
    if router is None:
        return StackLayer(0, 1, p(W1), p(b1), None, None, p(b2), None, None, p(W2), Router())
    return StackLayer(1, int(k), p(W1), p(b1), p(US), p(Vt), p(b2), p(P), p(Q), p(W2), router)


def stack_shape(x, H: int, E: int, r: int, q: int) -> Shape:
    T, D = x.shape
    return make_shape(T, D, E, 1, _dt(x), H=H, r=r, q=q)


def stack_workspace_bytes(shape: Shape, layers) -> int:
    arr = (StackLayer * len(layers))(*layers)
    return int(lib().clearmoe_stack_workspace_bytes(ctypes.byref(shape), arr, len(layers)))


def stack_forward(x, layers, H: int, E: int, r: int, q: int, residual: bool = True,
                  ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                  stream=None):
    """clearmoe_stack_forward: x through the chain of layers (each a
    StackLayer), x_{l+1} = x_l + f_l(x_l) with residual, else f_l(x_l).
    Returns y [T, D]."""
    s = stack_shape(x, H, E, r, q)
    arr = (StackLayer * len(layers))(*layers)
    if ws is None:
        n = int(lib().clearmoe_stack_workspace_bytes(ctypes.byref(s), arr, len(layers)))
        if n == 0:
            raise ClearMoEError("invalid stack")
        ws = torch.empty(n, dtype=torch.uint8, device=x.device)
    y = torch.empty_like(x) if out is None else out
    rc = lib().clearmoe_stack_forward(ctypes.byref(s), arr, len(layers), 1 if residual else 0,
                                      _p(x), _p(y), _p(ws), ws.numel(), _stream(stream))
    _check(rc, "clearmoe_stack_forward")
    return y


def stage_names():
    return [lib().clearmoe_stage_name(i).decode() for i in range(N_STAGES)]


def timing_start(stages, max_records: int, every: int = 1) -> None:
    """Time every every-th launch of the named stages (at most max_records
    timed launches)."""
    names = stage_names()
    mask = 0
    for s in stages:
        mask |= 1 << names.index(s)
    _check(lib().clearmoe_timing_start_sampled(mask, int(max_records), int(every)),
           "clearmoe_timing_start_sampled")


def timing_stop() -> dict:
    """Stop timing; {stage: (total_ms, launches)} for the stages that ran."""
    ms = (ctypes.c_double * N_STAGES)()
    n = (ctypes.c_int32 * N_STAGES)()
    _check(lib().clearmoe_timing_stop(ms, n), "clearmoe_timing_stop")
    return {name: (ms[i], n[i]) for i, name in enumerate(stage_names()) if n[i] > 0}


def from_stored(a: np.ndarray, device="cuda") -> torch.Tensor:
    """Stored host array -> device tensor: uint16 = bfloat16 bits, float32, int32."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def to_stored(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> host array in the stored convention (bf16 -> uint16 bits)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
