"""ctypes wrapper of the C oracle (``clearmoe_ref.c``).  Test infrastructure only.

Inputs are stored arrays: float32, or bfloat16 bit patterns held as uint16.
They are widened exactly to float64 here and handed to the C code, which
does all arithmetic in double.  Outputs are float64 (values) and int32
(indices).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "clearmoe_ref.c")
_LIB_PATH = os.path.join(_HERE, "libclearmoe_ref.so")
_lib = None

__all__ = ["build", "lib", "widen", "num_threads", "set_num_threads", "gelu", "router_logits",
           "topk", "route", "dispatch", "permute_rows", "fc1_gelu", "shared", "residual",
           "ffn_forward", "ffn_forward_layer", "combine", "margins", "adaptive_topk",
           "round_to_storage", "mlp_router_logits", "route_layer", "ffn_forward_routed",
           "confidence", "dense_fc2", "class_tokens", "full_softmax_gates"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, OpenMP over tokens)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        L = ctypes.CDLL(_LIB_PATH)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        i64, i32 = ctypes.c_int64, ctypes.c_int
        L.ref_num_threads.restype = i32
        L.ref_set_num_threads.argtypes = [i32]
        L.ref_gelu.restype = ctypes.c_double
        L.ref_gelu.argtypes = [ctypes.c_double]
        L.ref_router_logits.argtypes = [i64, i32, i32, dp, dp, dp, dp]
        L.ref_topk.argtypes = [i64, i32, i32, dp, ip, dp]
        L.ref_dispatch.argtypes = [i64, i32, i32, ip, ip, ip, ip, ip]
        L.ref_dispatch.restype = i32
        L.ref_permute_rows.argtypes = [i64, i32, i32, dp, ip, dp]
        L.ref_fc1_gelu.argtypes = [i64, i32, i32, dp, dp, dp, dp]
        L.ref_shared.argtypes = [i64, i32, i32, i32, dp, dp, dp, dp, dp]
        L.ref_residual.argtypes = [i64, i32, i32, i32, i32, i32, dp, dp, dp, ip, dp, dp]
        L.ref_ffn_forward.argtypes = [i64] + [i32] * 6 + [dp] * 10 + [dp, ip, dp, dp]
        L.ref_ffn_forward.restype = i32
        L.ref_combine.argtypes = [i64, i32, i32, dp, ip, dp, dp]
        L.ref_adaptive_topk.argtypes = [i64, i32, ctypes.c_double, dp, ip, dp]
        L.ref_dense_fc2.argtypes = [i64, i32, i32, dp, dp, dp, dp]
        _lib = L
    return _lib


def widen(a) -> np.ndarray:
    """Stored array -> float64, exactly.  uint16 is read as bfloat16 bits."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (np.ascontiguousarray(a).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.ascontiguousarray(a, dtype=np.float64)


def _dp(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f64(a):
    return None if a is None else np.ascontiguousarray(widen(a))


def num_threads() -> int:
    return lib().ref_num_threads()


def set_num_threads(n: int) -> None:
    lib().ref_set_num_threads(int(n))


def gelu(v: float) -> float:
    return lib().ref_gelu(float(v))


def router_logits(x, Wg, bg=None) -> np.ndarray:
    x, Wg, bg = _f64(x), _f64(Wg), _f64(bg)
    T, D = x.shape
    E = Wg.shape[0]
    out = np.empty((T, E))
    lib().ref_router_logits(T, D, E, _dp(x), _dp(Wg), _dp(bg), _dp(out))
    return out


def topk(logits, k: int):
    logits = np.ascontiguousarray(logits, dtype=np.float64)
    T, E = logits.shape
    idx = np.empty((T, k), dtype=np.int32)
    gate = np.empty((T, k))
    lib().ref_topk(T, E, k, _dp(logits), _ip(idx), _dp(gate))
    return idx, gate


def adaptive_topk(logits, tau: float):
    """Adaptive router's choice (Sec. III Phase 4): (idx [T,2], gate [T,2]);
    slot 1 is -1 (gate 0) for tokens whose confidence is at least tau."""
    logits = np.ascontiguousarray(logits, dtype=np.float64)
    T, E = logits.shape
    idx = np.empty((T, 2), dtype=np.int32)
    gate = np.empty((T, 2))
    lib().ref_adaptive_topk(T, E, float(tau), _dp(logits), _ip(idx), _dp(gate))
    return idx, gate


def full_softmax_gates(logits, idx) -> np.ndarray:
    """Gates without renormalisation (shape field renorm = 0): the chosen
    experts' probabilities under the softmax over all E logits of the token
    (Sec. III Phase 4: the router's scores as a distribution over experts).
    An empty slot (idx -1) gets 0.  Plain loops over tokens and slots."""
    lg = np.asarray(logits, dtype=np.float64)
    idx = np.asarray(idx)
    T, k = idx.shape
    gate = np.zeros((T, k))
    for t in range(T):
        m = lg[t].max()
        den = np.sum(np.exp(lg[t] - m))
        for j in range(k):
            if idx[t, j] >= 0:
                gate[t, j] = np.exp(lg[t, idx[t, j]] - m) / den
    return gate


def confidence(logits) -> np.ndarray:
    """Largest softmax probability of each token (the adaptive router's
    confidence), in double."""
    lg = np.asarray(logits, dtype=np.float64)
    return 1.0 / np.sum(np.exp(lg - lg.max(axis=1, keepdims=True)), axis=1)


def round_to_storage(v, dtype: str) -> np.ndarray:
    """Round exact values once to the storage precision: float32, or bfloat16
    (8 significant bits, ties to even).  Returns float64."""
    v = np.asarray(v, dtype=np.float64)
    if dtype == "f32":
        return v.astype(np.float32).astype(np.float64)
    if dtype != "bf16":
        raise ValueError(dtype)
    m, e = np.frexp(v)                       # v = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.round(np.ldexp(m, 8)), e - 8)


def mlp_router_logits(x, Wh, bh, Wg, bg, dtype: str):
    """MLP router (Sec. III Phase 4, hidden width h = d/6): the hidden layer
    hr = GELU(x Wh^T + bh) is rounded to the storage precision (where the
    kernels keep it), then l = hr Wg^T + bg exactly.  Returns (logits, hr)."""
    hr = round_to_storage(fc1_gelu(x, Wh, bh), dtype)
    return router_logits(hr, Wg, bg), hr


def route_layer(layer: dict, rows=None):
    """Routing of a layer dict by its router (linear when the dict has no
    "router" entry).  Returns (idx, gate, logits)."""
    x = layer["x"] if rows is None else layer["x"][np.asarray(rows)]
    rt = layer.get("router") or {"kind": "linear"}
    k = layer["cfg"].k
    if rt["kind"] == "mlp":
        lg, _ = mlp_router_logits(x, rt["Wh"], rt["bh"], layer["Wg"], layer["bg"],
                                  layer["cfg"].dtype)
    else:
        lg = router_logits(x, layer["Wg"], layer["bg"])
    if rt["kind"] == "adaptive":
        idx, gate = adaptive_topk(lg, rt["tau"])
    else:
        idx, gate = topk(lg, k)
    if int(layer.get("renorm", 1)) == 0:
        gate = full_softmax_gates(lg, idx)
    return idx, gate, lg


def route(x, Wg, bg, k: int):
    """(idx [T,k], gate [T,k], logits [T,E])."""
    lg = router_logits(x, Wg, bg)
    idx, gate = topk(lg, k)
    return idx, gate, lg


def dispatch(idx, E: int):
    """(counts [E], offsets [E+1], perm [T*k], inv [T*k]) of an idx [T,k] array."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    T, k = idx.shape
    counts = np.empty(E, dtype=np.int32)
    offsets = np.empty(E + 1, dtype=np.int32)
    perm = np.empty(T * k, dtype=np.int32)
    inv = np.empty(T * k, dtype=np.int32)
    rc = lib().ref_dispatch(T, E, k, _ip(idx), _ip(counts), _ip(offsets), _ip(perm), _ip(inv))
    if rc != 0:
        raise ValueError("expert index out of range")
    return counts, offsets, perm, inv


def permute_rows(x, perm, k: int) -> np.ndarray:
    x = _f64(x)
    perm = np.ascontiguousarray(perm, dtype=np.int32)
    T, D = x.shape
    out = np.empty((T * k, D))
    lib().ref_permute_rows(T, D, k, _dp(x), _ip(perm), _dp(out))
    return out


def fc1_gelu(x, W1, b1=None) -> np.ndarray:
    x, W1, b1 = _f64(x), _f64(W1), _f64(b1)
    T, D = x.shape
    H = W1.shape[0]
    z = np.empty((T, H))
    lib().ref_fc1_gelu(T, D, H, _dp(x), _dp(W1), _dp(b1), _dp(z))
    return z


def shared(z, Vt, US, b2=None) -> np.ndarray:
    z, Vt, US, b2 = _f64(z), _f64(Vt), _f64(US), _f64(b2)
    T, H = z.shape
    D, r = US.shape
    out = np.empty((T, D))
    lib().ref_shared(T, D, H, r, _dp(z), _dp(Vt), _dp(US), _dp(b2), _dp(out))
    return out


def dense_fc2(z, W2, b2=None) -> np.ndarray:
    """z W2^T + b2: fc2 of the unexpertised FFN (the class tokens' dense path)."""
    z, W2, b2 = _f64(z), _f64(W2), _f64(b2)
    T, H = z.shape
    D = W2.shape[0]
    out = np.empty((T, D))
    lib().ref_dense_fc2(T, D, H, _dp(z), _dp(W2), _dp(b2), _dp(out))
    return out


def class_tokens(tokens, stride: int) -> np.ndarray:
    """Mask of the class tokens among the given token indices: one per image of
    `stride` tokens, the first (Table C6: 197 tokens per image, the class token
    excluded from dispatch).  stride <= 0: none."""
    tokens = np.asarray(tokens)
    if stride <= 0:
        return np.zeros(tokens.shape, dtype=bool)
    return tokens % stride == 0


def residual(z, Q, P, idx, gate) -> np.ndarray:
    z, Q, P = _f64(z), _f64(Q), _f64(P)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    gate = np.ascontiguousarray(gate, dtype=np.float64)
    T, H = z.shape
    E, D, q = P.shape
    k = idx.shape[1]
    out = np.empty((T, D))
    lib().ref_residual(T, D, H, E, k, q, _dp(z), _dp(Q), _dp(P), _ip(idx), _dp(gate), _dp(out))
    return out


def ffn_forward(x, W1, b1, US, Vt, b2, P, Q, Wg, bg, k: int):
    """Whole layer.  Returns dict(y [T,D] f64, idx, gate, logits)."""
    x, W1, b1, US, Vt, b2 = _f64(x), _f64(W1), _f64(b1), _f64(US), _f64(Vt), _f64(b2)
    P, Q, Wg, bg = _f64(P), _f64(Q), _f64(Wg), _f64(bg)
    T, D = x.shape
    H = W1.shape[0]
    r = US.shape[1]
    E, _, q = P.shape
    y = np.empty((T, D))
    idx = np.empty((T, k), dtype=np.int32)
    gate = np.empty((T, k))
    logits = np.empty((T, E))
    rc = lib().ref_ffn_forward(T, D, H, E, k, r, q, _dp(x), _dp(W1), _dp(b1), _dp(US), _dp(Vt),
                               _dp(b2), _dp(P), _dp(Q), _dp(Wg), _dp(bg), _dp(y), _ip(idx),
                               _dp(gate), _dp(logits))
    if rc != 0:
        raise ValueError(f"oracle ffn_forward failed ({rc})")
    return dict(y=y, idx=idx, gate=gate, logits=logits)


def ffn_forward_routed(x, W1, b1, US, Vt, b2, P, Q, idx, gate):
    """The layer after routing (Eq. 2, Algorithm 3): y = h_sh + h_res with the
    given idx [T,k] (-1 = empty slot) and gates."""
    z = fc1_gelu(x, W1, b1)
    return shared(z, Vt, US, b2) + residual(z, Q, P, idx, gate)


def ffn_forward_layer(layer: dict, rows=None):
    """ffn_forward on a layer dict as drawn by the input generator.

    ``rows`` (optional index array) evaluates only those tokens: every output
    of the layer depends on its own token alone, so a sample of rows gives the
    same values as the full run at those rows.  A "router" entry (MLP or
    adaptive) routes through route_layer; without it the linear router runs.
    A "renorm" entry 0 gives the unrenormalised gates (full_softmax_gates).
    A "dense_stride" entry s > 0 makes every token t with t % s == 0 a class
    token (Table C6): it takes no expert slot (idx -1, gate 0) and its output
    is the dense FFN's, GELU(x W1^T + b1) W2^T + b2 with the layer's "W2".
    """
    x = layer["x"] if rows is None else layer["x"][np.asarray(rows)]
    stride = int(layer.get("dense_stride") or 0)
    if stride > 0:
        # class tokens: no expert slot, and the dense FFN's output (Table C6)
        tok = np.arange(layer["x"].shape[0]) if rows is None else np.asarray(rows)
        cls = class_tokens(tok, stride)
        idx, gate, lg = route_layer(layer, rows)
        idx[cls] = -1
        gate[cls] = 0.0
        z = fc1_gelu(x, layer["W1"], layer["b1"])
        y = shared(z, layer["Vt"], layer["US"], layer["b2"]) + residual(z, layer["Q"], layer["P"],
                                                                        idx, gate)
        y[cls] = dense_fc2(z[cls], layer["W2"], layer["b2"])
        return dict(y=y, idx=idx, gate=gate, logits=lg, cls=cls)
    if (layer.get("router") is not None and layer["router"]["kind"] != "linear") or \
            int(layer.get("renorm", 1)) == 0:
        idx, gate, lg = route_layer(layer, rows)
        y = ffn_forward_routed(x, layer["W1"], layer["b1"], layer["US"], layer["Vt"],
                               layer["b2"], layer["P"], layer["Q"], idx, gate)
        return dict(y=y, idx=idx, gate=gate, logits=lg)
    return ffn_forward(x, layer["W1"], layer["b1"], layer["US"], layer["Vt"], layer["b2"],
                       layer["P"], layer["Q"], layer["Wg"], layer["bg"], layer["cfg"].k)


def combine(ye, inv, gate, k: int) -> np.ndarray:
    ye = _f64(ye)
    inv = np.ascontiguousarray(inv, dtype=np.int32)
    gate = np.ascontiguousarray(gate, dtype=np.float64)
    D = ye.shape[1]
    T = inv.size // k
    y = np.empty((T, D))
    lib().ref_combine(T, D, k, _dp(ye), _ip(inv), _dp(gate), _dp(y))
    return y


def margins(logits, k: int) -> np.ndarray:
    """Per-token decision margin: the smallest gap between consecutive sorted
    logits among the first min(k+1, E) (covers the selection boundary and the
    slot order).  Infinite when E == 1."""
    s = -np.sort(-np.asarray(logits, dtype=np.float64), axis=1)
    E = s.shape[1]
    m = min(k, E - 1)
    if m <= 0:
        return np.full(s.shape[0], np.inf)
    return np.min(s[:, :m] - s[:, 1:m + 1], axis=1)
