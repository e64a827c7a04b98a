"""Host-only checks of the C ABI: the library loads, exports every function
include/clearmoe.h declares, and rejects bad arguments before touching the GPU
(every call here fails validation, so no HIP call is made)."""
import ctypes
import os
import re

import pytest

from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "clearmoe.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(clearmoe_[a-z_]+)\s*\(", src)))


def test_header_declarations_match_binding():
    assert _declared() == sorted(cm.SYMBOLS)


def test_library_exports_every_declared_symbol():
    L = cm.lib()
    for name in _declared():
        assert hasattr(L, name), name
    nm = os.popen(f"nm -D --defined-only {cm.LIB_PATH}").read()
    for name in _declared():
        assert re.search(rf"\bT {name}\b", nm), name


def test_version_and_status_strings():
    assert cm.version() == 3
    L = cm.lib()
    # the library carries the digest of the sources in the tree
    from paper_2606_28516_amd import build as hb
    assert L.clearmoe_source_digest().decode() == hb.source_digest() == hb.built_digest()
    assert L.clearmoe_status_string(0) == b"ok"
    assert L.clearmoe_status_string(3).startswith(b"workspace")
    assert L.clearmoe_status_string(99) == b"unknown status"


def test_timing_start_rejects_bad_arguments_before_creating_events():
    L = cm.lib()
    assert L.clearmoe_timing_start_sampled(1, 4, 0) == 1      # every < 1
    assert L.clearmoe_timing_start_sampled(1, 0, 2) == 1      # max_records < 1
    assert L.clearmoe_timing_start(1, 0) == 1
    # nothing was started: stopping reports that timing is off
    assert L.clearmoe_timing_stop(None, None) == 1


def _shape(**kw):
    d = dict(T=100, D=64, H=128, E=4, k=2, r=16, q=8, dtype=cm.BF16, renorm=1)
    d.update(kw)
    return cm.make_shape(d["T"], d["D"], d["E"], d["k"], d["dtype"], H=d["H"], r=d["r"], q=d["q"],
                         renorm=d["renorm"])


def test_workspace_bytes_grows_with_shape_and_rejects_bad_shapes():
    a = cm.workspace_bytes(_shape())
    b = cm.workspace_bytes(_shape(T=1000))
    assert 0 < a < b and a % 256 == 0
    assert cm.workspace_bytes(_shape(k=5)) == 0          # k > E
    assert cm.workspace_bytes(_shape(E=65, k=1)) == 0    # E > 64
    # r > min(D, H): not a layer, so the routing / dispatch workspace (D = 12
    # routes on padded copies)
    assert cm.workspace_bytes(_shape(D=12)) == cm.workspace_bytes(_shape(D=12, H=0, r=0, q=0)) > 0
    assert cm.workspace_bytes(_shape(D=0)) == 0
    assert cm.workspace_bytes(_shape(D=12, dtype=cm.F32, H=128, r=4, q=4)) > 0
    # unaligned layer shapes: the aligned layer's workspace plus padded copies
    assert cm.workspace_bytes(_shape(D=60, H=100, r=12, q=6)) > cm.workspace_bytes(_shape(H=104, r=16))
    assert cm.workspace_bytes(_shape(T=0)) > 0
    # the gate rule: 1 (renormalised) or 0 (softmax over all E); nothing else
    assert cm.workspace_bytes(_shape(renorm=0)) == a
    assert cm.workspace_bytes(_shape(renorm=2)) == 0
    assert cm.workspace_bytes(_shape(renorm=-1)) == 0
    # the configurations of the benchmark and tests are all valid
    for c in synth.CONFIGS.values():
        s = cm.make_shape(c.T, c.D, c.E, c.k, cm.F32 if c.dtype == "f32" else cm.BF16,
                          H=c.H, r=c.r, q=c.q)
        assert cm.workspace_bytes(s) > 0


FAKE = ctypes.c_void_p(0x10000)      # aligned, never dereferenced: validation fails first


def test_route_rejects_before_launch():
    L = cm.lib()
    s = _shape()
    ws_n = cm.workspace_bytes(s)
    # NULL x
    assert L.clearmoe_route(ctypes.byref(s), None, FAKE, None, FAKE, FAKE, FAKE, ws_n, None) == 1
    # misaligned x
    assert L.clearmoe_route(ctypes.byref(s), ctypes.c_void_p(0x10002), FAKE, None, FAKE, FAKE,
                            FAKE, ws_n, None) == 1
    # missing / small workspace
    assert L.clearmoe_route(ctypes.byref(s), FAKE, FAKE, None, FAKE, FAKE, None, ws_n, None) == 3
    assert L.clearmoe_route(ctypes.byref(s), FAKE, FAKE, None, FAKE, FAKE, FAKE, 16, None) == 3
    # bad shapes / dtype
    bad = _shape(k=0)
    assert L.clearmoe_route(ctypes.byref(bad), FAKE, FAKE, None, FAKE, FAKE, FAKE, ws_n, None) == 1
    bad = _shape(dtype=7)
    assert L.clearmoe_route(ctypes.byref(bad), FAKE, FAKE, None, FAKE, FAKE, FAKE, ws_n, None) == 2
    bad = _shape(renorm=3)
    assert L.clearmoe_route(ctypes.byref(bad), FAKE, FAKE, None, FAKE, FAKE, FAKE, ws_n, None) == 1
    big = _shape(T=1 << 30, k=2)                                    # T*k >= 2^31
    assert L.clearmoe_route(ctypes.byref(big), FAKE, FAKE, None, FAKE, FAKE, FAKE, ws_n, None) == 1
    assert L.clearmoe_route(None, FAKE, FAKE, None, FAKE, FAKE, FAKE, ws_n, None) == 1


def test_dispatch_combine_ffn_reject_before_launch():
    L = cm.lib()
    s = _shape()
    n = cm.workspace_bytes(s)
    # x without xperm
    assert L.clearmoe_dispatch(ctypes.byref(s), FAKE, FAKE, n, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                               0, None) == 1
    # unknown flag
    assert L.clearmoe_dispatch(ctypes.byref(s), FAKE, FAKE, n, FAKE, FAKE, FAKE, FAKE, None, None,
                               8, None) == 1
    assert L.clearmoe_dispatch(ctypes.byref(s), FAKE, FAKE, 4, FAKE, FAKE, FAKE, FAKE, None, None,
                               0, None) == 3
    assert L.clearmoe_combine(ctypes.byref(s), None, FAKE, FAKE, FAKE, None) == 1
    args = [FAKE] * 13
    # NULL W1
    a = list(args)
    a[1] = None
    assert L.clearmoe_ffn_forward(ctypes.byref(s), *a, FAKE, n, None) == 1
    # r > min(D, H)
    bad = _shape(r=72)
    assert L.clearmoe_ffn_forward(ctypes.byref(bad), *args, FAKE, n, None) == 1
    # q not a multiple of 8 in bf16: a valid layer shape that runs on padded
    # copies, which the workspace of the aligned shape cannot hold
    odd = _shape(q=6)
    assert cm.workspace_bytes(odd) > n
    assert L.clearmoe_ffn_forward(ctypes.byref(odd), *args, FAKE, n, None) == 3
    # routing with D = 60 runs on padded copies too: it needs their workspace,
    # and element alignment of x and Wg
    odd_d = _shape(D=60, r=8)
    big_n = cm.workspace_bytes(odd_d)
    assert big_n > n
    assert L.clearmoe_route(ctypes.byref(odd_d), FAKE, FAKE, None, FAKE, FAKE, FAKE, n, None) == 3
    assert L.clearmoe_route(ctypes.byref(odd_d), ctypes.c_void_p(0x10001), FAKE, None, FAKE, FAKE,
                            FAKE, big_n, None) == 1
    route_only = _shape(D=60, H=0, r=0, q=0)          # no layer fields: routing's own pads
    assert 0 < cm.workspace_bytes(route_only) < big_n
    # dispatch / combine rows of 60 elements need element alignment only
    assert L.clearmoe_combine(ctypes.byref(route_only), ctypes.c_void_p(0x10001), FAKE, FAKE, FAKE,
                              None) == 1
    assert L.clearmoe_dispatch(ctypes.byref(route_only), FAKE, FAKE, 4, FAKE, FAKE, FAKE, FAKE,
                               ctypes.c_void_p(0x10002), FAKE, 0, None) == 3
    # workspace one byte short
    assert L.clearmoe_ffn_forward(ctypes.byref(s), *args, FAKE, n - 1, None) == 3


def test_noalloc_rejects_before_launch():
    """The no-allocation variant checks its arguments like clearmoe_ffn_forward
    and refuses a shape whose regions exceed its fixed scratch, all before any
    HIP call."""
    L = cm.lib()
    s = _shape()
    args = [FAKE] * 13
    a = list(args)
    a[1] = None                                   # NULL W1
    assert L.clearmoe_ffn_forward_noalloc(ctypes.byref(s), *a, None) == 1
    bad = _shape(q=6)
    assert L.clearmoe_ffn_forward_noalloc(ctypes.byref(bad), *args, None) == 1
    # the DeiT-Base top-2 layer keeps z [T, H] (310 MB): too large
    big = cm.make_shape(50432, 768, 8, 2, cm.BF16, H=3072, r=256, q=64)
    assert L.clearmoe_ffn_forward_noalloc(ctypes.byref(big), *args, None) == cm.ERR_TOO_LARGE
    assert L.clearmoe_status_string(cm.ERR_TOO_LARGE).startswith(b"shape needs more scratch")


def _prototypes():
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    out = {}
    for m in re.finditer(r"\b(clearmoe_[a-z_]+)\s*\(([^)]*)\)\s*;", src):
        params = m.group(2).strip()
        out[m.group(1)] = 0 if params in ("", "void") else params.count(",") + 1
    return out


def test_binding_signatures_match_header():
    L = cm.lib()
    protos = _prototypes()
    assert set(protos) == set(cm.SYMBOLS)
    for name, n in protos.items():
        argtypes = getattr(L, name).argtypes
        assert len(argtypes or []) == n, (name, len(argtypes or []), n)


def test_padded_entry_point_workspace_and_rejections():
    L = cm.lib()
    s = _shape()
    n = cm.workspace_bytes(s)
    npad = cm.padded_workspace_bytes(s)
    # room for E * T * k padded rows of u (dtype) and h_res (float32) on top
    # of the grouped workspace
    E, T, k, D, q = s.E, s.T, s.k, s.D, s.q
    assert npad >= n + E * T * k * (2 * q + 4 * D)
    assert cm.padded_workspace_bytes(_shape(k=5)) == 0
    assert cm.padded_workspace_bytes(_shape(T=2 * s.T)) > npad
    args = [FAKE] * 13
    a = list(args)
    a[1] = None                                                    # NULL W1
    assert L.clearmoe_ffn_forward_padded(ctypes.byref(s), *a, FAKE, npad, None) == 1
    assert L.clearmoe_ffn_forward_padded(ctypes.byref(_shape(q=6)), *args, FAKE, npad,
                                         None) == 1
    # the grouped workspace is not enough for the padded batch
    assert L.clearmoe_ffn_forward_padded(ctypes.byref(s), *args, FAKE, n, None) == 3
    assert L.clearmoe_ffn_forward_padded(ctypes.byref(s), *args, FAKE, npad - 1, None) == 3
    assert L.clearmoe_ffn_forward_padded(ctypes.byref(s), *args, None, npad, None) == 3


def _router(**kw):
    d = dict(Wg=FAKE.value, bg=None, Wh=None, bh=None, W2=None, hidden=0, adaptive=0,
             dense_stride=0, reserved=0, tau=0.0)
    d.update(kw)
    return cm.Router(d["Wg"], d["bg"], d["Wh"], d["bh"], d["W2"], d["hidden"], d["adaptive"],
                     d["dense_stride"], d["reserved"], d["tau"])


def test_shape_descriptor_layout():
    """The ctypes mirror of clearmoe_shape: nine int32 (the gate rule last)."""
    assert ctypes.sizeof(cm.Shape) == 36
    assert cm.Shape.dtype.offset == 28 and cm.Shape.renorm.offset == 32
    assert cm.make_shape(1, 8, 2, 1, cm.BF16).renorm == 1


def test_router_descriptor_layout():
    """The ctypes mirror of clearmoe_router: five pointers, four int32, one
    double, no padding (64 bytes)."""
    assert ctypes.sizeof(cm.Router) == 64
    assert cm.Router.hidden.offset == 40 and cm.Router.dense_stride.offset == 48
    assert cm.Router.tau.offset == 56


def test_route_ex_and_ffn_ex_reject_bad_routers_before_launch():
    L = cm.lib()
    s = _shape()                                   # E = 4, k = 2
    n = cm.workspace_bytes(s)
    ok_args = (FAKE, FAKE, FAKE, FAKE, n, None)    # x, idx, gate, ws, bytes, stream

    def route(r, shape=s):
        return L.clearmoe_route_ex(ctypes.byref(shape), None if r is None else ctypes.byref(r),
                                   *ok_args)
    assert route(None) == 1                                         # no router
    assert route(_router(Wg=None)) == 1                             # no output layer
    assert route(_router(Wg=0x10002)) == 1                          # misaligned Wg
    assert route(_router(hidden=-1)) == 1
    assert route(_router(hidden=257, Wh=FAKE.value)) == 1           # above the MLP limit
    assert route(_router(hidden=64)) == 1                           # MLP without Wh
    assert route(_router(hidden=64, Wh=0x10008)) == 1               # misaligned Wh
    assert route(_router(hidden=64, Wh=FAKE.value, bh=0x10001)) == 1
    assert route(_router(adaptive=2)) == 1
    assert route(_router(adaptive=1, tau=float("nan"))) == 1        # NaN threshold
    assert route(_router(adaptive=1, tau=0.5), _shape(k=1)) == 1    # adaptive needs k = 2
    assert route(_router(adaptive=1, tau=0.5), _shape(E=1, k=1)) == 1
    assert route(_router(dense_stride=-1)) == 1
    assert route(_router(reserved=1)) == 1
    assert route(_router(dense_stride=197, W2=0x10004)) == 1        # misaligned W2
    assert L.clearmoe_route_ex(ctypes.byref(s), ctypes.byref(_router()), FAKE, FAKE, FAKE, FAKE,
                               8, None) == 3                        # workspace too small
    args = [FAKE] * 11
    assert L.clearmoe_ffn_forward_ex(ctypes.byref(s), None, *args, FAKE, n, None) == 1
    assert L.clearmoe_ffn_forward_ex(ctypes.byref(s), ctypes.byref(_router(hidden=300,
                                     Wh=FAKE.value)), *args, FAKE, n, None) == 1
    assert L.clearmoe_ffn_forward_ex(ctypes.byref(_shape(k=1)),
                                     ctypes.byref(_router(adaptive=1, tau=0.9)), *args, FAKE, n,
                                     None) == 1
    a = list(args)
    a[1] = None                                                     # NULL W1
    assert L.clearmoe_ffn_forward_ex(ctypes.byref(s), ctypes.byref(_router()), *a, FAKE, n,
                                     None) == 1
    # class tokens need the dense fc2 weight
    assert L.clearmoe_ffn_forward_ex(ctypes.byref(s), ctypes.byref(_router(dense_stride=197)),
                                     *args, FAKE, n, None) == 1
    assert L.clearmoe_ffn_forward_ex(ctypes.byref(s), ctypes.byref(_router()), *args, FAKE, n - 1,
                                     None) == 3


def test_stack_workspace_and_rejections_before_launch():
    """The stack entry point sizes its workspace from its largest layer plus
    three activation buffers, and checks every layer before launching any."""
    L = cm.lib()
    s = _shape(k=1)
    f = FAKE.value
    router = cm.Router(f, None, None, None, None, 0, 0, 0, 0, 0.0)
    moe1 = cm.StackLayer(1, 1, f, None, f, f, None, f, f, None, router)
    moe2 = cm.StackLayer(1, 2, f, None, f, f, None, f, f, None, router)
    dense = cm.StackLayer(0, 1, f, None, None, None, None, None, None, f, cm.Router())
    arr = (cm.StackLayer * 3)(moe1, dense, moe2)
    n = L.clearmoe_stack_workspace_bytes(ctypes.byref(s), arr, 3)
    act = 100 * 64 * 2
    assert n >= cm.workspace_bytes(_shape(k=2)) + 3 * act
    assert L.clearmoe_stack_workspace_bytes(ctypes.byref(s), arr, 0) == 0
    bad = (cm.StackLayer * 3)(moe1, dense, cm.StackLayer(2, 1, f, None, f, f, None, f, f, None,
                                                         router))
    assert L.clearmoe_stack_workspace_bytes(ctypes.byref(s), bad, 3) == 0
    # the third layer has no W1: refused although the first two are valid
    nw1 = cm.StackLayer(1, 2, None, None, f, f, None, f, f, None, router)
    arr2 = (cm.StackLayer * 3)(moe1, dense, nw1)
    assert L.clearmoe_stack_forward(ctypes.byref(s), arr2, 3, 1, FAKE, FAKE, FAKE, n, None) == 1
    # k > E in a layer, a dense layer without W2, a bad residual flag
    bigk = (cm.StackLayer * 1)(cm.StackLayer(1, 5, f, None, f, f, None, f, f, None, router))
    assert L.clearmoe_stack_forward(ctypes.byref(s), bigk, 1, 1, FAKE, FAKE, FAKE, n, None) == 1
    nw2 = (cm.StackLayer * 1)(cm.StackLayer(0, 1, f, None, None, None, None, None, None, None,
                                            cm.Router()))
    assert L.clearmoe_stack_forward(ctypes.byref(s), nw2, 1, 1, FAKE, FAKE, FAKE, n, None) == 1
    assert L.clearmoe_stack_forward(ctypes.byref(s), arr, 3, 2, FAKE, FAKE, FAKE, n, None) == 1
    # workspace one byte short
    assert L.clearmoe_stack_forward(ctypes.byref(s), arr, 3, 1, FAKE, FAKE, FAKE, n - 1, None) == 3
