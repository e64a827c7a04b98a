"""GPU parity of the class-token dense path (Table C6: the class token of each
image is excluded from expert dispatch and runs on the dense path, the
original fc1 + GELU + fc2): routing marks every token t with t % s == 0 as
having no expert, dispatch leaves it out, and the layer gives it the dense
FFN's output, against the CPU oracle on seeded inputs."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

from parity_util import (bound_excluded, BF16_FROB_REGRESS, F32_MAXREL, MARGIN, check_dispatch, confidence_gap,
                         dev, frob_rel, gpu_ffn_ex, gpu_router, max_rel)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    cm.lib()
    yield
    torch.cuda.synchronize()


def _check_layer(C, g, ref, excl, dt):
    cls = ref["cls"]
    assert np.all(g["idx"][cls] == -1) and np.all(g["gate"][cls] == 0.0)
    ok = ~excl
    assert np.array_equal(g["idx"][ok], ref["idx"][ok])
    for rows in (ok & cls, ok & ~cls):               # the dense rows and the expert rows apart
        if dt == "f32":
            assert max_rel(g["y"][rows], ref["y"][rows]) <= F32_MAXREL
        else:
            e = frob_rel(g["y"][rows], ref["y"][rows])
            assert e <= BF16_FROB_REGRESS, e


LAYERS = [
    # dtype, T, D, H, E, k, r, q, stride  (the first two take the fused top-1 kernel)
    ("bf16", 197 * 3, 128, 256, 4, 1, 64, 16, 197),
    ("bf16", 1000, 64, 192, 6, 1, 32, 32, 77),          # T not a multiple of the stride
    ("bf16", 400, 64, 192, 6, 2, 32, 24, 13),
    ("f32", 300, 64, 128, 4, 1, 16, 8, 50),             # the GEMM chain of top-1
    ("f32", 257, 96, 160, 5, 3, 32, 16, 16),
    ("bf16", 5, 64, 128, 3, 1, 32, 8, 1),               # every token a class token
]


@pytest.mark.parametrize("dt,T,D,H,E,k,r,q,stride", LAYERS)
def test_class_tokens_layer(dt, T, D, H, E, k, r, q, stride):
    cfg = synth.LayerConfig("cls", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dt, seed=T + stride,
                            residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(stride)
    L["b1"] = (0.1 * rng.standard_normal(H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    C = synth.with_class_tokens(L, stride=stride)
    g = gpu_ffn_ex(C)
    ref = oracle.ffn_forward_layer(C)
    assert ref["cls"].sum() == (T + stride - 1) // stride
    excl = bound_excluded(oracle.margins(ref["logits"], k) < MARGIN)
    _check_layer(C, g, ref, excl, dt)


def test_class_tokens_route_and_dispatch():
    """route_ex leaves every slot of a class token empty; dispatch counts only
    the routed tokens, bit for bit against the oracle."""
    L = synth.make_dispatch(T=4000, D=128, E=8, k=2, dtype="bf16", seed=6)
    L["dense_stride"] = 197
    L["W2"] = None
    r, keep = gpu_router({"Wg": L["Wg"], "bg": L["bg"], "dense_stride": 197,
                          "W2": np.zeros((128, 16), np.uint16)})
    x = dev(L["x"])
    s = cm.make_shape(4000, 128, 8, 2, cm.BF16)
    ws = cm.alloc_workspace(s)
    idx, gate = cm.route_ex(x, r, 8, 2, ws=ws)
    counts, offsets, perm, inv, _ = cm.dispatch(idx, 8, ws=ws, x=x, hist_in_ws=True)
    torch.cuda.synchronize()
    idx_h, gate_h = idx.cpu().numpy(), gate.cpu().numpy()
    cls = np.arange(4000) % 197 == 0
    assert np.all(idx_h[cls] == -1) and np.all(gate_h[cls] == 0.0)
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    want, _ = oracle.topk(lg, 2)
    ok = ~cls & ~bound_excluded(oracle.margins(lg, 2) < MARGIN)
    assert np.array_equal(idx_h[ok], want[ok])
    check_dispatch(idx_h, 8, counts.cpu().numpy(), offsets.cpu().numpy(), perm.cpu().numpy(),
                   inv.cpu().numpy())
    assert offsets.cpu().numpy()[-1] == 2 * (4000 - cls.sum())


def test_class_tokens_with_adaptive_and_mlp_routers():
    cfg = synth.LayerConfig("clsr", T=600, D=96, H=192, E=5, k=1, r=32, q=16, dtype="bf16",
                            seed=3, residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    tau = float(np.quantile(oracle.confidence(lg), 0.5))
    A = synth.with_class_tokens(synth.with_adaptive_router(L, tau), stride=100)
    g = gpu_ffn_ex(A)
    ref = oracle.ffn_forward_layer(A)
    excl = bound_excluded((oracle.margins(lg, 2) < MARGIN) | (confidence_gap(lg, tau) < 1e-9))
    _check_layer(A, g, ref, excl, "bf16")
    M = synth.with_class_tokens(synth.with_mlp_router(L, h=16, seed=2), stride=60)
    g = gpu_ffn_ex(M)
    ref = oracle.ffn_forward_layer(M)
    excl = bound_excluded(oracle.margins(ref["logits"], 1) < MARGIN)
    _check_layer(M, g, ref, excl, "bf16")


def _sample_rows(T, n, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, T - 1], rng.choice(T, size=min(n, T), replace=False)]))


def test_class_tokens_at_deit_small():
    """The DeiT-Small-shaped layer (64 images x 197 tokens) with its 64 class
    tokens on the dense path: routing on every token, values on every class
    row and a sample of the others."""
    C = synth.with_class_tokens(synth.make_layer(synth.CONFIGS["C2"]), stride=197)
    g = gpu_ffn_ex(C)
    T = C["cfg"].T
    lg = oracle.router_logits(C["x"], C["Wg"], C["bg"])
    cls = np.arange(T) % 197 == 0
    assert np.all(g["idx"][cls] == -1)
    ok = ~cls & ~bound_excluded(oracle.margins(lg, 1) < MARGIN)
    assert np.array_equal(g["idx"][ok, 0], oracle.topk(lg, 1)[0][ok, 0])
    rows = np.unique(np.concatenate([np.nonzero(cls)[0], _sample_rows(T, 192, 4)]))
    rows = rows[cls[rows] | ok[rows]]
    ref = oracle.ffn_forward_layer(C, rows=rows)
    for sel in (ref["cls"], ~ref["cls"]):
        e = frob_rel(g["y"][rows][sel], ref["y"][sel])
        assert e <= BF16_FROB_REGRESS, e


IN_LAUNCH = [
    # T, D, H, E, r, q, stride: enough 64-row tiles for one workgroup per tile,
    # so the class rows run on extra workgroups of the fused launch
    (9000, 264, 1000, 4, 64, 32, 150),   # D % 16 = 8, H % 128 = 104; 60 class rows: two blocks
                                         # of 32, the second partial, each split over the hidden width
    (9000, 320, 512, 4, 32, 16, 5),      # 1800 class rows: 57 blocks, too many to split
]


@pytest.mark.parametrize("T,D,H,E,r,q,stride", IN_LAUNCH)
def test_class_rows_inside_fused_launch(T, D, H, E, r, q, stride):
    """The fused launch's class-row workgroups: no launch of their own (no
    dense-path stage runs), every class row and a sample of the others
    against the oracle."""
    cfg = synth.LayerConfig("clsin", T=T, D=D, H=H, E=E, k=1, r=r, q=q, dtype="bf16", seed=T + stride,
                            residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(stride)
    L["b1"] = (0.1 * rng.standard_normal(H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    C = synth.with_class_tokens(L, stride=stride)
    cm.timing_start(cm.stage_names(), max_records=64)
    try:
        g = gpu_ffn_ex(C)
    finally:
        t = cm.timing_stop()
    launched = {k for k, v in t.items() if v[1] > 0}
    assert "fused_top1" in launched and not launched & {"fc1_gelu", "dense_fc2"}, launched
    lg = oracle.router_logits(C["x"], C["Wg"], C["bg"])
    cls = np.arange(T) % stride == 0
    assert np.all(g["idx"][cls] == -1)
    ok = ~cls & ~bound_excluded(oracle.margins(lg, 1) < MARGIN)
    assert np.array_equal(g["idx"][ok, 0], oracle.topk(lg, 1)[0][ok, 0])
    rows = np.unique(np.concatenate([np.nonzero(cls)[0], _sample_rows(T, 256, 5)]))
    rows = rows[cls[rows] | ok[rows]]
    ref = oracle.ffn_forward_layer(C, rows=rows)
    for what, sel in (("class", ref["cls"]), ("routed", ~ref["cls"])):
        e = frob_rel(g["y"][rows][sel], ref["y"][sel])
        print(f"{what} rows: relative Frobenius error {e:.3e}")
        assert e <= BF16_FROB_REGRESS, e
    assert np.all(np.isfinite(g["y"]))


def test_class_rows_ordered_on_the_callers_stream():
    """The class rows come from a side stream that the caller's stream joins:
    work queued after the call on a user stream (here a copy of y, with no
    device-wide synchronisation in between) sees them, on every call of a
    repeated sequence."""
    C = synth.with_class_tokens(
        synth.make_layer(synth.LayerConfig("ord", T=197 * 8, D=128, H=256, E=4, k=1, r=64, q=16,
                                           dtype="bf16", seed=9, residual="random",
                                           n_cal=2000)), stride=197)
    d = {n: dev(C[n]) for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q")}
    r, keep = gpu_router(C)
    ref = oracle.ffn_forward_layer(C)
    cls = ref["cls"]
    s = torch.cuda.Stream()
    y = torch.empty_like(d["x"])
    copies = []
    with torch.cuda.stream(s):
        for _ in range(3):
            y.fill_(float("nan"))
            cm.ffn_forward_ex(d["x"], d["W1"], d["b1"], d["US"], d["Vt"], d["b2"], d["P"], d["Q"],
                              r, 1, out=y, stream=s)
            copies.append(y.clone())
    torch.cuda.synchronize()
    for c in copies:
        got = oracle.widen(cm.to_stored(c))
        assert np.isfinite(got).all()
        e = frob_rel(got[cls], ref["y"][cls])
        assert e <= BF16_FROB_REGRESS, e
