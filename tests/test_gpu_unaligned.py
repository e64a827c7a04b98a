"""GPU parity of the entry points on unaligned shapes (D, H, r or q not a
multiple of the elements of a 16-byte piece): the layer entry points and
routing run on zero-padded copies of their operands, dispatch and combine
copy rows element by element.  Routing bit-exact and y within the bars
against the oracle, which computes the unpadded layer.  Cases: top-1 and top-2, both
dtypes, class tokens, the MLP router, the dense FFN, and a shape that pads
into the fused top-1 kernel's range (one workgroup per tile, class rows in
its launch)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

from parity_util import (BF16_FROB_REGRESS, F32_MAXREL, MARGIN, assert_elementwise, assert_gates,
                         assert_routing, bound_excluded, check_dispatch, confidence_gap, dev, frob_rel,
                         gpu_ffn, gpu_ffn_ex, gpu_router, max_rel)

pytestmark = pytest.mark.gpu

CASES = [
    # dtype, T, D, H, E, k, r, q
    ("bf16", 300, 100, 200, 4, 1, 20, 12),
    ("bf16", 517, 90, 150, 6, 2, 30, 10),
    ("f32", 257, 101, 203, 5, 2, 17, 9),
    ("f32", 64, 7, 9, 3, 1, 0, 5),            # tiny, no shared basis
]


def _layer(dt, T, D, H, E, k, r, q, seed):
    cfg = synth.LayerConfig("unaligned", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dt, seed=seed,
                            residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(seed + 1)
    L["b1"] = (0.1 * rng.standard_normal(H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    return L


def _check(L, g, ref):
    k, dt = L["cfg"].k, L["cfg"].dtype
    tie = bound_excluded(oracle.margins(ref["logits"], k) < MARGIN)
    if "cls" in ref:
        tie &= ~ref["cls"]
    ok = ~tie
    assert np.array_equal(g["idx"][ok], ref["idx"][ok])
    if dt == "f32":
        assert max_rel(g["y"][ok], ref["y"][ok]) <= F32_MAXREL
    else:
        e = frob_rel(g["y"][ok], ref["y"][ok])
        assert e <= BF16_FROB_REGRESS, e
        assert_elementwise(g["y"][ok], ref["y"][ok], "bf16")
    assert np.all(np.isfinite(g["y"]))


@pytest.mark.parametrize("dt,T,D,H,E,k,r,q", CASES)
def test_unaligned_layer(dt, T, D, H, E, k, r, q):
    L = _layer(dt, T, D, H, E, k, r, q, seed=T + D)
    s = cm.make_shape(T, D, E, k, cm.BF16 if dt == "bf16" else cm.F32, H=H, r=r, q=q)
    assert cm.workspace_bytes(s) > 0
    g = gpu_ffn(L)
    _check(L, g, oracle.ffn_forward_layer(L))


def test_unaligned_with_class_tokens_and_mlp_router():
    L = _layer("bf16", 600, 196, 390, 5, 1, 60, 20, seed=11)
    C = synth.with_class_tokens(L, stride=50)
    g = gpu_ffn_ex(C)
    _check(C, g, oracle.ffn_forward_layer(C))
    M = synth.with_mlp_router(L, h=16, seed=2)
    g = gpu_ffn_ex(M)
    _check(M, g, oracle.ffn_forward_layer(M))


def test_unaligned_into_the_fused_kernel():
    """D = 380, H = 1530, q = 30 pad to 384, 1536, 32: the padded layer runs
    the fused top-1 kernel with its class rows in the same launch."""
    L = _layer("bf16", 9000, 380, 1530, 4, 1, 128, 30, seed=5)
    C = synth.with_class_tokens(L, stride=197)
    cm.timing_start(cm.stage_names(), max_records=64)
    try:
        g = gpu_ffn_ex(C)
    finally:
        t = cm.timing_stop()
    assert t.get("fused_top1", (0, 0))[1] == 1, t
    T = C["cfg"].T
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([np.arange(0, T, 197), rng.choice(T, 300, replace=False)]))
    ref = oracle.ffn_forward_layer(C, rows=rows)
    lg = oracle.router_logits(C["x"][rows], C["Wg"], C["bg"])
    ok = ref["cls"] | ~bound_excluded(oracle.margins(lg, 1) < MARGIN)
    assert np.array_equal(g["idx"][rows][ok], ref["idx"][ok])
    e = frob_rel(g["y"][rows][ok], ref["y"][ok])
    assert e <= BF16_FROB_REGRESS, e


@pytest.mark.parametrize("dt,T,D,H", [("bf16", 333, 100, 250), ("f32", 70, 33, 45)])
def test_unaligned_dense_ffn(dt, T, D, H):
    rng = np.random.default_rng(T)
    x = rng.standard_normal((T, D)).astype(np.float32)
    W1 = (0.05 * rng.standard_normal((H, D))).astype(np.float32)
    W2 = (0.05 * rng.standard_normal((D, H))).astype(np.float32)
    b1 = (0.1 * rng.standard_normal(H)).astype(np.float32)
    b2 = (0.1 * rng.standard_normal(D)).astype(np.float32)
    if dt == "bf16":
        x, W1, W2 = (synth.to_bf16_bits(a) for a in (x, W1, W2))
    y = cm.dense_ffn_forward(dev(x), dev(W1), dev(b1), dev(W2), dev(b2))
    torch.cuda.synchronize()
    got = oracle.widen(cm.to_stored(y))
    ref = oracle.dense_fc2(oracle.fc1_gelu(x, W1, b1), W2, b2)
    if dt == "f32":
        assert max_rel(got, ref) <= F32_MAXREL
    else:
        assert frob_rel(got, ref) <= BF16_FROB_REGRESS


@pytest.mark.parametrize("dt,T,D,E,k", [
    ("bf16", 3001, 60, 8, 2),       # 64-token histogram tiles, inline scan
    ("f32", 1500, 30, 5, 1),
    ("bf16", 70001, 100, 8, 2),     # 256-token tiles, chunked scan
])
def test_unaligned_route_dispatch_combine(dt, T, D, E, k):
    """Routing on padded copies of x and Wg, dispatch with element-wise row
    copies and the element-wise gated combine (D not a multiple of the
    elements of a 16-byte piece): routing bit-exact (near ties excluded),
    gates within 2e-5, the dispatch bit-exact against the oracle's of the
    same indices, every copied row bit for bit, and the combine of the
    copied rows (identity experts) against the oracle's combine."""
    L = synth.make_dispatch(T=T, D=D, E=E, k=k, dtype=dt, seed=T + D)
    x, Wg, bg = dev(L["x"]), dev(L["Wg"]), dev(L["bg"])
    s = cm.make_shape(T, D, E, k, cm.BF16 if dt == "bf16" else cm.F32)
    ws = cm.alloc_workspace(s)
    idx, gate = cm.route(x, Wg, bg, k, ws=ws)
    counts, offsets, perm, inv, xperm = cm.dispatch(idx, E, ws=ws, x=x, hist_in_ws=True)
    y = cm.combine(xperm, inv, gate)
    torch.cuda.synchronize()
    idx_np, gate_np = idx.cpu().numpy(), gate.cpu().numpy()
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    tie = assert_routing(idx_np, lg, k)
    assert_gates(gate_np, lg, idx_np, k, tie)
    perm_np, inv_np = perm.cpu().numpy(), inv.cpu().numpy()
    check_dispatch(idx_np, E, counts.cpu().numpy(), offsets.cpu().numpy(), perm_np, inv_np)
    xs = cm.to_stored(x)
    rows = cm.to_stored(xperm)
    assert np.array_equal(rows, xs[perm_np // k])
    ref = oracle.combine(rows, inv_np, gate_np, k)
    got = oracle.widen(cm.to_stored(y))
    bound = (2.0 ** -8 if dt == "bf16" else 1e-6) * np.abs(ref) + 1e-6
    assert np.all(np.abs(got - ref) <= bound)


def test_unaligned_route_ex_mlp_and_adaptive():
    """route_ex with D = 60: the MLP router (its Wh padded) and the adaptive
    router, against the oracle."""
    L = synth.make_dispatch(T=2000, D=60, E=6, k=2, dtype="bf16", seed=3)
    lay = {"x": L["x"], "Wg": L["Wg"], "bg": L["bg"],
           "cfg": synth.LayerConfig("u", T=2000, D=60, H=8, E=6, k=2, r=0, q=0, dtype="bf16", seed=3)}
    M = synth.with_mlp_router(lay, h=16, seed=5)
    r, keep = gpu_router(M)
    s = cm.make_shape(2000, 60, 6, 2, cm.BF16)
    idx, gate = cm.route_ex(dev(L["x"]), r, 6, 2, ws=cm.alloc_workspace(s))
    torch.cuda.synchronize()
    lg, _ = oracle.mlp_router_logits(L["x"], M["router"]["Wh"], M["router"]["bh"], M["Wg"], M["bg"], "bf16")
    tie = assert_routing(idx.cpu().numpy(), lg, 2)
    assert_gates(gate.cpu().numpy(), lg, idx.cpu().numpy(), 2, tie)
    del keep
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    tau = float(np.quantile(oracle.confidence(lg), 0.5))
    A = dict(lay, router={"kind": "adaptive", "tau": tau})
    r, keep = gpu_router(A)
    idx, gate = cm.route_ex(dev(L["x"]), r, 6, 2, ws=cm.alloc_workspace(s))
    torch.cuda.synchronize()
    i_ref, g_ref = oracle.adaptive_topk(lg, tau)
    ok = ~bound_excluded((oracle.margins(lg, 2) < MARGIN) | (confidence_gap(lg, tau) < 1e-9))
    assert np.array_equal(idx.cpu().numpy()[ok], i_ref[ok])
    assert np.all(np.abs(gate.cpu().numpy()[ok] - g_ref[ok]) <= 2e-5)
    del keep
