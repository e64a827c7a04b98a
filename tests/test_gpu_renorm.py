"""GPU parity with the unrenormalised gates (shape field renorm = 0): each
chosen expert's gate is its probability under the softmax over all E logits
(Sec. III Phase 4 reads the router as a distribution over the experts).
Routing is the same as with renormalised gates, bit for bit; gates within
2e-5 of the oracle's double gates; y against the oracle's layer with those
gates (residual experts that differ, so a wrong gate shows).  Paths: the
router alone (linear, both dtypes, k = 1, 2, 3), the fused top-1 layer (with
and without the hidden split), the top-2 pair order, the float32 GEMM chain
with the combine (E > 10), the padded backend, the adaptive router (a token
kept on one expert gets its confidence as gate) and the MLP router."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

from parity_util import (BF16_FROB_REGRESS, F32_MAXREL, MARGIN, assert_elementwise, assert_gates,
                         assert_routing, bound_excluded, confidence_gap, dev, frob_rel, gpu_ffn,
                         gpu_ffn_ex, max_rel)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt,k", [("bf16", 1), ("bf16", 2), ("f32", 2), ("bf16", 3)])
def test_route_full_softmax_gates(dt, k):
    L = synth.make_dispatch(T=3000, D=384, E=8, k=k, dtype=dt, seed=31 + k)
    x, Wg, bg = dev(L["x"]), dev(L["Wg"]), dev(L["bg"])
    idx0, g0 = cm.route(x, Wg, bg, k, renorm=0)
    idx1, g1 = cm.route(x, Wg, bg, k, renorm=1)
    torch.cuda.synchronize()
    idx0, g0, idx1, g1 = (t.cpu().numpy() for t in (idx0, g0, idx1, g1))
    assert np.array_equal(idx0, idx1)          # the choice does not depend on the gate rule
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    tie = assert_routing(idx0, lg, k)
    assert_gates(g0, lg, idx0, k, tie, renorm=0)
    assert_gates(g1, lg, idx1, k, tie, renorm=1)
    s = g0.sum(axis=1)
    assert np.all(s <= 1.0 + 1e-6) and np.all(s > 0.0)


def _layer(dt, T, D, H, E, k, r, q, seed):
    cfg = synth.LayerConfig("renorm0", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dt, seed=seed,
                            residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    L["renorm"] = 0
    return L


def _check(L, g, extra_excl=None):
    k, dt = L["cfg"].k, L["cfg"].dtype
    ref = oracle.ffn_forward_layer(L)
    tie = bound_excluded(oracle.margins(ref["logits"], k) < MARGIN)
    if extra_excl is not None:
        tie |= extra_excl
    ok = ~tie
    assert np.array_equal(g["idx"][ok], ref["idx"][ok])
    assert np.all(np.abs(g["gate"][ok] - ref["gate"][ok]) <= 2e-5)
    if dt == "f32":
        assert max_rel(g["y"][ok], ref["y"][ok]) <= F32_MAXREL
    else:
        e = frob_rel(g["y"][ok], ref["y"][ok])
        assert e <= BF16_FROB_REGRESS, e
        assert_elementwise(g["y"][ok], ref["y"][ok], "bf16")
    return ref


LAYERS = [
    # dt, T, D, H, E, k, r, q: the path it takes
    ("bf16", 2000, 384, 1536, 8, 1, 128, 32),      # fused top-1 with the hidden split
    ("bf16", 9000, 384, 1536, 8, 1, 128, 32),      # fused top-1, one workgroup per tile, own dispatch
    ("bf16", 3000, 256, 1024, 8, 2, 64, 32),       # top-2 in pair order
    ("f32", 1500, 128, 512, 12, 2, 32, 16),        # E > 10: float32 GEMM chain and the combine
    ("bf16", 1200, 128, 512, 6, 3, 32, 16),        # k = 3: GEMM chain and the combine
]


@pytest.mark.parametrize("dt,T,D,H,E,k,r,q", LAYERS)
def test_layer_full_softmax_gates(dt, T, D, H, E, k, r, q):
    L = _layer(dt, T, D, H, E, k, r, q, seed=T + E)
    g = gpu_ffn(L)
    ref = _check(L, g)
    # the gate rule matters here: the renormalised gates' y fails the bar
    y1 = oracle.ffn_forward_layer(dict(L, renorm=1))["y"]
    if dt == "f32":
        assert max_rel(y1, ref["y"]) > 100 * F32_MAXREL
    else:
        assert frob_rel(y1, ref["y"]) > BF16_FROB_REGRESS


def test_padded_backend_full_softmax_gates():
    L = _layer("bf16", 2500, 256, 1024, 4, 2, 64, 32, seed=77)
    g = gpu_ffn(L, padded=True)
    _check(L, g)


def test_adaptive_router_full_softmax_gates():
    """A token kept on one expert gets its confidence as gate (not 1); an
    escalated one its two probabilities."""
    L = _layer("bf16", 4000, 384, 1536, 8, 1, 128, 32, seed=91)
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    tau = float(np.quantile(oracle.confidence(lg), 0.3))
    A = synth.with_adaptive_router(L, tau)
    g = gpu_ffn_ex(A)
    ref = _check(A, g, extra_excl=bound_excluded(confidence_gap(lg, tau) < 1e-9))
    one = ref["idx"][:, 1] < 0
    assert 0 < one.sum() < len(one)
    assert np.all(ref["gate"][one, 0] < 1.0)


def test_mlp_router_full_softmax_gates():
    L = _layer("bf16", 3000, 384, 1536, 8, 2, 128, 32, seed=55)
    M = synth.with_mlp_router(L, h=64, seed=3)
    M["renorm"] = 0
    g = gpu_ffn_ex(M)
    _check(M, g)


def test_class_tokens_in_the_fused_launch_full_softmax_gates():
    """renorm = 0 with class tokens: the dispatch kernels order the expert
    tokens (the fused kernel's own dispatch assumes gates of 1) and the class
    rows still run inside the fused launch (one workgroup per tile)."""
    L = _layer("bf16", 9000, 384, 1536, 8, 1, 128, 32, seed=21)
    C = synth.with_class_tokens(L, stride=197)
    C["renorm"] = 0
    cm.timing_start(cm.stage_names(), max_records=64)
    try:
        g = gpu_ffn_ex(C)
    finally:
        t = cm.timing_stop()
    assert t.get("fused_top1", (0, 0))[1] == 1 and t.get("permute", (0, 0))[1] >= 1, t
    ref = oracle.ffn_forward_layer(C)
    tie = bound_excluded(oracle.margins(ref["logits"], 1) < MARGIN) & ~ref["cls"]
    ok = ~tie
    assert np.array_equal(g["idx"][ok], ref["idx"][ok])
    assert np.all(np.abs(g["gate"][ok] - ref["gate"][ok]) <= 2e-5)
    e = frob_rel(g["y"][ok], ref["y"][ok])
    assert e <= BF16_FROB_REGRESS, e
    assert_elementwise(g["y"][ok], ref["y"][ok], "bf16")


def test_unaligned_layer_full_softmax_gates():
    """An unaligned shape (padded copies) keeps the gate rule."""
    L = _layer("bf16", 700, 100, 250, 5, 2, 20, 12, seed=8)
    g = gpu_ffn(L)
    _check(L, g)
