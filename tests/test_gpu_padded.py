"""GPU parity of the padded batched backend (clearmoe_ffn_forward_padded),
through the C ABI, against the fp64 oracle and against the grouped backend.

The padded backend pads every expert's sub-batch to the largest one and runs
the residual products over the whole padded batch (the paper's cuBLAS-style
dispatch backend, Sec. III "Dispatch Backends").  Its result must not depend
on the padding: y matches the oracle to the same bar as the grouped path, and
for k > 1, where both backends run the same products row by row, y is
bit-identical to clearmoe_ffn_forward's.  Cases cover balanced and skewed
loads, the imbalance recipe of the dispatch benchmark, empty experts, every
token on one expert (the largest padded batch, E * T * k rows), ragged tails
and a single token.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth
from tests.parity_util import (BF16_FROB_REGRESS, F32_MAXREL, assert_gates, assert_routing,
                               frob_rel, gpu_ffn, max_rel)

pytestmark = pytest.mark.gpu

PADDED_LAYERS = [
    # T, D, H, E, k, r, q, dtype, imbalance (None = uniform mixture)
    (1, 64, 128, 2, 1, 32, 8, "f32", None),
    (333, 96, 192, 4, 1, 32, 16, "f32", 0.8),
    (517, 128, 256, 5, 2, 64, 24, "f32", 0.4),
    (700, 384, 1536, 4, 1, 128, 32, "bf16", 0.6),
    (411, 192, 384, 8, 2, 64, 32, "bf16", None),
    (250, 64, 64, 3, 3, 0, 8, "bf16", 0.8),          # k = E, r = 0
    (300, 64, 128, 11, 2, 16, 8, "bf16", 0.4),       # top-2 beyond the pair order
]


def _layer(T, D, H, E, k, r, q, dt, imb, seed):
    mix = None if imb is None else synth.imbalance_mixture(E, imb)
    cfg = synth.LayerConfig("padded", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dt, seed=seed,
                            mixture=mix, residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(seed + 1)
    L["b1"] = (0.1 * rng.standard_normal(H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    return L


def _check_against_oracle(L, g):
    cfg = L["cfg"]
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(g["idx"], ref["logits"], cfg.k)
    assert_gates(g["gate"], ref["logits"], g["idx"], cfg.k, tie)
    ok = ~tie
    if cfg.dtype == "f32":
        e = max_rel(g["y"][ok], ref["y"][ok])
        assert e <= F32_MAXREL, e
    else:
        e = frob_rel(g["y"][ok], ref["y"][ok])
        assert e <= BF16_FROB_REGRESS, e
    assert np.all(np.isfinite(g["y"]))


@pytest.mark.parametrize("T,D,H,E,k,r,q,dt,imb", PADDED_LAYERS)
def test_padded_against_oracle(T, D, H, E, k, r, q, dt, imb):
    L = _layer(T, D, H, E, k, r, q, dt, imb, seed=T + D + 7 * E)
    g = gpu_ffn(L, padded=True)
    _check_against_oracle(L, g)
    # same routing as the grouped backend.  For k > 1 the grouped backend
    # forms h_sh and h_res apart like the padded one (same y, bit for bit),
    # except for top-2 with E (E + 1) / 2 <= 64, which runs in expert-pair
    # order (one product per pair segment): there the two agree to the bars.
    grouped = gpu_ffn(L)
    assert np.array_equal(g["idx"], grouped["idx"])
    assert np.array_equal(g["gate"], grouped["gate"])
    if k == 2 and E * (E + 1) // 2 <= 64:
        if dt == "f32":
            assert max_rel(g["y"], grouped["y"]) <= F32_MAXREL
        else:
            assert frob_rel(g["y"], grouped["y"]) <= BF16_FROB_REGRESS
    elif k > 1:
        assert np.array_equal(g["y"], grouped["y"])


@pytest.mark.parametrize("mode", ["one_expert", "empty_experts"])
@pytest.mark.parametrize("k", [1, 2])
def test_padded_skewed_routing(mode, k):
    L = _layer(700, 128, 256, 5, k, 32, 16, "f32", None, seed=19 + k)
    bg = np.zeros(5, np.float32)
    if mode == "one_expert":
        bg[2] = 1e4          # slot 0 of every token on expert 2: C = T, 5 T padded rows
    else:
        bg[[0, 3]] = -1e4    # two empty sub-batches (all padding)
    L["bg"] = bg
    g = gpu_ffn(L, padded=True)
    ref = oracle.ffn_forward_layer(L)
    assert np.array_equal(g["idx"], ref["idx"])
    assert max_rel(g["y"], ref["y"]) <= F32_MAXREL


def test_padded_stages_and_reuse_of_workspace():
    """One pad-index launch, the residual products over the padded batch, and
    no grouped top-1 stages; a workspace reused across calls with different
    routing gives each call's own result (padding rows are rewritten)."""
    L1 = _layer(300, 128, 256, 4, 1, 64, 16, "bf16", 0.8, seed=3)
    L2 = _layer(300, 128, 256, 4, 1, 64, 16, "bf16", None, seed=4)
    cm.timing_start(cm.stage_names(), max_records=64)
    try:
        gpu_ffn(L1, padded=True)
    finally:
        t = cm.timing_stop()
    launched = {k: v[1] for k, v in t.items() if v[1] > 0}
    assert launched.get("pad_index") == 1 and launched.get("res_h") == 1, launched
    for s in ("fused_top1", "tu_grouped", "y_grouped"):
        assert s not in launched, launched
    s = cm.make_shape(300, 128, 4, 1, cm.BF16, H=256, r=64, q=16)
    ws = torch.empty(cm.padded_workspace_bytes(s), dtype=torch.uint8, device="cuda")
    a1 = gpu_ffn(L1, ws=ws, padded=True)
    a2 = gpu_ffn(L2, ws=ws, padded=True)
    b2 = gpu_ffn(L2, padded=True)
    _check_against_oracle(L1, a1)
    assert np.array_equal(a2["y"], b2["y"])


def test_padded_deterministic():
    L = _layer(2000, 384, 1536, 8, 2, 128, 32, "bf16", 0.6, seed=23)
    a, b = gpu_ffn(L, padded=True), gpu_ffn(L, padded=True)
    assert np.array_equal(a["y"], b["y"])
