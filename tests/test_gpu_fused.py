"""GPU parity of the fused top-1 bf16 layer (fc1 + GELU, [t|u] and y in one
kernel), through the C ABI, against the fp64 oracle.

Shapes sweep the kernel's edges: token counts that leave ragged 64-row tiles
in every expert segment, widths D that are not multiples of 64 (padded input
groups), hidden widths H that are not multiples of the 4 x 64 round (waves with
partial or no slices), every count of 32-row [t|u] tiles (1 to 5), q = 0,
r = 0, the widest D (x rows beyond 64 KB of LDS), and small batches whose
tiles split their hidden units over 2 to 8 workgroups.  The GELU test isolates
the activation (W1, Vt and US identities) and checks it against the exact erf
form to the bound of the published approximation the kernels use.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth
from tests.parity_util import (BF16_FROB_REGRESS, F32_MAXREL, assert_gates, assert_routing,
                               dev, frob_rel, gpu_ffn, max_rel)

pytestmark = pytest.mark.gpu

FUSED_LAYERS = [
    # T, D, H, E, r, q
    (1, 64, 128, 2, 32, 8),          # one token, NFT = 2
    (63, 64, 64, 1, 32, 0),          # one expert, q = 0, NFT = 1
    (65, 128, 256, 3, 64, 16),       # NFT = 3
    (700, 384, 1536, 8, 128, 32),    # DeiT-S widths, NFT = 5
    (517, 200, 200, 5, 96, 24),      # D, H off the 64 / 256 grids, NFT = 4
    (300, 192, 136, 4, 0, 24),       # r = 0 (residual only), odd input-group count, idle waves
    (250, 96, 8, 3, 0, 8),           # H = 8: one partial slice in wave 0 only (r, q <= H)
    (411, 256, 512, 6, 128, 32),     # rq = 160, NFT = 5, D = 256 (two input groups of zeros)
    (129, 384, 3072, 4, 128, 32),    # widest fused D, H = 3072: x rows + b1 beyond 64 KB of LDS
    (129, 768, 3072, 4, 128, 32),    # D > 384: the GEMM chain takes the layer
    (20000, 128, 256, 20, 64, 16),   # E > 16: 79 router tiles, the in-kernel scans cross rows and waves
    (5000, 64, 128, 64, 32, 8),      # E = 64, the most experts: expert totals over a whole wave
    # small batches: each tile's hidden units split over S workgroups
    (300, 128, 1024, 4, 32, 0),      # S = 4, NFT = 1
    (200, 192, 768, 3, 64, 0),       # S = 3, NFT = 2
    (150, 64, 2048, 2, 64, 32),      # S = 8, NFT = 3
    (260, 200, 1000, 5, 96, 24),     # S = 4, NFT = 4, the last slot partial
    (1, 64, 2048, 2, 32, 8),         # S = 8, one token: one tile with rows, two empty
    (1568, 384, 1536, 8, 128, 32),   # S = 6: eight images of DeiT-S tokens
]


def _layer(T, D, H, E, r, q, seed, residual="random"):
    cfg = synth.LayerConfig("fused", T=T, D=D, H=H, E=E, k=1, r=r, q=q, dtype="bf16",
                            seed=seed, residual=residual, n_cal=2000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(seed + 1)
    L["b1"] = (0.1 * rng.standard_normal(H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    return L


def _stages_of(L):
    cm.timing_start(cm.stage_names(), max_records=64)
    try:
        gpu_ffn(L)
    finally:
        t = cm.timing_stop()
    return {k: v[1] for k, v in t.items() if v[1] > 0}


@pytest.mark.parametrize("T,D,H,E,r,q", FUSED_LAYERS)
def test_fused_top1_against_oracle(T, D, H, E, r, q):
    L = _layer(T, D, H, E, r, q, seed=T + D + H)
    g = gpu_ffn(L)
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(g["idx"], ref["logits"], 1)
    assert_gates(g["gate"], ref["logits"], g["idx"], 1, tie)
    e = frob_rel(g["y"][~tie], ref["y"][~tie])
    assert e <= BF16_FROB_REGRESS, e
    # every row written and finite
    assert np.all(np.isfinite(g["y"]))


def test_sampled_timing_times_every_nth_launch():
    L = _layer(300, 128, 256, 4, 64, 16, seed=6)
    gpu_ffn(L)
    cm.timing_start(["fused_top1"], max_records=16, every=3)
    try:
        for _ in range(7):
            gpu_ffn(L)
    finally:
        t = cm.timing_stop()
    ms, n = t["fused_top1"]
    assert n == 3 and ms > 0, t                 # launches 0, 3 and 6


def test_fused_stage_replaces_the_gemm_chain():
    L = _layer(300, 128, 256, 4, 64, 16, seed=5)
    launched = _stages_of(L)
    assert launched.get("fused_top1") == 1, launched
    for s in ("fc1_gelu", "tu_grouped", "y_grouped", "basis_t", "res_u"):
        assert s not in launched, launched
    # r not a multiple of 32, or r + q above 160: the grouped-GEMM path (and
    # still parity)
    for shape, seed in (((300, 128, 256, 4, 48, 16), 6), ((411, 256, 512, 6, 160, 32), 7)):
        L = _layer(*shape, seed=seed)
        launched = _stages_of(L)
        assert "fused_top1" not in launched and launched.get("tu_grouped") == 1, launched
        g = gpu_ffn(L)
        ref = oracle.ffn_forward_layer(L)
        tie = assert_routing(g["idx"], ref["logits"], 1)
        assert frob_rel(g["y"][~tie], ref["y"][~tie]) <= BF16_FROB_REGRESS


@pytest.mark.parametrize("T,D,H,E,r,q", [(20000, 128, 256, 20, 64, 16), (5000, 64, 128, 64, 32, 8),
                                          (12608, 128, 256, 16, 64, 16)])
def test_fused_kernel_dispatches_in_its_prologue(T, D, H, E, r, q):
    # router histogram small enough for the kernel's own dispatch: no
    # permute launch, and the fused kernel's result still matches the oracle
    # (the E = 16 case has 197 router tiles of 64 tokens, the others 256)
    L = _layer(T, D, H, E, r, q, seed=T + E)
    launched = _stages_of(L)
    assert launched.get("fused_top1") == 1 and "permute" not in launched, launched
    g = gpu_ffn(L)
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(g["idx"], ref["logits"], 1)
    assert frob_rel(g["y"][~tie], ref["y"][~tie]) <= BF16_FROB_REGRESS


@pytest.mark.parametrize("mode", ["one_expert", "empty_experts"])
def test_fused_skewed_routing(mode):
    L = _layer(700, 128, 256, 5, 32, 16, seed=9)
    bg = np.zeros(5, np.float32)
    if mode == "one_expert":
        bg[2] = 1e4                       # every token to expert 2: 11 tiles of one segment
    else:
        bg[[0, 3]] = -1e4                 # two empty segments
    L["bg"] = bg
    g = gpu_ffn(L)
    ref = oracle.ffn_forward_layer(L)
    assert np.array_equal(g["idx"], ref["idx"])
    assert frob_rel(g["y"], ref["y"]) <= BF16_FROB_REGRESS


@pytest.mark.parametrize("T", [1000, 12608])
def test_fused_deterministic(T):
    # T = 1000: hidden split (partials summed in part order whatever the
    # order the parts finish in); T = 12608: one workgroup per tile
    L = _layer(T, 384, 1536, 8, 128, 32, seed=21)
    a, b = gpu_ffn(L), gpu_ffn(L)
    assert np.array_equal(a["y"], b["y"])


def test_fused_split_reuses_a_dirty_workspace():
    # the split's arrival counters and partials live in the caller's
    # workspace: filled with 0xFF first, then reused by three calls (each
    # leaves its counters at S), every result the same and at the oracle
    L = _layer(700, 384, 1536, 8, 128, 32, seed=23)
    shape = cm.make_shape(700, 384, 8, 1, cm.BF16, H=1536, r=128, q=32)
    ws = cm.alloc_workspace(shape)
    ws.fill_(255)
    outs = [gpu_ffn(L, ws=ws)["y"] for _ in range(3)]
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(gpu_ffn(L, ws=ws)["idx"], ref["logits"], 1)
    assert frob_rel(outs[0][~tie], ref["y"][~tie]) <= BF16_FROB_REGRESS


def _gelu_exact(v):
    return np.array([0.5 * t * (1.0 + math.erf(t / math.sqrt(2.0))) for t in v.ravel()]).reshape(
        v.shape)


def _identity_layer(dt, T, D, seed):
    """E = 1, W1 = I, Vt = I, US = I, P = Q = 0, biases 0: y = GELU(x) exactly
    as the kernel evaluates it (every product is by 1 or 0)."""
    rng = np.random.default_rng(seed)
    x = np.linspace(-8.0, 8.0, T * D).astype(np.float32)
    x = x[rng.permutation(T * D)].reshape(T, D)
    eye = np.eye(D, dtype=np.float32)
    st = (lambda a: synth.to_bf16_bits(a)) if dt == "bf16" else (lambda a: a)
    q = 8
    L = dict(x=st(x), W1=st(eye), b1=np.zeros(D, np.float32), US=st(eye), Vt=st(eye),
             b2=np.zeros(D, np.float32), P=st(np.zeros((1, D, q), np.float32)),
             Q=st(np.zeros((1, q, D), np.float32)), Wg=st(np.zeros((1, D), np.float32)),
             bg=np.zeros(1, np.float32),
             cfg=synth.LayerConfig("gelu", T=T, D=D, H=D, E=1, k=1, r=D, q=q, dtype=dt,
                                   seed=seed))
    return L, (synth.bf16_bits_to_f32(st(x)) if dt == "bf16" else x)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_gelu_matches_exact_erf(dt):
    """The erf of Abramowitz & Stegun 7.1.26 is within 1.5e-7 of the exact
    one, so GELU is within 0.5 |v| 1.5e-7 (plus float32 rounding).
    fp32 (GEMM epilogue): |y - GELU(v)| within that bound.
    bf16 (fused kernel): y is the bf16 rounding of a value within that bound,
    and bit-identical to the bf16 rounding of the fp32 path's GELU of the same
    inputs (no extra rounding anywhere on the fused path)."""
    L, xv = _identity_layer(dt, 512, 64, seed=4)
    g = gpu_ffn(L)
    ref = _gelu_exact(xv.astype(np.float64))
    got = g["y"].astype(np.float64)
    bound = 0.5 * np.abs(xv.astype(np.float64)) * 1.5e-7 + 4 * np.finfo(np.float32).eps * np.abs(ref)
    if dt == "f32":
        assert np.all(np.abs(got - ref) <= bound), float(np.max(np.abs(got - ref) - bound))
    else:
        # rounding to bf16 (8 significant bits) moves a value w by at most 2^-8 |w|
        assert np.all(np.abs(got - ref) <= bound + 2.0 ** -8 * (np.abs(ref) + bound))
        Lf, _ = _identity_layer("f32", 512, 64, seed=4)
        Lf["x"] = xv.astype(np.float32)
        yf = gpu_ffn(Lf)["y"].astype(np.float32)
        assert np.array_equal(g["y"], synth.bf16_bits_to_f32(synth.to_bf16_bits(yf)))
    assert ("fused_top1" in _stages_of(L)) == (dt == "bf16")
