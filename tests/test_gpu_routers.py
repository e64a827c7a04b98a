"""GPU parity of the router variants (Sec. III Phase 4: Linear, MLP and
Adaptive routers) and of empty dispatch slots, through the C ABI, against the
CPU oracle on seeded inputs.

Exclusions from the bit-exact routing comparison, each a decision that
floating point takes at a boundary:
  * top-k margin below 1e-6 (as for the linear router);
  * adaptive: |log p - log tau| below 1e-9, p the oracle's confidence;
  * MLP: a hidden value within 1e-12 (relative to its binade) of a rounding
    midpoint of the storage type, where double rounding order may flip the
    one rounding both sides take.
Everything else (indices, empty slots, counts, offsets, permutations) is
compared bit for bit; gates within 2e-5; layer outputs at the bf16 / f32 bars.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

from parity_util import (bound_excluded, BF16_FROB_REGRESS, F32_MAXREL, MARGIN, check_dispatch, confidence_gap,
                         dev, frob_rel, gpu_ffn_ex, gpu_router, max_rel, rounding_gap)

pytestmark = pytest.mark.gpu

CONF_GAP = 1e-9
ROUND_GAP = 1e-12


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    cm.lib()
    yield
    torch.cuda.synchronize()


def _route_gpu(L, k):
    r, keep = gpu_router(L)
    T, D = L["x"].shape
    E = L["Wg"].shape[0]
    s = cm.make_shape(T, D, E, k, cm.F32 if L["x"].dtype == np.float32 else cm.BF16)
    ws = cm.alloc_workspace(s)
    x = dev(L["x"])
    idx, gate = cm.route_ex(x, r, E, k, ws=ws)
    counts, offsets, perm, inv, xperm = cm.dispatch(idx, E, ws=ws, x=x, hist_in_ws=True)
    torch.cuda.synchronize()
    del keep
    return (idx.cpu().numpy(), gate.cpu().numpy(), counts.cpu().numpy(), offsets.cpu().numpy(),
            perm.cpu().numpy(), inv.cpu().numpy(), cm.to_stored(xperm))


def _compare_choice(idx, gate, idx_ref, gate_ref, excluded):
    ok = ~excluded
    bad = np.any(idx != idx_ref, axis=1) & ok
    assert not bad.any(), f"{bad.sum()} tokens chose differently (first {np.nonzero(bad)[0][:5]})"
    assert np.all(np.abs(gate[ok] - gate_ref[ok]) <= 2e-5), float(np.abs(gate[ok] - gate_ref[ok]).max())
    # an empty slot is exactly (-1, 0), and only slot 1 can be empty
    empty = idx == -1
    assert not empty[:, 0].any()
    assert np.all(gate[empty] == 0.0)
    assert np.all(gate[empty[:, 1], 0] == 1.0)


def _check_dispatch_and_rows(L, k, idx, counts, offsets, perm, inv, xperm):
    E = L["Wg"].shape[0]
    check_dispatch(idx, E, counts, offsets, perm, inv)
    n = int(offsets[-1])
    assert np.array_equal(xperm[:n], L["x"][perm[:n] // k])


# ------------------------------------------------------------- adaptive ----
ADAPTIVE_CASES = [
    # dtype, T, D, E, quantile of the confidence used as tau
    ("bf16", 1, 8, 2, 0.5), ("bf16", 257, 64, 4, 0.3), ("bf16", 1000, 384, 8, 0.5),
    ("bf16", 700, 136, 13, 0.7), ("bf16", 600, 64, 40, 0.5),
    ("f32", 513, 192, 4, 0.4), ("f32", 300, 100, 6, 0.6),
]


@pytest.mark.parametrize("dt,T,D,E,qt", ADAPTIVE_CASES)
def test_adaptive_linear_router(dt, T, D, E, qt):
    L = synth.make_dispatch(T=T, D=D, E=E, k=2, dtype=dt, seed=T + 3 * E)
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    tau = float(np.quantile(oracle.confidence(lg), qt))
    L["router"] = {"kind": "adaptive", "tau": tau}
    idx, gate, counts, offsets, perm, inv, xperm = _route_gpu(L, 2)
    idx_ref, gate_ref = oracle.adaptive_topk(lg, tau)
    excl = bound_excluded((oracle.margins(lg, 2) < MARGIN) | (confidence_gap(lg, tau) < CONF_GAP))
    _compare_choice(idx, gate, idx_ref, gate_ref, excl)
    if T > 100:                                    # both outcomes are exercised
        assert 0 < (idx[:, 1] == -1).sum() < T
    _check_dispatch_and_rows(L, 2, idx, counts, offsets, perm, inv, xperm)
    assert np.all(perm[offsets[-1]:] == -1)


@pytest.mark.parametrize("tau,top1", [(0.0, True), (-3.0, True), (1.5, False)])
def test_adaptive_threshold_limits(tau, top1):
    """tau <= 1/E: nobody escalates (p >= 1/E always); tau > 1: everybody
    takes the plain top-2."""
    L = synth.make_dispatch(T=333, D=64, E=5, k=2, dtype="bf16", seed=9)
    L["router"] = {"kind": "adaptive", "tau": tau}
    idx, gate, counts, offsets, perm, inv, _ = _route_gpu(L, 2)
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    if top1:
        assert np.all(idx[:, 1] == -1) and np.all(gate[:, 0] == 1.0)
        i1, _ = oracle.topk(lg, 1)
        ok = ~bound_excluded(oracle.margins(lg, 1) < MARGIN)
        assert np.array_equal(idx[ok, 0], i1[ok, 0])
        assert offsets[-1] == 333 and np.all(perm[333:] == -1)
    else:
        i2, g2 = oracle.topk(lg, 2)
        ok = ~bound_excluded(oracle.margins(lg, 2) < MARGIN)
        assert np.array_equal(idx[ok], i2[ok])
        assert np.all(np.abs(gate[ok] - g2[ok]) <= 2e-5)
        assert offsets[-1] == 666
    check_dispatch(idx, 5, counts, offsets, perm, inv)


def test_adaptive_exact_ties_and_threshold_on_integers():
    """Integer inputs: every double sum is exact on both sides, so tied logits
    are decided by the index rule alone: all tokens bit-exact, ties included."""
    rng = np.random.default_rng(17)
    T, D, E = 640, 24, 3
    xf = rng.integers(-2, 3, size=(T, D)).astype(np.float32)
    wf = rng.integers(-1, 2, size=(E, D)).astype(np.float32)
    lg = oracle.router_logits(xf, wf, None)
    # tau halfway between two neighbouring confidence levels: integer logits
    # give a few distinct levels, far apart, so every token is decided
    levels = np.unique(oracle.confidence(lg))
    i = len(levels) // 2
    tau = float(0.5 * (levels[i - 1] + levels[i]))
    L = {"x": synth.to_bf16_bits(xf), "Wg": synth.to_bf16_bits(wf), "bg": None,
         "router": {"kind": "adaptive", "tau": tau}}
    idx, gate, counts, offsets, perm, inv, _ = _route_gpu(L, 2)
    idx_ref, gate_ref = oracle.adaptive_topk(lg, tau)
    assert (oracle.margins(lg, 2) == 0).sum() > 20
    assert np.array_equal(idx, idx_ref)
    assert np.all(np.abs(gate - gate_ref) <= 2e-7)
    check_dispatch(idx, E, counts, offsets, perm, inv)


# ------------------------------------------------------------------ MLP ----
MLP_CASES = [
    # dtype, T, D, E, k, hidden
    ("bf16", 1, 64, 4, 1, 16), ("bf16", 255, 96, 4, 2, 16), ("bf16", 1000, 384, 8, 1, 64),
    ("bf16", 500, 384, 8, 2, 64), ("bf16", 300, 128, 20, 3, 40), ("bf16", 130, 64, 40, 2, 200),
    ("bf16", 99, 64, 3, 1, 256), ("f32", 257, 192, 4, 1, 32), ("f32", 400, 100, 6, 2, 17),
]


def _mlp_layer(dt, T, D, E, hidden, seed):
    cfg = synth.LayerConfig("mlp", T=T, D=D, H=max(64, D), E=E, k=1, r=8, q=8, dtype=dt,
                            seed=seed, n_cal=1000)
    L = synth.with_mlp_router(synth.make_layer(cfg), h=hidden, seed=seed)
    rng = np.random.default_rng(seed)
    L["router"]["bh"] = (0.2 * rng.standard_normal(hidden)).astype(np.float32)
    L["bg"] = (0.2 * rng.standard_normal(E)).astype(np.float32)
    return L


def _mlp_ref(L, dt):
    rt = L["router"]
    lg, _ = oracle.mlp_router_logits(L["x"], rt["Wh"], rt["bh"], L["Wg"], L["bg"], dt)
    pre = oracle.fc1_gelu(L["x"], rt["Wh"], rt["bh"])          # exact hidden values
    near = np.any(rounding_gap(pre, dt) < ROUND_GAP, axis=1)
    return lg, near


@pytest.mark.parametrize("dt,T,D,E,k,hidden", MLP_CASES)
def test_mlp_router(dt, T, D, E, k, hidden):
    L = _mlp_layer(dt, T, D, E, hidden, seed=T + hidden)
    lg, near = _mlp_ref(L, dt)
    idx, gate, counts, offsets, perm, inv, xperm = _route_gpu(L, k)
    idx_ref, gate_ref = oracle.topk(lg, k)
    excl = bound_excluded(near | (oracle.margins(lg, k) < MARGIN))
    assert excl.mean() < 0.01
    ok = ~excl
    assert np.array_equal(idx[ok], idx_ref[ok])
    assert np.all(np.abs(gate[ok] - gate_ref[ok]) <= 2e-5)
    _check_dispatch_and_rows(L, k, idx, counts, offsets, perm, inv, xperm)


def test_mlp_router_hidden_rounding_matters():
    """The hidden layer's rounding is visible in the logits: routing the same
    tokens with unrounded hidden values changes some near-tie choices, and the
    GPU follows the rounded (stored) definition."""
    L = _mlp_layer("bf16", 2000, 384, 8, 64, seed=5)
    lg, near = _mlp_ref(L, "bf16")
    rt = L["router"]
    exact = oracle.router_logits(oracle.fc1_gelu(L["x"], rt["Wh"], rt["bh"]),
                                 L["Wg"], L["bg"])
    assert np.max(np.abs(exact - lg)) > 1e-4                   # the rounding moves logits
    idx, *_ = _route_gpu(L, 1)
    ok = ~near & ~bound_excluded(oracle.margins(lg, 1) < MARGIN)
    assert np.array_equal(idx[ok, 0], oracle.topk(lg, 1)[0][ok, 0])


@pytest.mark.parametrize("qt", [0.3, 0.8])
def test_mlp_router_adaptive(qt):
    L = _mlp_layer("bf16", 700, 192, 6, 32, seed=21)
    lg, near = _mlp_ref(L, "bf16")
    tau = float(np.quantile(oracle.confidence(lg), qt))
    L["router"]["adaptive"] = True
    L["router"]["tau"] = tau
    idx, gate, counts, offsets, perm, inv, xperm = _route_gpu(L, 2)
    idx_ref, gate_ref = oracle.adaptive_topk(lg, tau)
    excl = bound_excluded(near | (oracle.margins(lg, 2) < MARGIN) | (confidence_gap(lg, tau) < CONF_GAP))
    _compare_choice(idx, gate, idx_ref, gate_ref, excl)
    assert 0 < (idx[:, 1] == -1).sum() < 700
    _check_dispatch_and_rows(L, 2, idx, counts, offsets, perm, inv, xperm)


# -------------------------------------------------------- empty slots ----
@pytest.mark.parametrize("T,E,k,p_empty", [(1, 3, 2, 1.0), (600, 5, 2, 0.5), (1300, 8, 3, 0.3),
                                           (513, 4, 2, 0.0), (300, 6, 2, 1.0)])
def test_dispatch_and_combine_with_empty_slots(T, E, k, p_empty):
    """-1 entries (empty slots) are in no sub-batch: counts, offsets, perm
    (with its -1 tail) and inv bit-exact against the oracle; rows copied only
    for real assignments; the gated combine skips empty slots."""
    rng = np.random.default_rng(T + E)
    idx_np = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    drop = rng.random((T, k)) < p_empty
    drop[:, 0] = False                                 # slot 0 always has an expert
    idx_np[drop] = -1
    D = 64
    xf = rng.standard_normal((T, D)).astype(np.float32)
    x = synth.to_bf16_bits(xf)
    counts, offsets, perm, inv, xperm = cm.dispatch(torch.from_numpy(idx_np).cuda(), E, x=dev(x))
    torch.cuda.synchronize()
    counts, offsets, perm, inv = (a.cpu().numpy() for a in (counts, offsets, perm, inv))
    check_dispatch(idx_np, E, counts, offsets, perm, inv)
    n = int(offsets[-1])
    assert n == int((idx_np >= 0).sum())
    xp = cm.to_stored(xperm)
    assert np.array_equal(xp[:n], x[perm[:n] // k])
    gate_np = rng.random((T, k)).astype(np.float32)
    gate_np[drop] = 0.0
    y = cm.combine(xperm, torch.from_numpy(inv).cuda(), torch.from_numpy(gate_np).cuda())
    torch.cuda.synchronize()
    ye = oracle.widen(xp)
    ye[n:] = 0.0                                       # rows past the assignments are unused
    ref = oracle.combine(ye, inv, gate_np, k)
    got = oracle.widen(cm.to_stored(y))
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6)


# ------------------------------------------------------- whole layer ----
LAYER_CASES = [
    # router, dtype, T, D, H, E, r, q, k, residual
    ("adaptive", "bf16", 300, 64, 192, 6, 32, 24, 2, "random"),
    ("adaptive", "f32", 257, 64, 128, 4, 16, 16, 2, "random"),
    ("adaptive", "bf16", 1000, 128, 256, 8, 64, 16, 2, "svd_tail"),
    ("mlp", "bf16", 400, 128, 256, 8, 64, 16, 1, "random"),      # top-1: the fused kernel
    ("mlp", "bf16", 333, 96, 192, 5, 32, 16, 2, "random"),
    ("mlp", "f32", 200, 64, 128, 4, 16, 8, 1, "random"),
]


@pytest.mark.parametrize("kind,dt,T,D,H,E,r,q,k,res", LAYER_CASES)
def test_ffn_forward_ex_small(kind, dt, T, D, H, E, r, q, k, res):
    cfg = synth.LayerConfig("rt", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dt, seed=T + E,
                            residual=res, n_cal=2000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(4)
    L["b1"] = (0.1 * rng.standard_normal(H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    if kind == "mlp":
        L = synth.with_mlp_router(L, h=max(16, D // 6), seed=3)
        lg, near = _mlp_ref(L, dt)
        excl = bound_excluded(near | (oracle.margins(lg, k) < MARGIN))
    else:
        lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
        tau = float(np.quantile(oracle.confidence(lg), 0.5))
        L = synth.with_adaptive_router(L, tau)
        excl = bound_excluded((oracle.margins(lg, 2) < MARGIN) | (confidence_gap(lg, tau) < CONF_GAP))
    g = gpu_ffn_ex(L)
    ref = oracle.ffn_forward_layer(L)
    ok = ~excl
    assert np.array_equal(g["idx"][ok], ref["idx"][ok])
    if kind == "adaptive":
        assert 0 < (g["idx"][:, 1] == -1).sum() < T
    if dt == "f32":
        assert max_rel(g["y"][ok], ref["y"][ok]) <= F32_MAXREL
    else:
        e = frob_rel(g["y"][ok], ref["y"][ok])
        assert e <= BF16_FROB_REGRESS, e


def test_adaptive_layer_isolates_residual():
    """US = 0 and random experts: y is the routed residual alone, so a wrong
    empty-slot decision or gate shows at the float32 bar."""
    cfg = synth.LayerConfig("ad", T=517, D=64, H=128, E=6, k=2, r=16, q=16, dtype="f32", seed=3,
                            residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    L["US"] = np.zeros_like(L["US"])
    lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
    tau = float(np.quantile(oracle.confidence(lg), 0.4))
    L = synth.with_adaptive_router(L, tau)
    g = gpu_ffn_ex(L)
    ref = oracle.ffn_forward_layer(L)
    ok = ~bound_excluded((oracle.margins(lg, 2) < MARGIN) | (confidence_gap(lg, tau) < CONF_GAP))
    assert np.array_equal(g["idx"][ok], ref["idx"][ok])
    assert max_rel(g["y"][ok], ref["y"][ok]) <= F32_MAXREL


def _sample_rows(T, n, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, T - 1], rng.choice(T, size=min(n, T), replace=False)]))


@pytest.mark.parametrize("kind", ["mlp", "adaptive"])
def test_router_variants_at_deit_small(kind):
    """The DeiT-Small-shaped layer (12608 tokens, D = 384, H = 1536, E = 8,
    r = 128, q = 32, bf16) with the MLP router (hidden d/6 = 64, top-1) or the
    adaptive router (tau at the 25 % confidence quantile): routing on every
    token, values on a sample of rows."""
    L = synth.make_layer(synth.CONFIGS["C2"])
    if kind == "mlp":
        L = synth.with_mlp_router(L, seed=1)
        lg, near = _mlp_ref(L, "bf16")
        k = 1
        excl = bound_excluded(near | (oracle.margins(lg, 1) < MARGIN))
    else:
        lg = oracle.router_logits(L["x"], L["Wg"], L["bg"])
        tau = float(np.quantile(oracle.confidence(lg), 0.25))
        L = synth.with_adaptive_router(L, tau)
        k = 2
        excl = bound_excluded((oracle.margins(lg, 2) < MARGIN) | (confidence_gap(lg, tau) < CONF_GAP))
    g = gpu_ffn_ex(L)
    idx_ref, _ = (oracle.topk(lg, 1) if kind == "mlp"
                  else oracle.adaptive_topk(lg, L["router"]["tau"]))
    ok = ~excl
    assert np.array_equal(g["idx"][ok], idx_ref[ok])
    rows = _sample_rows(L["cfg"].T, 256, 8)
    rows = rows[ok[rows]]
    ref = oracle.ffn_forward_layer(L, rows=rows)
    assert np.array_equal(ref["idx"], g["idx"][rows])
    e = frob_rel(g["y"][rows], ref["y"])
    assert e <= BF16_FROB_REGRESS, e
