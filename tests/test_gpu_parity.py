"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle on
the same seeded inputs.

Bars: routing indices, counts, offsets and permutations bit-exact (a token
whose top-k logit margin is below 1e-6 may route differently and is then
excluded from the value comparison); outputs within 1e-4 normwise max
relative error in float32 mode and 2e-2 relative Frobenius error in bfloat16
mode (with a 1e-2 internal regression bar).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

from parity_util import (BF16_FROB, BF16_FROB_REGRESS, F32_MAXREL, assert_elementwise, assert_gates,
                         assert_routing,
                         check_dispatch, dev, frob_rel, gpu_ffn, max_rel)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    cm.lib()
    yield
    torch.cuda.synchronize()


# ------------------------------------------------------------------ route ----
ROUTE_CASES = [
    # dtype, T, D, E, k
    ("bf16", 1, 8, 1, 1), ("bf16", 255, 72, 3, 2), ("bf16", 256, 64, 8, 1),
    ("bf16", 257, 384, 8, 2), ("bf16", 1000, 136, 13, 3), ("bf16", 700, 64, 64, 2),
    ("bf16", 300, 32, 5, 5), ("f32", 1, 4, 2, 2), ("f32", 513, 192, 4, 1),
    ("f32", 999, 100, 6, 2), ("f32", 260, 64, 17, 4),
]


@pytest.mark.parametrize("dt,T,D,E,k", ROUTE_CASES)
def test_route_and_dispatch(dt, T, D, E, k):
    L = synth.make_dispatch(T=T, D=D, E=E, k=k, dtype=dt, seed=T + E)
    x, Wg, bg = dev(L["x"]), dev(L["Wg"]), dev(L["bg"])
    s = cm.make_shape(T, D, E, k, cm.F32 if dt == "f32" else cm.BF16)
    ws = cm.alloc_workspace(s)
    idx, gate = cm.route(x, Wg, bg, k, ws=ws)
    counts, offsets, perm, inv, xperm = cm.dispatch(idx, E, ws=ws, x=x, hist_in_ws=True)
    torch.cuda.synchronize()
    idx_h, gate_h = idx.cpu().numpy(), gate.cpu().numpy()
    _, _, lg = oracle.route(L["x"], L["Wg"], L["bg"], k)
    tie = assert_routing(idx_h, lg, k)
    assert_gates(gate_h, lg, idx_h, k, tie)
    check_dispatch(idx_h, E, counts.cpu().numpy(), offsets.cpu().numpy(), perm.cpu().numpy(),
                   inv.cpu().numpy())
    # rows copied into expert order, byte for byte
    p = perm.cpu().numpy()
    assert np.array_equal(cm.to_stored(xperm), L["x"][p // k])
    # the histogram pass of dispatch (no route histogram) gives the same result
    c2, o2, p2, i2, _ = cm.dispatch(idx, E, D=D)
    torch.cuda.synchronize()
    assert torch.equal(c2, counts) and torch.equal(o2, offsets)
    assert torch.equal(p2, perm) and torch.equal(i2, inv)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("E,k", [(4, 1), (6, 2), (8, 3)])
def test_route_exact_ties_take_lower_index(dt, E, k):
    """Integer inputs make every double sum exact, so tied logits are exactly
    equal on both sides and the tie rule alone decides: all tokens bit-exact."""
    rng = np.random.default_rng(E * 7 + k)
    T, D = 777, 24
    xf = rng.integers(-2, 3, size=(T, D)).astype(np.float32)
    wf = rng.integers(-1, 2, size=(E, D)).astype(np.float32)
    x = synth.to_bf16_bits(xf) if dt == "bf16" else xf
    w = synth.to_bf16_bits(wf) if dt == "bf16" else wf
    idx, gate = cm.route(dev(x), dev(w), None, k)
    torch.cuda.synchronize()
    lg = oracle.router_logits(x, w, None)
    idx_ref, gate_ref = oracle.topk(lg, k)
    assert (oracle.margins(lg, k) == 0).sum() > 50           # many real ties
    assert np.array_equal(idx.cpu().numpy(), idx_ref)
    assert np.all(np.abs(gate.cpu().numpy() - gate_ref) <= 2e-7)


def test_dispatch_edge_cases():
    # all tokens on one expert, empty experts, k = E
    T, E = 600, 5
    for idx_np in (np.full((T, 1), 3, np.int32),
                   np.tile(np.arange(E, dtype=np.int32), (T, 1)),
                   np.random.default_rng(0).integers(0, 2, size=(T, 1)).astype(np.int32)):
        k = idx_np.shape[1]
        counts, offsets, perm, inv, _ = cm.dispatch(torch.from_numpy(idx_np).cuda(), E, D=8)
        torch.cuda.synchronize()
        check_dispatch(idx_np, E, counts.cpu().numpy(), offsets.cpu().numpy(),
                       perm.cpu().numpy(), inv.cpu().numpy())


@pytest.mark.parametrize("T,E,k", [(256 * 549, 64, 2), (256 * 1030 + 17, 16, 3)])
def test_dispatch_chunked_scan(T, E, k):
    """Histograms too large for the permutation's inline scan go through the
    chunked scan (256 tiles per chunk, the chunk prefixes added by the
    permutation): several chunks and a ragged last one, bit-exact against the
    oracle, with empty slots mixed in."""
    rng = np.random.default_rng(T)
    idx_np = np.stack([rng.choice(E, size=k, replace=False) for _ in range(T)]).astype(np.int32)
    idx_np[rng.random((T, k)) < 0.1] = -1
    counts, offsets, perm, inv, _ = cm.dispatch(torch.from_numpy(idx_np).cuda(), E, D=8)
    torch.cuda.synchronize()
    check_dispatch(idx_np, E, counts.cpu().numpy(), offsets.cpu().numpy(), perm.cpu().numpy(),
                   inv.cpu().numpy())


@pytest.mark.parametrize("dt,k", [("bf16", 1), ("bf16", 2), ("f32", 3)])
def test_combine_against_oracle(dt, k):
    T, D, E = 513, 136 if dt == "bf16" else 100, 6
    rng = np.random.default_rng(k)
    idx_np = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    gate_np = rng.random((T, k)).astype(np.float32)
    yef = rng.standard_normal((T * k, D)).astype(np.float32)
    ye = synth.to_bf16_bits(yef) if dt == "bf16" else yef
    _, _, _, inv_np = oracle.dispatch(idx_np, E)
    y = cm.combine(dev(ye), torch.from_numpy(inv_np).cuda(), torch.from_numpy(gate_np).cuda())
    torch.cuda.synchronize()
    ref = oracle.combine(ye, inv_np, gate_np, k)
    got = oracle.widen(cm.to_stored(y))
    bound = (2.0 ** -8 if dt == "bf16" else 1e-6) * np.abs(ref) + 1e-6
    assert np.all(np.abs(got - ref) <= bound)


# ------------------------------------------------------------ ffn_forward ----
SMALL_LAYERS = [
    # dtype, T, D, H, E, k, r, q, residual
    ("f32", 1, 64, 128, 1, 1, 16, 8, "random"),
    ("f32", 97, 64, 128, 3, 1, 32, 16, "random"),
    ("f32", 300, 96, 160, 4, 2, 32, 8, "random"),
    ("f32", 129, 64, 64, 8, 8, 64, 0, "zero"),
    ("f32", 200, 64, 96, 3, 2, 0, 16, "random"),
    ("bf16", 1, 64, 128, 2, 1, 16, 8, "random"),
    ("bf16", 257, 128, 256, 8, 1, 64, 16, "random"),
    ("bf16", 400, 64, 192, 6, 2, 32, 24, "random"),
    ("bf16", 333, 192, 384, 5, 3, 64, 32, "svd_tail"),
    # top-2 with more experts than the pair order covers (E (E + 1) / 2 >
    # 64): the chain with h_sh, h_res and the combine
    ("bf16", 700, 64, 128, 11, 2, 16, 8, "random"),
    ("f32", 301, 64, 96, 12, 2, 16, 8, "random"),
    # the pair order at its largest key count (E = 10: 55 keys)
    ("bf16", 1500, 64, 128, 10, 2, 32, 16, "random"),
]


@pytest.mark.parametrize("dt,T,D,H,E,k,r,q,res", SMALL_LAYERS)
def test_ffn_forward_small(dt, T, D, H, E, k, r, q, res):
    cfg = synth.LayerConfig("small", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dt, seed=T + D,
                            residual=res, n_cal=3000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(1)
    L["b1"] = (0.1 * rng.standard_normal(H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    L["bg"] = (0.3 * rng.standard_normal(E)).astype(np.float32)
    g = gpu_ffn(L)
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(g["idx"], ref["logits"], k)
    assert_gates(g["gate"], ref["logits"], g["idx"], k, tie)
    ok = ~tie
    if dt == "f32":
        assert max_rel(g["y"][ok], ref["y"][ok]) <= F32_MAXREL
    else:
        e = frob_rel(g["y"][ok], ref["y"][ok])
        assert e <= BF16_FROB_REGRESS, e


def _sample_rows(T, n, seed):
    rng = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([[0, T - 1], rng.choice(T, size=min(n, T), replace=False)]))
    return rows


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C5-E2", "C5-E6"])
def test_ffn_forward_configs(name):
    """Full-size layers in the benchmark's launch configuration.  Routing and
    dispatch are compared on every token; values on a sample of rows (every
    output row depends on its own token only)."""
    cfg = synth.CONFIGS[name]
    L = synth.make_layer(cfg)
    g = gpu_ffn(L)
    _, _, lg = oracle.route(L["x"], L["Wg"], L["bg"], cfg.k)
    tie = assert_routing(g["idx"], lg, cfg.k)
    assert_gates(g["gate"], lg, g["idx"], cfg.k, tie)
    rows = _sample_rows(cfg.T, 256 if cfg.T > 2000 else cfg.T, 5)
    rows = rows[~tie[rows]]
    ref = oracle.ffn_forward_layer(L, rows=rows)
    if cfg.dtype == "f32":
        e = max_rel(g["y"][rows], ref["y"])
        assert e <= F32_MAXREL, e
    else:
        e = frob_rel(g["y"][rows], ref["y"])
        assert e <= BF16_FROB and e <= BF16_FROB_REGRESS, e


def test_pair_order_launches():
    """The top-2 layer in pair order: one key pass (with its tile histogram),
    one permutation (over keys; no expert-order dispatch), fc1 once (beside
    the routing, on the side stream), the two pair products; the result
    against the oracle."""
    cfg = synth.LayerConfig("pairlaunch", T=1500, D=128, H=256, E=6, k=2, r=32, q=16, dtype="bf16",
                            seed=12, residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    cm.timing_start(cm.stage_names(), max_records=64)
    try:
        g = gpu_ffn(L)
    finally:
        t = cm.timing_stop()
    launched = {k: v[1] for k, v in t.items() if v[1] > 0}
    assert launched == {"route": 1, "pair_key": 1, "permute": 1, "fc1_gelu": 1, "tu_pair": 1,
                        "y_pair": 1}, launched
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(g["idx"], ref["logits"], 2)
    e = frob_rel(g["y"][~tie], ref["y"][~tie])
    assert e <= BF16_FROB_REGRESS, e


@pytest.mark.parametrize("dt,r", [("bf16", 32), ("f32", 16), ("bf16", 0)])
def test_pair_order_every_pair(dt, r):
    """Top-2 over E = 8 experts in pair order: tokens spread over all 28
    expert pairs (uniform clusters and a router with small weights, plus
    a random bias), segments of every length from a few rows to several
    tiles, r = 0 included (no shared basis: only the two residuals)."""
    cfg = synth.LayerConfig("pairs", T=3001, D=64, H=192, E=8, k=2, r=r, q=16, dtype=dt,
                            seed=21 + r, residual="random", n_cal=2000, router_noise=2.0)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(4)
    L["bg"] = (0.5 * rng.standard_normal(8)).astype(np.float32)
    L["b1"] = (0.1 * rng.standard_normal(cfg.H)).astype(np.float32)
    L["b2"] = (0.1 * rng.standard_normal(cfg.D)).astype(np.float32)
    g = gpu_ffn(L)
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(g["idx"], ref["logits"], 2)
    pairs = {tuple(sorted(p)) for p in g["idx"].tolist()}
    assert len(pairs) == 28, len(pairs)
    ok = ~tie
    if dt == "f32":
        assert max_rel(g["y"][ok], ref["y"][ok]) <= F32_MAXREL
    else:
        assert frob_rel(g["y"][ok], ref["y"][ok]) <= BF16_FROB_REGRESS
    assert_elementwise(g["y"][ok], ref["y"][ok], dt)


def test_ffn_zero_shared_basis_isolates_residual_dispatch():
    """US = 0, random experts: y is the routed residual alone, so a token sent
    to a wrong expert or with a wrong gate shows at the float32 bar."""
    cfg = synth.LayerConfig("res", T=517, D=64, H=128, E=6, k=2, r=16, q=16, dtype="f32", seed=3,
                            residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    L["US"] = np.zeros_like(L["US"])
    g = gpu_ffn(L)
    ref = oracle.ffn_forward_layer(L)
    tie = assert_routing(g["idx"], ref["logits"], 2)
    assert max_rel(g["y"][~tie], ref["y"][~tie]) <= F32_MAXREL


@pytest.mark.parametrize("mode", ["one_expert", "empty_experts"])
def test_ffn_skewed_routing(mode):
    cfg = synth.LayerConfig("skew", T=300, D=64, H=128, E=5, k=1, r=16, q=8, dtype="bf16",
                            seed=8, residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    bg = np.zeros(5, np.float32)
    if mode == "one_expert":
        bg[2] = 1e4
    else:
        bg[[0, 3]] = -1e4
    L["bg"] = bg
    g = gpu_ffn(L)
    ref = oracle.ffn_forward_layer(L)
    assert np.array_equal(g["idx"], ref["idx"])
    assert frob_rel(g["y"], ref["y"]) <= BF16_FROB_REGRESS


def test_ffn_deterministic_and_zero_tokens():
    L = synth.make_layer(synth.LayerConfig("det", T=1000, D=128, H=256, E=8, k=2, r=32, q=16,
                                           dtype="bf16", seed=12, n_cal=2000))
    a, b = gpu_ffn(L), gpu_ffn(L)
    assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["idx"], b["idx"])
    L0 = dict(L)
    L0["x"] = L["x"][:0]
    L0["cfg"] = synth.LayerConfig("det0", T=0, D=128, H=256, E=8, k=2, r=32, q=16, dtype="bf16",
                                  seed=12)
    y = cm.ffn_forward(*[dev(L0[n]) for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg",
                                              "bg")], 2)
    torch.cuda.synchronize()
    assert y.shape == (0, 128)


# ------------------------------------------------- dispatch-only workload ----
def test_dispatch_workload_full_size():
    """2^20 tokens, D = 384, E = 8, top-2, Zipf-skewed router bias, bf16:
    route + histogram -> scan + permute (+ rows) -> gated combine, exactly the
    sequence the benchmark times."""
    L = synth.make_dispatch()
    c = L["cfg"]
    T, D, E, k = c["T"], c["D"], c["E"], c["k"]
    x, Wg, bg = dev(L["x"]), dev(L["Wg"]), dev(L["bg"])
    s = cm.make_shape(T, D, E, k, cm.BF16)
    ws = cm.alloc_workspace(s)
    idx, gate = cm.route(x, Wg, bg, k, ws=ws)
    counts, offsets, perm, inv, xperm = cm.dispatch(idx, E, ws=ws, x=x, hist_in_ws=True)
    y = cm.combine(xperm, inv, gate)
    torch.cuda.synchronize()
    idx_h, gate_h = idx.cpu().numpy(), gate.cpu().numpy()
    _, _, lg = oracle.route(L["x"], L["Wg"], L["bg"], k)
    tie = assert_routing(idx_h, lg, k)
    assert_gates(gate_h, lg, idx_h, k, tie)
    check_dispatch(idx_h, E, counts.cpu().numpy(), offsets.cpu().numpy(), perm.cpu().numpy(),
                   inv.cpu().numpy())
    cnt = counts.cpu().numpy()
    assert cnt[0] > cnt[-1]                               # Zipf skew visible in the load
    p = perm.cpu().numpy()
    xp = cm.to_stored(xperm)
    rows = _sample_rows(T * k, 4096, 3)
    assert np.array_equal(xp[rows], L["x"][p[rows] // k])
    # combine on sampled tokens against the oracle (same definition on the gathered rows)
    toks = _sample_rows(T, 4096, 4)
    inv_h = inv.cpu().numpy().reshape(T, k)
    ye_sub = xp[inv_h[toks].ravel()]
    ref = oracle.combine(ye_sub, np.arange(toks.size * k, dtype=np.int32), gate_h[toks], k)
    got = oracle.widen(cm.to_stored(y))[toks]
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6)
    # identity experts + renormalised gates: the round trip returns x (up to one bf16 ulp)
    xs = oracle.widen(L["x"][toks])
    assert np.all(np.abs(got - xs) <= 2.0 ** -7 * np.abs(xs))
    assert np.mean(got == xs) > 0.99


@pytest.mark.parametrize("name", ["C1", "C2"])
def test_dense_comparator(name):
    """Dense FFN through the same GEMM kernels.  The oracle's layer reduces to
    it exactly with US = I, Vt = W2 (r = D) and a zero residual."""
    cfg = synth.CONFIGS[name]
    L = synth.make_layer(cfg)
    W2 = L["W2"].astype(np.float32) if cfg.dtype == "f32" else synth.to_bf16_bits(L["W2"])
    rng = np.random.default_rng(2)
    b1 = (0.1 * rng.standard_normal(cfg.H)).astype(np.float32)
    b2 = (0.1 * rng.standard_normal(cfg.D)).astype(np.float32)
    # the workspace of the CLEAR-MoE layer of the same shape serves the dense
    # FFN too (the benchmark's dense comparator reuses it)
    ws = cm.alloc_workspace(cm.make_shape(cfg.T, cfg.D, cfg.E, cfg.k,
                                          cm.F32 if cfg.dtype == "f32" else cm.BF16,
                                          H=cfg.H, r=cfg.r, q=cfg.q))
    y = cm.dense_ffn_forward(dev(L["x"]), dev(L["W1"]), dev(b1), dev(W2), dev(b2), ws=ws)
    torch.cuda.synchronize()
    rows = _sample_rows(cfg.T, 256, 6)
    D = cfg.D
    eye = np.eye(D, dtype=np.float32)
    ref = oracle.ffn_forward(L["x"][rows], L["W1"], b1, eye, W2, b2, np.zeros((1, D, 8)),
                             np.zeros((1, 8, cfg.H)), np.zeros((1, D), np.float32), None, 1)
    got = oracle.widen(cm.to_stored(y))[rows]
    if cfg.dtype == "f32":
        assert max_rel(got, ref["y"]) <= F32_MAXREL
    else:
        assert frob_rel(got, ref["y"]) <= BF16_FROB_REGRESS


@pytest.mark.parametrize("T,D,H", [
    (20011, 1672, 1032),   # both products: 256x128 tiles, 64-byte stages (largest)
    (16411, 520, 1032),    # both products: 256x128 tiles by row count (M >= 16384)
    (16411, 264, 1032),    # fc2 (N = 264, K = 1032): 256x128 tiles, long K with N <= 512
    (5003, 136, 1032),     # fc1 (N = 1032, K = 136): 128x128 tiles over eight waves
    (20011, 1672, 2056),   # fc2 with K >= 2048: 256x128 tiles, the staged epilogue, last column tile 8 wide
    (9001, 264, 2056),     # fc2 (N = 264, K = 2056): 64x64 tiles, the staged epilogue
])
def test_dense_gemm_tile_rules_ragged(T, D, H):
    """The dense FFN (bf16) at shapes that select each bf16 tile rule of the
    GEMM, with ragged row, column and k edges (no dimension a multiple of the
    tile; K ends inside a 32-element stage).  Sampled rows against the oracle,
    to which the dense FFN reduces with US = I, Vt = W2 and no residual."""
    rng = np.random.default_rng(T + D)
    x = synth.to_bf16_bits(rng.standard_normal((T, D)).astype(np.float32))
    W1 = synth.to_bf16_bits((0.02 * rng.standard_normal((H, D))).astype(np.float32))
    W2 = synth.to_bf16_bits((0.02 * rng.standard_normal((D, H))).astype(np.float32))
    b1 = (0.1 * rng.standard_normal(H)).astype(np.float32)
    b2 = (0.1 * rng.standard_normal(D)).astype(np.float32)
    y = cm.dense_ffn_forward(dev(x), dev(W1), dev(b1), dev(W2), dev(b2))
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([_sample_rows(T, 200, T), np.arange(T - 40, T)]))
    eye = np.eye(D, dtype=np.float32)
    ref = oracle.ffn_forward(x[rows], W1, b1, eye, W2, b2, np.zeros((1, D, 8)),
                             np.zeros((1, 8, H)), np.zeros((1, D), np.float32), None, 1)
    got = oracle.widen(cm.to_stored(y))[rows]
    e = frob_rel(got, ref["y"])
    assert e <= BF16_FROB_REGRESS, e
    assert_elementwise(got, ref["y"], "bf16")


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_large_fc1_tiles_with_ragged_edges(dt):
    """fc1 of this layer (M = T = 52517, N = H = 1032, K = D = 72) has
    206 x 5 = 1030 tiles of 256 x 256, which selects the product's 8-wave
    large-tile configuration; the last row tile holds 37 rows, the last
    column tile 8 columns, and K ends inside its second 128-byte stage.
    Top-2, so the layer runs the GEMM chain.  Routing on every token, values
    on a sample of rows."""
    cfg = synth.LayerConfig("bigtile", T=52517, D=72, H=1032, E=4, k=2, r=32, q=8, dtype=dt,
                            seed=11, residual="random", n_cal=2000)
    L = synth.make_layer(cfg)
    rng = np.random.default_rng(12)
    L["b1"] = (0.1 * rng.standard_normal(cfg.H)).astype(np.float32)
    g = gpu_ffn(L)
    _, _, lg = oracle.route(L["x"], L["Wg"], L["bg"], cfg.k)
    tie = assert_routing(g["idx"], lg, cfg.k)
    rows = _sample_rows(cfg.T, 512, 13)
    rows = np.unique(np.concatenate([rows, np.arange(cfg.T - 40, cfg.T)]))   # the last row tile
    rows = rows[~tie[rows]]
    ref = oracle.ffn_forward_layer(L, rows=rows)
    if dt == "f32":
        e = max_rel(g["y"][rows], ref["y"])
        assert e <= F32_MAXREL, e
    else:
        e = frob_rel(g["y"][rows], ref["y"])
        assert e <= BF16_FROB_REGRESS, e
