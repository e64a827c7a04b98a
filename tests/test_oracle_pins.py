"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: each check is a closed form,
an invariant, a special case that reduces to a textbook / library routine,
brute force on tiny inputs, or a number the paper prints.  Every plausible
slip in the oracle (a dropped bias, a wrong sign or index, a transposed
operand, a wrong slot or gate) breaks at least one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy.special import erf as sp_erf

import oracle
from paper_2606_28516_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _gelu_lib(v):
    return 0.5 * v * (1.0 + sp_erf(v / math.sqrt(2.0)))


def _small(E=4, k=1, T=97, D=24, H=40, r=8, q=6, residual="random", seed=11, dtype="f32",
           **kw):
    cfg = synth.LayerConfig("pin", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dtype, seed=seed,
                            residual=residual, n_cal=2000, **kw)
    return synth.make_layer(cfg)


def _with_biases(L, seed=5):
    """Non-zero b1, b2, bg so that a dropped bias term shows."""
    rng = np.random.default_rng(seed)
    L = dict(L)
    L["b1"] = (0.3 * rng.standard_normal(L["b1"].shape)).astype(np.float32)
    L["b2"] = (0.3 * rng.standard_normal(L["b2"].shape)).astype(np.float32)
    L["bg"] = (0.5 * rng.standard_normal(L["bg"].shape)).astype(np.float32)
    return L


def _run(L, **over):
    a = dict(L)
    a.update(over)
    return oracle.ffn_forward(a["x"], a["W1"], a["b1"], a["US"], a["Vt"], a["b2"], a["P"],
                              a["Q"], a["Wg"], a["bg"], a["cfg"].k)


def _dense(x, W1, b1, W, b2):
    """Textbook two-layer MLP y = GELU(x W1^T + b1) W^T + b2 (numpy + scipy erf)."""
    h = oracle.widen(x) @ oracle.widen(W1).T + oracle.widen(b1)
    return _gelu_lib(h) @ np.asarray(W).T + oracle.widen(b2)


# ---------------------------------------------------------------- GELU ----
def test_gelu_closed_forms():
    assert oracle.gelu(0.0) == 0.0
    # Phi(1) from the standard normal table.
    assert abs(oracle.gelu(1.0) - 0.8413447460685429) < 1e-15
    assert abs(oracle.gelu(-1.0) + (1 - 0.8413447460685429)) < 1e-15
    # GELU(v) - GELU(-v) = v Phi(v) + v (1 - Phi(v)) = v.
    for v in (0.1, 0.7, 1.3, 2.9, 5.0):
        assert abs(oracle.gelu(v) - oracle.gelu(-v) - v) < 1e-14
    # Far tails: GELU(v) -> v and -> 0.
    assert abs(oracle.gelu(12.0) - 12.0) < 1e-14 and abs(oracle.gelu(-12.0)) < 1e-14


# -------------------------------------------------------------- router ----
def test_router_logits_exact_integers():
    rng = np.random.default_rng(0)
    x = rng.integers(-8, 9, size=(33, 17)).astype(np.float32)
    Wg = rng.integers(-8, 9, size=(5, 17)).astype(np.float32)
    bg = rng.integers(-50, 51, size=5).astype(np.float32)
    want = x.astype(np.int64) @ Wg.astype(np.int64).T + bg.astype(np.int64)
    got = oracle.router_logits(x, Wg, bg)
    assert np.array_equal(got, want.astype(np.float64))
    # NULL bias is a zero bias
    assert np.array_equal(oracle.router_logits(x, Wg, None), (want - bg.astype(np.int64)).astype(float))


def test_router_params_match_table_c5():
    g = json.load(open(os.path.join(GOLDEN, "table_c5_router_params.json")))
    # The oracle's router consumes Wg [E, D] and bg [E].
    L = synth.make_dispatch(T=4, D=g["d"], E=g["E"], k=1, seed=0)
    per_layer = L["Wg"].size + L["bg"].size
    assert per_layer * g["layers"] == g["linear_params_total"]
    d, h, E = g["d"], g["mlp_hidden"], g["E"]
    assert g["layers"] * ((d * h + h) + (h * E + E)) == g["mlp_params_total"]
    assert h == d // 6


def _brute_topk(l, k):
    E = len(l)
    best = None
    for tup in itertools.permutations(range(E), k):
        key = tuple((-l[e], e) for e in tup)
        # a valid top-k tuple is sorted and no unchosen expert beats its last
        if any(key[i] > key[i + 1] for i in range(k - 1)):
            continue
        rest = [(-l[e], e) for e in range(E) if e not in tup]
        if rest and min(rest) < key[-1]:
            continue
        assert best is None, "brute force found two valid tuples"
        best = tup
    return best


@pytest.mark.parametrize("E,k", [(1, 1), (2, 1), (2, 2), (3, 2), (5, 3), (6, 1), (6, 6)])
def test_topk_brute_force_with_ties(E, k):
    rng = np.random.default_rng(E * 10 + k)
    logits = rng.integers(-2, 3, size=(16, E)).astype(np.float64)   # many exact ties
    idx, gate = oracle.topk(logits, k)
    for t in range(16):
        assert tuple(idx[t]) == _brute_topk(list(logits[t]), k)


def test_margins_hand_computed():
    """The decision margin that decides which tokens a routing comparison may
    leave out (Algorithm 3's argmax, extended to the top-k order): the
    smallest gap between neighbours among the sorted top min(k + 1, E)
    logits.  Values worked by hand, with ties, k = 1..3, E = 1 and E = k."""
    inf = float("inf")
    cases = [
        # logits, k, margin
        ([3.0, 1.0, 2.0], 1, 1.0),            # 3 | 2: one gap
        ([3.0, 1.0, 2.0], 2, 1.0),            # 3, 2 | 1: gaps 1, 1
        ([5.0, 5.0, 0.0], 1, 0.0),            # tie for the top slot
        ([5.0, 5.0, 0.0], 2, 0.0),            # tie decides the slot order only
        ([0.0, 5.0, 5.0, 9.0], 1, 4.0),       # tie below the selection boundary
        ([0.0, 4.0, 4.5, 1.0], 1, 0.5),
        ([0.0, 4.0, 4.5, 1.0], 2, 0.5),       # gaps 0.5, 3
        ([0.0, 4.0, 4.5, 1.0], 3, 0.5),       # gaps 0.5, 3, 1
        ([1.0, 2.0, 4.0, 10.0], 1, 6.0),      # descending order: 10 | 4
        ([1.0, 2.0, 4.0, 10.0], 2, 2.0),      # 10, 4 | 2: gaps 6, 2
        ([1.0, 2.0, 4.0, 10.0], 3, 1.0),      # 10, 4, 2 | 1: gaps 6, 2, 1
        ([-1.0, -3.0, -2.0], 1, 1.0),         # negative logits
        ([7.0], 1, inf),                      # E = 1: nothing to decide
        ([1.0, 5.0, 2.0], 3, 1.0),            # E = k: slot-order gaps 3, 1 only
        ([4.0, 4.0], 2, 0.0),                 # E = k with a tie
        ([4.0, 3.0], 2, 1.0),
    ]
    for lg, k, want in cases:
        got = oracle.margins(np.array([lg]), k)
        assert got.shape == (1,) and got[0] == want, (lg, k, got, want)
    # several tokens at once, one margin per row
    lg = np.array([[3.0, 1.0, 2.0], [5.0, 5.0, 0.0], [0.0, 0.25, 9.0]])
    assert oracle.margins(lg, 1).tolist() == [1.0, 0.0, 8.75]


@pytest.mark.parametrize("E,k", [(2, 1), (4, 1), (5, 2), (6, 3), (4, 4), (8, 2)])
def test_margins_bound_the_top_k_decision(E, k):
    """What the margin means: moving every logit by less than half the margin
    never changes the ordered top-k (brute force), and some move of just over
    half the margin does (the two logits at the smallest gap swap)."""
    rng = np.random.default_rng(100 * E + k)
    lg = rng.standard_normal((40, E))
    m = oracle.margins(lg, k)
    for t in range(lg.shape[0]):
        base = _brute_topk(list(lg[t]), k)
        for _ in range(20):
            d = rng.uniform(-1.0, 1.0, E) * (0.499 * m[t])
            assert _brute_topk(list(lg[t] + d), k) == base
        # close the smallest gap among the decided positions
        order = sorted(range(E), key=lambda e: (-lg[t, e], e))
        span = min(k, E - 1)
        gaps = [lg[t, order[j]] - lg[t, order[j + 1]] for j in range(span)]
        j = int(np.argmin(gaps))
        assert gaps[j] == m[t]
        d = np.zeros(E)
        d[order[j]] -= 0.51 * m[t]
        d[order[j + 1]] += 0.51 * m[t]
        assert _brute_topk(list(lg[t] + d), k) != base


def test_gates_closed_forms():
    lg = np.array([[0.5, 2.0, -1.0, 2.0], [3.0, 1.0, 0.0, -4.0], [1.0, 1.0, 1.0, 1.0]])
    idx, g1 = oracle.topk(lg, 1)
    assert np.array_equal(g1, np.ones((3, 1)))          # renormalised top-1 gate is 1
    idx, g2 = oracle.topk(lg, 2)
    assert idx.tolist() == [[1, 3], [0, 1], [0, 1]]
    # k = 2: g0 = sigmoid(l0 - l1)
    for t in range(3):
        d = lg[t, idx[t, 0]] - lg[t, idx[t, 1]]
        assert abs(g2[t, 0] - 1.0 / (1.0 + math.exp(-d))) < 1e-15
        assert abs(g2[t, 0] + g2[t, 1] - 1.0) < 1e-15
    _, g4 = oracle.topk(lg[2:], 4)
    assert np.allclose(g4, 0.25, atol=0, rtol=1e-15)
    # Renormalised top-k == softmax over all E, restricted to the k and renormalised.
    rng = np.random.default_rng(3)
    lg = rng.standard_normal((50, 7))
    idx, g3 = oracle.topk(lg, 3)
    sm = np.exp(lg - lg.max(1, keepdims=True))
    sm /= sm.sum(1, keepdims=True)
    sel = np.take_along_axis(sm, idx, 1)
    assert np.allclose(g3, sel / sel.sum(1, keepdims=True), rtol=1e-13, atol=0)


# ------------------------------------------------------------ dispatch ----
@pytest.mark.parametrize("T,E,k", [(1, 1, 1), (7, 3, 2), (300, 8, 2), (257, 5, 1), (64, 4, 4)])
def test_dispatch_against_library_routines(T, E, k):
    rng = np.random.default_rng(T + E + k)
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts, offsets, perm, inv = oracle.dispatch(idx, E)
    flat = idx.ravel()
    assert np.array_equal(counts, np.bincount(flat, minlength=E))
    assert np.array_equal(offsets, np.concatenate([[0], np.cumsum(counts)]))
    assert np.array_equal(perm, np.argsort(flat, kind="stable"))
    assert np.array_equal(inv[perm], np.arange(T * k))
    assert counts.sum() == T * k
    for e in range(E):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e)
        assert np.all(np.diff(seg // k) > 0)      # token ids strictly increase


def test_dispatch_rejects_bad_index():
    with pytest.raises(ValueError):
        oracle.dispatch(np.array([[0], [3]], dtype=np.int32), 3)


def test_dispatch_empty_and_all_on_one_expert():
    counts, offsets, perm, inv = oracle.dispatch(np.full((10, 1), 2, np.int32), 4)
    assert counts.tolist() == [0, 0, 10, 0] and offsets.tolist() == [0, 0, 0, 10, 10]
    assert np.array_equal(perm, np.arange(10))
    counts, offsets, perm, inv = oracle.dispatch(np.zeros((0, 2), np.int32), 3)
    assert counts.tolist() == [0, 0, 0] and perm.size == 0


# ---------------------------------------------------------- layer forms ----
def test_I1_zero_residual_is_dense_low_rank_ffn():
    """P = 0: y = GELU(x W1^T + b1) W_shared^T + b2, W_shared = US Vt materialised
    (the paper's own dense form of the shared basis)."""
    L = _with_biases(_small(E=4, k=2, D=24, H=40, r=8))
    out = _run(L, P=np.zeros_like(L["P"]))
    Wsh = oracle.widen(L["US"]) @ oracle.widen(L["Vt"])
    want = _dense(L["x"], L["W1"], L["b1"], Wsh, L["b2"])
    assert np.max(np.abs(out["y"] - want)) < 1e-12 * max(1.0, np.max(np.abs(want)))


def test_I2_full_rank_is_dense_ffn():
    """r = min(D, H), residual zero: the SVD basis reconstructs fc2 exactly."""
    L = _with_biases(_small(E=3, k=1, D=20, H=36, r=20, q=4, residual="zero", dtype="f32"))
    # fp64 factors so the reconstruction is exact up to double rounding
    U, S, Vh = np.linalg.svd(L["W2"], full_matrices=False)
    out = _run(L, US=U * S, Vt=Vh)
    want = _dense(L["x"], L["W1"], L["b1"], L["W2"], L["b2"])
    assert np.max(np.abs(out["y"] - want)) < 1e-12


def test_I3_single_expert():
    """E = 1: identity permutation, one segment, gate 1, y = dense FFN with
    weight W_shared + P_0 Q_0."""
    L = _with_biases(_small(E=1, k=1, T=53, D=16, H=32, r=6, q=5))
    out = _run(L)
    assert np.array_equal(out["idx"][:, 0], np.zeros(53, np.int32))
    assert np.array_equal(out["gate"], np.ones((53, 1)))
    counts, offsets, perm, inv = oracle.dispatch(out["idx"], 1)
    assert counts.tolist() == [53] and np.array_equal(perm, np.arange(53))
    W = oracle.widen(L["US"]) @ oracle.widen(L["Vt"]) + oracle.widen(L["P"])[0] @ oracle.widen(L["Q"])[0]
    want = _dense(L["x"], L["W1"], L["b1"], W, L["b2"])
    assert np.max(np.abs(out["y"] - want)) < 1e-12


@pytest.mark.parametrize("k", [1, 2])
def test_I5_full_residual_reconstructs_dense_for_any_routing(k):
    """D3: shared basis + the full tail (q = D - r, every s_e = 1) is fc2 exactly,
    whatever the routing (here a random router with a random bias)."""
    D, H, r = 18, 30, 7
    L = _with_biases(_small(E=5, k=k, D=D, H=H, r=r, q=D - r, residual="svd_tail"))
    U, S, Vh = np.linalg.svd(L["W2"], full_matrices=False)
    tail_P = U[:, r:] * S[r:]
    P = np.broadcast_to(tail_P, (5, D, D - r)).copy()           # s_e = 1
    Q = np.broadcast_to(Vh[r:], (5, D - r, H)).copy()
    rng = np.random.default_rng(9)
    Wg = rng.standard_normal((5, D))
    out = _run(L, US=U[:, :r] * S[:r], Vt=Vh[:r], P=P, Q=Q, Wg=Wg)
    assert len(set(out["idx"][:, 0].tolist())) > 2              # routing really varies
    want = _dense(L["x"], L["W1"], L["b1"], L["W2"], L["b2"])
    assert np.max(np.abs(out["y"] - want)) < 1e-12


def test_I6_equal_scales_make_output_routing_invariant():
    """All s_e equal: every expert has the same residual (Sec. III Phase 3), so y
    does not depend on the assignment."""
    L = _small(E=4, k=1, residual="svd_tail", D=24, H=40, r=8, q=6)
    Pe = oracle.widen(L["P"])[0] / L["s"][0] * 0.8
    P = np.broadcast_to(Pe, L["P"].shape).copy()
    a = _run(L, P=P)
    b = _run(L, P=P, Wg=oracle.widen(L["Wg"])[::-1].copy())       # a different router
    assert not np.array_equal(a["idx"], b["idx"])
    assert np.max(np.abs(a["y"] - b["y"])) < 1e-13


@pytest.mark.parametrize("k", [1, 2])
def test_residual_goes_to_routed_expert_with_its_gate(k):
    """Only expert e has a residual: tokens not routed to e get exactly the shared
    path; a token routed to e in slot j gets gate_j times the low-rank product
    P_e Q_e applied to its hidden activation (a plain dense matrix product)."""
    E = 4
    L = _with_biases(_small(E=E, k=k, T=120, D=24, H=40, r=8, q=6))
    base = _run(L, P=np.zeros_like(L["P"]))
    z = _gelu_lib(oracle.widen(L["x"]) @ oracle.widen(L["W1"]).T + oracle.widen(L["b1"]))
    for e in range(E):
        P = np.zeros(L["P"].shape)
        P[e] = oracle.widen(L["P"])[e]
        out = _run(L, P=P)
        R = oracle.widen(L["P"])[e] @ oracle.widen(L["Q"])[e]          # [D, H]
        hit = 0
        for t in range(L["cfg"].T):
            slots = np.nonzero(out["idx"][t] == e)[0]
            if slots.size == 0:
                assert np.array_equal(out["y"][t], base["y"][t])
            else:
                hit += 1
                j = slots[0]
                lg = np.sort(out["logits"][t])[::-1][:k]
                g = math.exp(lg[j] - lg[0]) / np.sum(np.exp(lg - lg[0]))
                want = base["y"][t] + g * (R @ z[t])
                assert np.max(np.abs(out["y"][t] - want)) < 1e-12
        assert hit > 0


def test_I9_token_permutation_equivariance():
    L = _with_biases(_small(E=4, k=2, T=77))
    a = _run(L)
    pi = np.random.default_rng(1).permutation(77)
    b = _run(L, x=L["x"][pi])
    assert np.array_equal(b["y"], a["y"][pi])
    assert np.array_equal(b["idx"], a["idx"][pi])
    ca = oracle.dispatch(a["idx"], 4)[0]
    cb = oracle.dispatch(b["idx"], 4)[0]
    assert np.array_equal(ca, cb)


def test_I10_zero_shared_basis_leaves_pure_residual():
    L = _small(E=4, k=1, T=64, D=24, H=40, r=8, q=6)
    out = _run(L, US=np.zeros_like(L["US"]))
    z = _gelu_lib(oracle.widen(L["x"]) @ oracle.widen(L["W1"]).T)
    P, Q = oracle.widen(L["P"]), oracle.widen(L["Q"])
    for t in range(64):
        e = out["idx"][t, 0]
        assert np.max(np.abs(out["y"][t] - P[e] @ (Q[e] @ z[t]))) < 1e-12


# ------------------------------------------------------------- combine ----
@pytest.mark.parametrize("k", [1, 2, 3])
def test_I8_identity_expert_round_trip(k):
    """Permute rows into expert order, combine back with renormalised gates:
    sum_j g_j x = x since the gates sum to one."""
    D = synth.make_dispatch(T=300, D=40, E=6, k=k, seed=7)
    idx, gate, _ = oracle.route(D["x"], D["Wg"], D["bg"], k)
    counts, offsets, perm, inv = oracle.dispatch(idx, 6)
    xp = oracle.permute_rows(D["x"], perm, k)
    for p in range(0, 300 * k, 37):
        assert np.array_equal(xp[p], oracle.widen(D["x"])[perm[p] // k])
    y = oracle.combine(xp, inv, gate, k)
    assert np.max(np.abs(y - oracle.widen(D["x"]))) < 1e-14 * np.max(np.abs(oracle.widen(D["x"])))


def test_combine_weights_by_slot_gate():
    """Experts that scale rows by a constant c_e: combine gives sum_j g_j c_{e_j} x."""
    T, k, E, Dm = 50, 2, 3, 8
    rng = np.random.default_rng(2)
    x = rng.standard_normal((T, Dm))
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    gate = rng.random((T, k))
    c = np.array([1.0, -2.0, 0.5])
    counts, offsets, perm, inv = oracle.dispatch(idx, E)
    ye = oracle.permute_rows(x, perm, k) * c[idx.ravel()[perm]][:, None]
    y = oracle.combine(ye, inv, gate, k)
    want = (gate * c[idx]).sum(1)[:, None] * x
    assert np.max(np.abs(y - want)) < 1e-13


# ---------------------------------------------------------- generator ----
def test_generator_deterministic_and_shapes():
    cfg = synth.LayerConfig("det", T=33, D=16, H=24, E=3, k=2, r=5, q=4, dtype="bf16", seed=4,
                            n_cal=500)
    a, b = synth.make_layer(cfg), synth.make_layer(cfg)
    assert synth.fingerprint(a) == synth.fingerprint(b)
    c = synth.make_layer(cfg, seed=5)
    assert synth.fingerprint(a) != synth.fingerprint(c)
    assert a["x"].shape == (33, 16) and a["x"].dtype == np.uint16
    assert a["US"].shape == (16, 5) and a["Vt"].shape == (5, 24)
    assert a["P"].shape == (3, 16, 4) and a["Q"].shape == (3, 4, 24)
    assert a["Wg"].shape == (3, 16) and a["bg"].dtype == np.float32


def test_bf16_storage_rounding():
    v = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.0e-3], dtype=np.float32)
    b = synth.to_bf16_bits(v)
    back = oracle.widen(b)
    # ties to even: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == 1.0 + 2 ** -6 and back[3] == -2.5
    assert abs(back[4] - 3.0e-3) <= 2 ** -8 * 3.0e-3     # unit roundoff of bf16


def test_svd_tail_experts_are_scaled_tail():
    """Algorithm 2: every residual expert is the SVD tail times its own s_e."""
    L = _small(E=4, k=1, residual="svd_tail", D=24, H=40, r=8, q=6)
    U, S, Vh = np.linalg.svd(L["W2"], full_matrices=False)
    tail = (U[:, 8:14] * S[8:14]) @ Vh[8:14]
    for e in range(4):
        R = oracle.widen(L["P"])[e] @ oracle.widen(L["Q"])[e]
        assert np.max(np.abs(R - L["s"][e] * tail)) < 1e-6
    assert np.all(np.abs(L["s"] - 1.0) < 0.2)


def test_imbalance_mixture_recipe():
    """The load-imbalance recipe of the dispatch benchmark: balanced at 0,
    cluster 0 holding p + (1 - p) / E of the mass at p, and the oracle's
    routing of a draw follows it (the router rows point at the centres)."""
    assert synth.imbalance_mixture(4, 0.0) == (0.25, 0.25, 0.25, 0.25)
    w = synth.imbalance_mixture(4, 0.8)
    assert abs(sum(w) - 1.0) < 1e-12 and abs(w[0] - 0.85) < 1e-12
    assert all(abs(v - 0.05) < 1e-12 for v in w[1:])
    with pytest.raises(ValueError):
        synth.imbalance_mixture(4, 1.0)
    cfg = synth.LayerConfig("imb", T=4000, D=32, H=32, E=4, k=1, r=8, q=8, dtype="f32", seed=3,
                            mixture=w, n_cal=500)
    L = synth.make_layer(cfg)
    idx, _, _ = oracle.route(L["x"], L["Wg"], L["bg"], 1)
    share = np.bincount(idx[:, 0], minlength=4) / 4000.0
    assert abs(share.max() - 0.85) < 0.05, share


# ---- router variants (Sec. III Phase 4: MLP and adaptive routers) ----------

def _worked():
    return json.load(open(os.path.join(GOLDEN, "router_variants_worked.json")))


def test_mlp_router_worked_example():
    """Hand-worked token (normal CDF table values): a transposed Wh, a dropped
    bias or GELU taken as the identity would all move these logits."""
    g = _worked()["mlp"]
    x = np.array([g["x"]], np.float32)
    Wh, bh = np.array(g["Wh"], np.float32), np.array(g["bh"], np.float32)
    Wg, bg = np.array(g["Wg"], np.float32), np.array(g["bg"], np.float32)
    lg, hr = oracle.mlp_router_logits(x, Wh, bh, Wg, bg, "f32")
    # table values carry 9 decimals; hr is rounded to float32 (2^-24 relative)
    assert np.allclose(hr[0], g["hidden"], rtol=0, atol=2e-7)
    assert np.allclose(lg[0], g["logits"], rtol=0, atol=4e-7)
    idx, _ = oracle.topk(lg, 1)
    assert idx[0, 0] == g["top1"]


def test_mlp_router_params_and_hidden_rounding():
    g = json.load(open(os.path.join(GOLDEN, "table_c5_router_params.json")))
    cfg = synth.LayerConfig("c5", T=8, D=g["d"], H=64, E=g["E"], k=1, r=8, q=8, dtype="f32",
                            seed=0, n_cal=50)
    M = synth.with_mlp_router(synth.make_layer(cfg))
    rt = M["router"]
    per_layer = rt["Wh"].size + rt["bh"].size + M["Wg"].size + M["bg"].size
    assert per_layer * g["layers"] == g["mlp_params_total"]
    assert rt["Wh"].shape == (g["mlp_hidden"], g["d"])
    # bf16 storage rounding of the hidden layer: 8 significant bits, ties to
    # even, and the same as the input generator's float32 -> bf16 rounding
    v = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -7 + 5 * 2 ** -10), 3.0e-3,
                  -7.5e5, 1 + 2 ** -7 + 2 ** -9])
    r = oracle.round_to_storage(v, "bf16")
    assert r[1] == 1.0 and r[2] == 1 + 2 ** -6 and r[3] == -(1 + 2 ** -6)
    assert r[6] == 1 + 2 ** -7
    assert np.array_equal(r, synth.bf16_bits_to_f32(synth.to_bf16_bits(v.astype(np.float32))))


def test_adaptive_router_worked_example_and_limits():
    g = _worked()["adaptive"]
    lg = np.array([g["logits"]])
    assert abs(oracle.confidence(lg)[0] - g["confidence"]) < 1e-9
    for c in g["cases"]:
        idx, gate = oracle.adaptive_topk(lg, c["tau"])
        assert idx[0].tolist() == c["idx"]
        assert np.allclose(gate[0], c["gate"], atol=1e-9)
    rng = np.random.default_rng(11)
    for E in (2, 3, 5, 8):
        lg = rng.standard_normal((300, E)) * 2.0
        i1, g1 = oracle.topk(lg, 1)
        i2, g2 = oracle.topk(lg, 2)
        # tau <= 1/E: the confidence is never below it, so every token is top-1
        ia, ga = oracle.adaptive_topk(lg, 1.0 / E)
        assert np.array_equal(ia[:, 0], i1[:, 0]) and np.all(ia[:, 1] == -1)
        assert np.all(ga[:, 0] == 1.0) and np.all(ga[:, 1] == 0.0)
        # tau above 1: every token escalates to the plain top-2
        ia, ga = oracle.adaptive_topk(lg, 1.5)
        assert np.array_equal(ia, i2) and np.allclose(ga, g2)
        if E == 2:
            # two experts: confidence = sigmoid(|l0 - l1|), so a token escalates
            # exactly when |l0 - l1| < log(tau / (1 - tau))
            tau = 0.8
            ia, _ = oracle.adaptive_topk(lg, tau)
            esc = np.abs(lg[:, 0] - lg[:, 1]) < math.log(tau / (1 - tau))
            assert np.array_equal(ia[:, 1] >= 0, esc)
    ia, ga = oracle.adaptive_topk(np.zeros((3, 1)), 0.99)       # one expert
    assert np.all(ia[:, 0] == 0) and np.all(ia[:, 1] == -1) and np.all(ga[:, 0] == 1.0)


def test_dispatch_with_empty_slots_brute_force():
    """-1 marks an empty slot: not counted, no row, inv = -1; the rest is the
    stable sort by expert."""
    rng = np.random.default_rng(5)
    for T, E, k in ((1, 2, 2), (7, 3, 2), (40, 5, 2), (25, 4, 3)):
        idx = rng.integers(-1, E, size=(T, k)).astype(np.int32)
        counts, offsets, perm, inv = oracle.dispatch(idx, E)
        flat = idx.ravel()
        valid = [a for a in range(T * k) if flat[a] >= 0]
        order = sorted(valid, key=lambda a: (flat[a], a))
        n = len(order)
        assert offsets[-1] == n and counts.sum() == n
        assert perm[:n].tolist() == order and np.all(perm[n:] == -1)
        for a in range(T * k):
            assert (inv[a] == -1) == (flat[a] < 0)
            if flat[a] >= 0:
                assert perm[inv[a]] == a
    with pytest.raises(ValueError):
        oracle.dispatch(np.array([[0, -2]], np.int32), 2)


def test_residual_and_layer_with_empty_slots():
    """An empty slot adds nothing: the same as any expert with gate 0; the
    adaptive layer equals the top-1 layer on confident tokens and the top-2
    layer on escalated ones."""
    cfg = synth.LayerConfig("ad", T=300, D=24, H=40, E=4, k=2, r=8, q=6, dtype="f32", seed=8,
                            residual="random", n_cal=200)
    L = synth.make_layer(cfg)
    A = synth.with_adaptive_router(L, 0.95)
    ref = oracle.ffn_forward_layer(A)
    esc = ref["idx"][:, 1] >= 0
    assert 0 < esc.sum() < cfg.T
    idx2 = ref["idx"].copy()
    idx2[~esc, 1] = 3                       # any expert, gate 0
    z = oracle.fc1_gelu(L["x"], L["W1"], L["b1"])
    r1 = oracle.residual(z, L["Q"], L["P"], ref["idx"], ref["gate"])
    r2 = oracle.residual(z, L["Q"], L["P"], idx2, ref["gate"])
    assert np.array_equal(r1, r2)
    y1 = oracle.ffn_forward_layer(L, )                       # k = 2 layer
    y0 = oracle.ffn_forward_layer(dict(L, cfg=synth.dataclasses.replace(cfg, k=1)))
    assert np.allclose(ref["y"][esc], y1["y"][esc], rtol=0, atol=1e-12)
    assert np.allclose(ref["y"][~esc], y0["y"][~esc], rtol=0, atol=1e-12)


# ---- class tokens (Table C6: excluded from dispatch, dense path) -----------
def test_class_tokens_take_the_dense_ffn():
    """With one class token per image of 13 tokens, the class rows equal the
    textbook dense FFN with the original fc2, take no expert slot, and leave
    every other row exactly as the layer without class tokens computes it."""
    L = _with_biases(_small(E=5, k=2, T=91, residual="random"))
    C = synth.with_class_tokens(L, stride=13)
    out = oracle.ffn_forward_layer(C)
    cls = np.arange(91) % 13 == 0
    assert np.array_equal(out["cls"], cls) and cls.sum() == 7
    assert np.all(out["idx"][cls] == -1) and np.all(out["gate"][cls] == 0.0)
    want = _dense(C["x"][cls], C["W1"], C["b1"], oracle.widen(C["W2"]), C["b2"])
    assert np.max(np.abs(out["y"][cls] - want)) < 1e-12
    base = oracle.ffn_forward_layer(L)
    assert np.array_equal(out["idx"][~cls], base["idx"][~cls])
    assert np.max(np.abs(out["y"][~cls] - base["y"][~cls])) < 1e-13
    # the class rows really differ from the expert path (the residual is low rank)
    assert np.max(np.abs(out["y"][cls] - base["y"][cls])) > 1e-4
    # dispatch counts only the routed tokens
    counts, offsets, _, _ = oracle.dispatch(out["idx"], 5)
    assert counts.sum() == (91 - 7) * 2 and offsets[-1] == (91 - 7) * 2


def test_class_tokens_with_full_residual_agree_with_experts():
    """D3 (q = D - r, every s_e = 1): the expert path reconstructs fc2
    exactly, so class and routed tokens alike give the dense FFN."""
    D, H, r = 18, 30, 7
    L = _with_biases(_small(E=3, k=1, T=40, D=D, H=H, r=r, q=D - r, residual="svd_tail"))
    U, S, Vh = np.linalg.svd(L["W2"], full_matrices=False)
    L["US"], L["Vt"] = U[:, :r] * S[:r], Vh[:r]
    L["P"] = np.broadcast_to(U[:, r:] * S[r:], (3, D, D - r)).copy()
    L["Q"] = np.broadcast_to(Vh[r:], (3, D - r, H)).copy()
    C = synth.with_class_tokens(L, stride=10)
    C["W2"] = L["W2"]                                   # float64 here: exact reconstruction
    out = oracle.ffn_forward_layer(C)
    want = _dense(L["x"], L["W1"], L["b1"], L["W2"], L["b2"])
    assert out["cls"].sum() == 4
    assert np.max(np.abs(out["y"] - want)) < 1e-12


def test_class_tokens_on_a_row_sample_use_global_positions():
    """A sample of rows is classified by its global token index."""
    L = _with_biases(_small(E=4, k=1, T=60))
    C = synth.with_class_tokens(L, stride=20)
    rows = np.array([0, 1, 20, 39, 40, 59])
    part = oracle.ffn_forward_layer(C, rows=rows)
    full = oracle.ffn_forward_layer(C)
    assert np.array_equal(part["cls"], [True, False, True, False, True, False])
    assert np.max(np.abs(part["y"] - full["y"][rows])) < 1e-13


def test_full_softmax_gates_hand_computed():
    """Unrenormalised gates (shape field renorm = 0): each chosen expert's
    probability under the softmax over all E logits.  Logits ln 1 .. ln 4
    give probabilities 1/10 .. 4/10 exactly; the top two are experts 3 and 2
    with 4/10 and 3/10 (renormalised: 4/7, 3/7); top-1 gives 4/10."""
    lg = np.log(np.array([[1.0, 2.0, 3.0, 4.0], [4.0, 3.0, 2.0, 1.0]]))
    idx, g2 = oracle.topk(lg, 2)
    assert idx.tolist() == [[3, 2], [0, 1]]
    assert np.allclose(g2, [[4 / 7, 3 / 7], [4 / 7, 3 / 7]], rtol=0, atol=1e-15)
    full = oracle.full_softmax_gates(lg, idx)
    assert np.allclose(full, [[0.4, 0.3], [0.4, 0.3]], rtol=0, atol=1e-15)
    i1, _ = oracle.topk(lg, 1)
    assert np.allclose(oracle.full_softmax_gates(lg, i1), [[0.4], [0.4]], rtol=0, atol=1e-15)
    # an empty slot (adaptive top-1) gets 0; equal logits split evenly
    assert oracle.full_softmax_gates(np.zeros((1, 5)), np.array([[2, -1]])).tolist() == [[0.2, 0.0]]


@pytest.mark.parametrize("E,k", [(2, 1), (4, 2), (8, 2), (6, 3), (5, 5)])
def test_full_softmax_gates_against_the_renormalised(E, k):
    """Properties that tie the two gate rules together: the unrenormalised
    gates divided by their sum over the k slots are the renormalised gates of
    the C oracle's top-k; each is below 1 and their sum is the probability
    mass of the chosen experts, which is 1 when every expert is chosen (k =
    E) and at most 1 otherwise; with k = 1 the gate is the confidence."""
    rng = np.random.default_rng(7 * E + k)
    lg = 2.0 * rng.standard_normal((50, E))
    idx, g = oracle.topk(lg, k)
    full = oracle.full_softmax_gates(lg, idx)
    s = full.sum(axis=1)
    assert np.allclose(full / s[:, None], g, rtol=1e-13, atol=0)
    assert np.all(full < 1.0 + 1e-15) and np.all(s <= 1.0 + 1e-13)
    if k == E:
        assert np.allclose(s, 1.0, rtol=0, atol=1e-13)
    if k == 1:
        assert np.allclose(full[:, 0], oracle.confidence(lg), rtol=1e-14, atol=0)
