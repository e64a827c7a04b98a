"""A chained FFN stack (clearmoe_stack_forward) against the oracle.

The paper expertises half of a ViT's blocks (Sec. III Phase 2) and runs each
image's class token on the dense path (Table C6).  Here three layers with
their own weights are chained -- a CLEAR-MoE top-1 layer with class tokens, a
dense FFN and a CLEAR-MoE top-2 layer -- each adding its input back
(x_{l+1} = x_l + f_l(x_l)).  Every layer is checked on its own, on the GPU's
own input to it (the oracle applies layer l to the stored x_l and adds it),
with routing near-ties excluded and bounded, and the chain end to end against
the oracle's double-precision chain from x_0.  Random residual factors make
a wrong expert move the output far beyond the bars (checked on the CPU).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

from parity_util import (BF16_FROB, BF16_FROB_REGRESS, MARGIN, assert_elementwise,
                         bound_excluded, dev, frob_rel)

pytestmark = pytest.mark.gpu

T, D, H, E, R, Q = 3000, 384, 1536, 8, 128, 32


def _layers():
    """Host layer dicts: MoE top-1 with class tokens, dense, MoE top-2."""
    out = []
    for l, (kind, k) in enumerate((("moe", 1), ("dense", 1), ("moe", 2))):
        cfg = synth.LayerConfig(f"stack{l}", T=T, D=D, H=H, E=E, k=k, r=R, q=Q, dtype="bf16",
                                seed=40 + l, residual="random", n_cal=4000)
        L = synth.make_layer(cfg)
        rng = np.random.default_rng(50 + l)
        L["b1"] = (0.05 * rng.standard_normal(H)).astype(np.float32)
        L["b2"] = (0.05 * rng.standard_normal(D)).astype(np.float32)
        if l == 0:
            L = synth.with_class_tokens(L, stride=197)
        if kind == "dense":
            L["W2"] = synth.to_bf16_bits(L["W2"])
        L["kind"] = kind
        out.append(L)
    return out


def _device_layers(layers):
    keep, stack = [], []
    for L in layers:
        d = {n: dev(L[n]) for n in ("W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg", "bg")}
        if L["kind"] == "dense":
            d["W2"] = dev(L["W2"])
            stack.append(cm.make_stack_layer(d["W1"], d["b1"], d["b2"], W2=d["W2"]))
        else:
            stride = int(L.get("dense_stride") or 0)
            if stride:
                d["W2"] = dev(L["W2"])
            router = cm.make_router(d["Wg"], d["bg"], dense_stride=stride, W2=d.get("W2"))
            stack.append(cm.make_stack_layer(d["W1"], d["b1"], d["b2"], d["US"], d["Vt"], d["P"],
                                             d["Q"], router, k=L["cfg"].k, W2=d.get("W2")))
        keep.append(d)
    return stack, keep


def _oracle_layer(L, x):
    """f_l(x) in double on inputs x (stored or double), the near-tie mask and
    the chosen experts (None for a dense layer)."""
    if L["kind"] == "dense":
        f = oracle.dense_fc2(oracle.fc1_gelu(x, L["W1"], L["b1"]), L["W2"], L["b2"])
        return f, np.zeros(x.shape[0], dtype=bool), None
    A = dict(L)
    A["x"] = x
    ref = oracle.ffn_forward_layer(A)
    tie = oracle.margins(ref["logits"], L["cfg"].k) < MARGIN
    if "cls" in ref:
        tie &= ~ref["cls"]                      # class tokens are not routed
    return ref["y"], tie, ref["idx"]


def _run(stack, x, n, residual=True):
    y = cm.stack_forward(x, stack[:n], H, E, R, Q, residual=residual)
    torch.cuda.synchronize()
    return cm.to_stored(y)


def test_stack_layer_by_layer_and_end_to_end():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    layers = _layers()
    stack, keep = _device_layers(layers)
    x0 = layers[0]["x"]
    xs = [x0] + [_run(stack, dev(x0), n) for n in (1, 2, 3)]
    excl_any = np.zeros(T, dtype=bool)
    idx_gpu_in = []
    for l, L in enumerate(layers):
        print(f"layer {l} ({L['kind']}, k={L['cfg'].k})", flush=True)
        xin = oracle.widen(xs[l])
        f, tie, idx_l = _oracle_layer(L, xs[l])
        idx_gpu_in.append(idx_l)
        bound_excluded(tie)
        excl_any |= tie
        want = xin + f
        got = oracle.widen(xs[l + 1])
        ok = ~tie
        e = frob_rel(got[ok], want[ok])
        print(f"  relative Frobenius error {e:.3e}")
        assert e <= BF16_FROB_REGRESS, e
        assert_elementwise(got[ok], want[ok], "bf16")
        # the layer's own contribution, x_{l+1} - x_l, against f_l: the bar
        # of a bf16 layer output plus the two roundings of the sum
        fe = frob_rel(got[ok] - xin[ok], f[ok])
        print(f"  layer output relative error {fe:.3e}")
        assert fe <= BF16_FROB, fe
        if L["kind"] == "moe":
            # a wrong expert would move the layer output by far more than that
            rows = np.nonzero(ok)[0][:200]
            lg = oracle.router_logits(xs[l][rows], L["Wg"], L["bg"])
            idx, gate = oracle.topk(lg, L["cfg"].k)
            wrong = oracle.ffn_forward_routed(xs[l][rows], L["W1"], L["b1"], L["US"], L["Vt"],
                                              L["b2"], L["P"], L["Q"], (idx + 1) % E, gate)
            right = oracle.ffn_forward_routed(xs[l][rows], L["W1"], L["b1"], L["US"], L["Vt"],
                                              L["b2"], L["P"], L["Q"], idx, gate)
            assert frob_rel(wrong, right) > 10 * BF16_FROB
    # end to end: the oracle's chain in double from x_0.  The GPU chain keeps
    # x_l in bfloat16, which moves the logits of later layers by ~1e-2; a
    # token whose routing differs between the two chains at some layer gets
    # another expert's residual, so the comparison covers the tokens that both
    # chains routed alike at every layer (their share is printed and bounded).
    x = oracle.widen(x0)
    same = ~excl_any
    for l, L in enumerate(layers):
        f, _, idx = _oracle_layer(L, x)
        if idx is not None:
            same &= np.all(idx == idx_gpu_in[l], axis=1)
        x = x + f
    print(f"tokens routed alike by both chains: {same.mean():.4f}")
    assert same.mean() >= 0.97
    ok = same
    e = frob_rel(oracle.widen(xs[3])[ok], x[ok])
    print(f"chain relative Frobenius error {e:.3e}")
    assert e <= BF16_FROB_REGRESS, e
    del keep


def test_stack_without_residual_and_determinism():
    """x_{l+1} = f_l(x_l): the same layers, no skip connection; two runs give
    the same bits."""
    layers = _layers()[:2]
    stack, keep = _device_layers(layers)
    x0 = layers[0]["x"]
    a = _run(stack, dev(x0), 2, residual=False)
    b = _run(stack, dev(x0), 2, residual=False)
    assert np.array_equal(a, b)
    x1 = _run(stack, dev(x0), 1, residual=False)
    f0, tie0, _ = _oracle_layer(layers[0], x0)
    bound_excluded(tie0)
    e = frob_rel(oracle.widen(x1)[~tie0], f0[~tie0])
    assert e <= BF16_FROB_REGRESS, e
    f1, _, _ = _oracle_layer(layers[1], x1)
    e = frob_rel(oracle.widen(a), f1)
    assert e <= BF16_FROB_REGRESS, e
    del keep
