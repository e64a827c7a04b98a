"""Helpers of the GPU parity tests: move seeded inputs to the device, run the
HIP path through the C ABI, and compare with the CPU oracle."""
import numpy as np
import torch

import oracle
from paper_2606_28516_amd import clearmoe as cm

# Tolerances (stated once, used by every parity test).
MARGIN = 1e-6          # tokens whose top-k logit margin is below this may route differently
F32_MAXREL = 1e-4      # fp32 mode: max|y - y_ref| / max|y_ref|
BF16_FROB = 2e-2       # bf16 mode: ||y - y_ref||_F / ||y_ref||_F
BF16_FROB_REGRESS = 1e-2   # internal regression bar for bf16 (expected error ~3e-3)
# Per-element bars (every element, beside the normwise ones above).  float32:
# |y - y_ref| <= F32_ELEM * (|y_ref| + rms(y_ref)); the float32 path's errors
# are ~2e-7 of that scale (accumulation order, the erf approximation).
# bfloat16: |y - y_ref| <= 2^-8 |y_ref| + BF16_ELEM_RMS * rms(y_ref): the
# output rounding is at most 2^-9 |y_ref|, and the roundings of z, t and u to
# bfloat16 add an absolute error that scales with the size of the sums, i.e.
# with rms(y_ref) (at most 0.021 rms(y_ref) when those roundings are replayed
# in double on 2000 rows of the DeiT-Small and DeiT-Base layers).
F32_ELEM = 1e-5
BF16_ELEM_REL = 2.0 ** -8
BF16_ELEM_RMS = 0.05
# Tokens excluded as near ties may be at most this share of a test's tokens
# (and at most one token when there are fewer than 1000).
EXCL_MAX = 1e-3


def dev(a):
    return None if a is None else cm.from_stored(a)


def layer_to_device(L):
    return {n: dev(L[n]) for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg", "bg")}


def gpu_ffn(L, ws=None, with_routing=True, padded=False):
    """The whole layer through clearmoe_ffn_forward (or, with padded=True,
    clearmoe_ffn_forward_padded)."""
    d = layer_to_device(L)
    T, k = L["cfg"].T, L["cfg"].k
    idx = torch.empty((T, k), dtype=torch.int32, device="cuda") if with_routing else None
    gate = torch.empty((T, k), dtype=torch.float32, device="cuda") if with_routing else None
    fwd = cm.ffn_forward_padded if padded else cm.ffn_forward
    y = fwd(d["x"], d["W1"], d["b1"], d["US"], d["Vt"], d["b2"], d["P"], d["Q"], d["Wg"],
            d["bg"], k, ws=ws, idx_out=idx, gate_out=gate, renorm=int(L.get("renorm", 1)))
    torch.cuda.synchronize()
    out = dict(y=oracle.widen(cm.to_stored(y)))
    if with_routing:
        out["idx"] = idx.cpu().numpy()
        out["gate"] = gate.cpu().numpy()
    return out


def frob_rel(y, ref):
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(y - ref) / den) if den > 0 else float(np.linalg.norm(y))


def assert_elementwise(y, ref, dtype):
    """Every element within the per-element bar of its storage type."""
    y, ref = np.asarray(y), np.asarray(ref)
    if ref.size == 0:
        return
    rms = float(np.sqrt(np.mean(ref * ref)))
    err = np.abs(y - ref)
    if dtype == "f32":
        bound = F32_ELEM * (np.abs(ref) + rms)
    else:
        bound = BF16_ELEM_REL * np.abs(ref) + BF16_ELEM_RMS * rms
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert np.all(err <= bound), (f"element {worst}: |err| {err[worst]:.3e} > bound "
                                  f"{bound[worst]:.3e} (rms {rms:.3e})")


def max_rel(y, ref):
    den = np.max(np.abs(ref)) if ref.size else 0.0
    return float(np.max(np.abs(y - ref)) / den) if den > 0 else float(np.max(np.abs(y), initial=0))


def bound_excluded(mask, what="near-tie"):
    """Print how many tokens a comparison leaves out and bound their share: at
    most EXCL_MAX of the tokens (one token below 1000 tokens)."""
    mask = np.asarray(mask, dtype=bool)
    n, N = int(mask.sum()), int(mask.size)
    print(f"excluded {what} tokens: {n} of {N} ({n / max(N, 1):.2e})")
    assert n <= max(1, int(EXCL_MAX * N)), f"{n} of {N} tokens excluded ({what})"
    return mask


def assert_routing(idx_gpu, logits_ref, k):
    """idx bit-exact wherever the oracle's margin >= MARGIN.  Returns the mask of
    tokens that are allowed to differ (near ties), whose share is bounded."""
    idx_ref, _ = oracle.topk(logits_ref, k)
    tie = bound_excluded(oracle.margins(logits_ref, k) < MARGIN)
    bad = np.any(idx_gpu != idx_ref, axis=1) & ~tie
    assert not bad.any(), f"{bad.sum()} tokens routed differently (first {np.nonzero(bad)[0][:5]})"
    return tie


def assert_gates(gate_gpu, logits_ref, idx_gpu, k, tie, renorm=1):
    """Gates against the oracle's double gates (float32 rounding), on the tokens
    where the GPU made the oracle's choice: renormalised over the chosen
    experts (renorm 1) or their probabilities under the softmax over all E
    (renorm 0)."""
    i, g = oracle.topk(logits_ref, k)
    if not renorm:
        g = oracle.full_softmax_gates(logits_ref, i)
    ok = ~tie
    err = np.abs(gate_gpu[ok] - g[ok])
    # gates come from float32 logits whose choice is certified (double for near ties)
    assert np.all(err <= 2e-5), float(err.max())
    if k == 1 and renorm:
        assert np.all(gate_gpu == 1.0)


def check_dispatch(idx_gpu, E, counts, offsets, perm, inv):
    """Bit-exact against the oracle's dispatch of the same indices."""
    c, o, p, i = oracle.dispatch(idx_gpu, E)
    assert np.array_equal(counts, c)
    assert np.array_equal(offsets, o)
    assert np.array_equal(perm, p)
    assert np.array_equal(inv, i)


def gpu_router(L, d=None):
    """A cm.Router for a layer dict (linear, or the "router" entry's MLP /
    adaptive variant) and the device tensors it points at (keep them alive)."""
    rt = L.get("router") or {"kind": "linear"}
    keep = {"Wg": dev(L["Wg"]), "bg": dev(L["bg"])}
    if rt["kind"] == "mlp":
        keep["Wh"], keep["bh"] = dev(rt["Wh"]), dev(rt["bh"])
    stride = int(L.get("dense_stride") or 0)
    if stride > 0:
        keep["W2"] = dev(L["W2"])
    r = cm.make_router(keep["Wg"], keep["bg"], keep.get("Wh"), keep.get("bh"),
                       adaptive=rt.get("adaptive", rt["kind"] == "adaptive"),
                       tau=rt.get("tau", 0.0), dense_stride=stride, W2=keep.get("W2"))
    return r, keep


def gpu_ffn_ex(L):
    """The whole layer through clearmoe_ffn_forward_ex with the layer's router."""
    d = layer_to_device(L)
    T, k = L["cfg"].T, L["cfg"].k
    r, keep = gpu_router(L)
    idx = torch.empty((T, k), dtype=torch.int32, device="cuda")
    gate = torch.empty((T, k), dtype=torch.float32, device="cuda")
    y = cm.ffn_forward_ex(d["x"], d["W1"], d["b1"], d["US"], d["Vt"], d["b2"], d["P"], d["Q"], r,
                          k, idx_out=idx, gate_out=gate, renorm=int(L.get("renorm", 1)))
    torch.cuda.synchronize()
    del keep
    return dict(y=oracle.widen(cm.to_stored(y)), idx=idx.cpu().numpy(), gate=gate.cpu().numpy())


def rounding_gap(v, dtype):
    """Distance of each exact value to the nearest rounding midpoint of the
    storage type, relative to the value's binade (0 = exactly halfway)."""
    bits = 8 if dtype == "bf16" else 24
    m, _ = np.frexp(np.asarray(v, dtype=np.float64))
    frac = np.ldexp(np.abs(m), bits)
    return np.abs(frac - np.floor(frac) - 0.5) * 2.0 ** -bits


def confidence_gap(logits, tau):
    """|log p - log tau| of the adaptive router's confidence p (inf if tau <= 0)."""
    if tau <= 0:
        return np.full(np.asarray(logits).shape[0], np.inf)
    return np.abs(np.log(oracle.confidence(logits)) - np.log(tau))
