"""Seeded synthetic inputs for the CLEAR-MoE FFN forward.

This module only draws and stores inputs.  It holds none of the forward
path's arithmetic (no router, GELU, GEMM or dispatch); both the HIP library's
tests/benchmark and the CPU oracle consume exactly the arrays it returns.

What it stands in for.  The paper calibrates on Imagenette activations of a
frozen DeiT (Sec. III, Phase 1) and extracts experts from the pretrained fc2
(Sec. III, Phase 3; Algorithm 2).  Neither data nor weights are available, so:

* tokens are drawn from a Gaussian mixture: centres of norm 3 in a random
  direction, per-token noise N(0, 1) (the cluster structure the router and
  the k-means of Phase 3 are meant to find);
* fc1 / fc2 weights are N(0, 0.02^2), biases zero (ViT initialisation scale);
* Phase 3's extraction is carried out on those weights as the paper states
  it: a truncated SVD of fc2 gives the shared basis (Eq. 2; Algorithm 2,
  first step) and the residual is the SVD tail scaled per cluster by s_e
  (Algorithm 2, the s_e and W_e^res steps);
* the mixture labels stand in for the k-means labels, and s_e is the ratio of
  the cluster-mean to the global-mean activation norm over a separate
  calibration draw of the recorded (pre-FFN) activations.

Storage: "f32" keeps float32 arrays; "bf16" stores bfloat16 bit patterns as
uint16 (round to nearest even from float32).  Biases are always float32.

Draw order (one PCG64 stream per call, ``numpy.random.default_rng(seed)``):
centres, labels, token noise, W1, W2, router noise, calibration labels,
calibration noise, and finally (``residual="random"`` only) P and Q.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Optional, Sequence

import numpy as np

__all__ = ["LayerConfig", "CONFIGS", "DISPATCH_CONFIG", "make_layer", "make_dispatch",
           "to_bf16_bits", "bf16_bits_to_f32", "fingerprint", "imbalance_mixture",
           "with_mlp_router", "with_adaptive_router", "with_class_tokens"]


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """Shape and input recipe of one CLEAR-MoE FFN layer."""
    name: str
    T: int                      # tokens
    D: int                      # model width d
    H: int                      # fc1 width d_ffn
    E: int                      # experts
    k: int                      # experts per token
    r: int                      # shared SVD rank
    q: int                      # residual rank per expert
    dtype: str                  # "f32" | "bf16"
    seed: int
    mixture: Optional[Sequence[float]] = None   # None = uniform over E clusters
    router: str = "centres_noise"              # "centres_unit" | "centres_noise"
    router_noise: float = 0.1
    router_bias: str = "zero"                  # "zero" | "zipf"
    zipf_s: float = 1.2
    residual: str = "svd_tail"                 # "svd_tail" | "random" | "zero"
    n_cal: int = 39400                         # calibration tokens (200 images x 197)
    n_clusters: Optional[int] = None           # default E


# The five workloads.  C4 is dispatch-only and has its own constructor.
CONFIGS = {
    "C1": LayerConfig("C1-deit-tiny-f32", T=8 * 197, D=192, H=768, E=4, k=1, r=64, q=16,
                      dtype="f32", seed=0, router="centres_unit"),
    "C2": LayerConfig("C2-deit-small-bf16", T=64 * 197, D=384, H=1536, E=8, k=1, r=128, q=32,
                      dtype="bf16", seed=1),
    "C3": LayerConfig("C3-deit-base-bf16-top2", T=256 * 197, D=768, H=3072, E=8, k=2, r=256,
                      q=64, dtype="bf16", seed=2,
                      mixture=(0.3, 0.2, 0.15, 0.1, 0.1, 0.05, 0.05, 0.05)),
}
for _e in (2, 4, 6, 8):
    CONFIGS[f"C5-E{_e}"] = LayerConfig(f"C5-deit-small-bf16-E{_e}", T=64 * 197, D=384, H=1536,
                                       E=_e, k=1, r=128, q=32, dtype="bf16", seed=4)

DISPATCH_CONFIG = dict(name="C4-dispatch-bf16", T=1 << 20, D=384, E=8, k=2, dtype="bf16",
                       seed=3, zipf_s=1.2)


def to_bf16_bits(a) -> np.ndarray:
    """float array -> bfloat16 bit patterns (uint16), round to nearest even."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "bf16":
        return to_bf16_bits(a)
    raise ValueError(f"unknown dtype {dtype!r}")


def imbalance_mixture(E: int, p: float) -> tuple:
    """Cluster mixture of the dispatch benchmark's imbalance level p in [0, 1):
    a share p of the tokens comes from cluster 0 on top of an even spread of
    the rest, i.e. weights (p + (1 - p) / E, (1 - p) / E, ...).  p = 0 is the
    balanced load.  (The paper sweeps 0/40/60/80 % imbalance without defining
    the term; this is the reading the benchmark and tests use.)"""
    if not 0.0 <= p < 1.0 or E < 1:
        raise ValueError("imbalance must be in [0, 1) and E >= 1")
    rest = (1.0 - p) / E
    return tuple([p + rest] + [rest] * (E - 1))


def _unit_rows(g: np.ndarray) -> np.ndarray:
    return g / np.linalg.norm(g, axis=1, keepdims=True)


def _mixture(cfg_mix, n: int) -> np.ndarray:
    if cfg_mix is None:
        return np.full(n, 1.0 / n)
    w = np.asarray(cfg_mix, dtype=np.float64)
    if w.shape != (n,):
        raise ValueError("mixture weights must have one entry per cluster")
    return w / w.sum()


def _draw_tokens(rng, centres, weights, n, dtype=np.float64):
    labels = rng.choice(len(weights), size=n, p=weights).astype(np.int32)
    x = rng.standard_normal((n, centres.shape[1]), dtype=dtype)
    x += centres[labels].astype(dtype)
    return labels, x


def make_layer(cfg: LayerConfig, **overrides) -> dict:
    """Draw one layer's inputs.  Returns a dict of stored arrays plus metadata.

    Keys: x [T,D], W1 [H,D], b1 [H], US [D,r], Vt [r,H], b2 [D], P [E,D,q],
    Q [E,q,H], Wg [E,D], bg [E], labels [T], s [E] (float64, svd_tail only),
    W2 [D,H] (float64, the pre-SVD fc2 this layer was extracted from),
    and "cfg".
    """
    if overrides:
        cfg = dataclasses.replace(cfg, **overrides)
    T, D, H, E, k, r, q = cfg.T, cfg.D, cfg.H, cfg.E, cfg.k, cfg.r, cfg.q
    if not (T >= 0 and D > 0 and H > 0 and 1 <= k <= E and 0 <= r <= min(D, H)
            and 0 <= q <= min(D, H)):
        raise ValueError(f"bad shape {cfg}")
    if cfg.residual == "svd_tail" and r + q > min(D, H):
        raise ValueError("svd_tail residual needs r + q <= min(D, H)")
    rng = np.random.default_rng(cfg.seed)
    ncl = cfg.n_clusters or E
    weights = _mixture(cfg.mixture, ncl)

    centres = 3.0 * _unit_rows(rng.standard_normal((ncl, D)))
    labels, x = _draw_tokens(rng, centres, weights, T)
    W1 = 0.02 * rng.standard_normal((H, D))
    W2 = 0.02 * rng.standard_normal((D, H))
    b1 = np.zeros(H)
    b2 = np.zeros(D)

    # Router rows: one per expert, built from the cluster centres (the router is
    # fitted to the cluster labels in Phase 4; its rows point at the centres).
    base = np.resize(centres, (E, D))
    if cfg.router == "centres_unit":
        Wg = _unit_rows(base)
        _ = rng.standard_normal((E, D))          # keep the draw order fixed
    elif cfg.router == "centres_noise":
        Wg = base + cfg.router_noise * rng.standard_normal((E, D))
    else:
        raise ValueError(cfg.router)
    if cfg.router_bias == "zero":
        bg = np.zeros(E)
    elif cfg.router_bias == "zipf":
        p = np.arange(1, E + 1, dtype=np.float64) ** (-cfg.zipf_s)
        bg = np.log(p / p.sum())
    else:
        raise ValueError(cfg.router_bias)

    # Phase 3 extraction: truncated SVD of fc2 (float64 LAPACK).
    U, S, Vh = np.linalg.svd(W2, full_matrices=False)
    US = U[:, :r] * S[:r]
    Vt = Vh[:r, :]

    # s_e: cluster-mean over global-mean activation norm on a calibration draw.
    cal_labels, cal_x = _draw_tokens(rng, centres, weights, cfg.n_cal)
    norms = np.linalg.norm(cal_x, axis=1)
    gmean = norms.mean()
    s = np.ones(E)
    for e in range(E):
        sel = norms[cal_labels == (e % ncl)]
        s[e] = (sel.mean() / gmean) if sel.size else 1.0

    if cfg.residual == "svd_tail":
        Pt = U[:, r:r + q] * S[r:r + q]                  # [D, q]
        P = np.stack([s[e] * Pt for e in range(E)])      # [E, D, q]
        Q = np.broadcast_to(Vh[r:r + q, :], (E, q, H)).copy()
    elif cfg.residual == "random":
        P = 0.1 * rng.standard_normal((E, D, q))
        Q = 0.05 * rng.standard_normal((E, q, H))
    elif cfg.residual == "zero":
        P = np.zeros((E, D, q))
        Q = np.zeros((E, q, H))
    else:
        raise ValueError(cfg.residual)

    dt = cfg.dtype
    return dict(
        cfg=cfg, x=_store(x, dt), W1=_store(W1, dt), b1=b1.astype(np.float32),
        US=_store(US, dt), Vt=_store(Vt, dt), b2=b2.astype(np.float32),
        P=_store(P, dt), Q=_store(Q, dt), Wg=_store(Wg, dt), bg=bg.astype(np.float32),
        labels=labels, s=s, W2=W2,
    )


def with_mlp_router(layer: dict, h: Optional[int] = None, seed: int = 0) -> dict:
    """The layer with an MLP router in place of the linear one (Sec. III
    Phase 4: one hidden layer of width h = d/6).  Stand-in for a router fitted
    to the cluster labels: the first E hidden units look along the linear
    router's rows (unit vectors towards the cluster centres), the other h - E
    are random N(0, 1/d) directions; the output layer reads hidden unit e with
    weight 2 for expert e plus N(0, 0.05^2) from every unit; biases zero.
    Adds "router" = {"kind": "mlp", "Wh" [h,D], "bh" [h]} and replaces Wg [E,h]
    and bg [E]."""
    cfg = layer["cfg"]
    D, E, dt = cfg.D, cfg.E, cfg.dtype
    h = D // 6 if h is None else h
    if h < E:
        raise ValueError("the MLP router needs h >= E")
    rng = np.random.default_rng(seed)
    lin = layer["Wg"]
    lin = bf16_bits_to_f32(lin) if lin.dtype == np.uint16 else lin
    Wh = rng.standard_normal((h, D)) / np.sqrt(D)
    Wh[:E] = _unit_rows(lin.astype(np.float64))
    Wo = 0.05 * rng.standard_normal((E, h))
    Wo[np.arange(E), np.arange(E)] += 2.0
    out = dict(layer)
    out["router"] = {"kind": "mlp", "Wh": _store(Wh, dt), "bh": np.zeros(h, np.float32)}
    out["Wg"] = _store(Wo, dt)
    out["bg"] = np.zeros(E, np.float32)
    return out


def with_adaptive_router(layer: dict, tau: float) -> dict:
    """The layer with the adaptive router (Sec. III Phase 4): the linear
    router's weights, top-1 escalated to top-2 below confidence tau.  The
    layer gets k = 2 slots per token."""
    out = dict(layer)
    out["cfg"] = dataclasses.replace(layer["cfg"], k=2)
    out["router"] = {"kind": "adaptive", "tau": float(tau)}
    return out


def with_class_tokens(layer: dict, stride: int = 197) -> dict:
    """The layer with one class token per image of `stride` tokens (token t
    with t % stride == 0; DeiT / ViT put it first): Table C6 excludes it from
    expert dispatch and runs it on the dense path, the original fc1 + GELU +
    fc2.  Adds "dense_stride" and stores "W2" in the storage precision (the
    dense path's fc2 weight as the kernels receive it)."""
    out = dict(layer)
    out["dense_stride"] = int(stride)
    out["W2"] = _store(layer["W2"], layer["cfg"].dtype)
    return out


def make_dispatch(T=None, D=None, E=None, k=None, dtype=None, seed=None, zipf_s=None) -> dict:
    """Inputs of the routing/dispatch-only workload: x [T,D], Wg [E,D], bg [E].

    Tokens from E uniform clusters (centre norm 3, N(0,1) noise); router rows
    are the centres plus N(0, 0.1^2); the router bias is log of a Zipf(s)
    distribution over experts, which skews the expert load.
    """
    c = dict(DISPATCH_CONFIG)
    for key, val in dict(T=T, D=D, E=E, k=k, dtype=dtype, seed=seed, zipf_s=zipf_s).items():
        if val is not None:
            c[key] = val
    T, D, E, k, dt = c["T"], c["D"], c["E"], c["k"], c["dtype"]
    rng = np.random.default_rng(c["seed"])
    centres = 3.0 * _unit_rows(rng.standard_normal((E, D)))
    labels = rng.choice(E, size=T).astype(np.int32)
    # Large T: draw float32 noise in row blocks to bound host memory.
    x = np.empty((T, D), dtype=np.float32)
    blk = 1 << 16
    for s0 in range(0, T, blk):
        s1 = min(T, s0 + blk)
        x[s0:s1] = rng.standard_normal((s1 - s0, D), dtype=np.float32)
        x[s0:s1] += centres[labels[s0:s1]].astype(np.float32)
    Wg = centres + 0.1 * rng.standard_normal((E, D))
    p = np.arange(1, E + 1, dtype=np.float64) ** (-c["zipf_s"])
    bg = np.log(p / p.sum())
    return dict(cfg=c, x=_store(x, dt), Wg=_store(Wg, dt), bg=bg.astype(np.float32),
                labels=labels)


def fingerprint(arrays: dict) -> str:
    """SHA-256 over every stored array (names sorted), for determinism checks."""
    h = hashlib.sha256()
    for name in sorted(arrays):
        v = arrays[name]
        if isinstance(v, np.ndarray):
            h.update(name.encode())
            h.update(str(v.dtype).encode())
            h.update(np.ascontiguousarray(v).tobytes())
    return h.hexdigest()
