#!/usr/bin/env python3
"""Benchmark of the CLEAR-MoE FFN forward on one MI355X.

A step is one clearmoe_ffn_forward call (router, dispatch, fc1 + GELU, shared
SVD basis, grouped residual experts, combine) over the DeiT-Base-shaped layer,
the largest configuration: T = 256 x 197 = 50432 tokens, D = 768, H = 3072,
E = 8, top-2 with renormalised gates, r = 256, q = 64, bf16 storage with
float32 accumulation, synthetic seeded inputs already in HBM.

Prints one JSON line.  Besides the contract fields it carries
  roofline     the dominant kernel's algorithmic rate (HIP events written by
               the kernel's own dispatch, on its stream, for every launch of
               it in the timed region, at least 20) against its MI355X peak,
               plus measured HBM traffic when counters exist for the current
               kernel source;
  cpu_baseline the CPU oracle on a bounded sample of the same workload, on all
               host threads and on one (the analogue of the paper's serial
               CPU row), with the CPU model;
  stages       per-kernel times of one step;
  cold         the step with the 256 MB last-level cache flushed before it;
  dense        the dense fc1 + GELU + fc2 comparator through the same kernels;
  deit_small   the DeiT-Small-shaped top-1 layer (12608 tokens, D = 384), the
               fused kernel, with its own roofline and dense comparator;
  dispatch     the routing/dispatch-only workload (2^20 tokens, D = 384, E = 8,
               top-2, Zipf-skewed bias): route -> dispatch (+ rows) -> combine,
               with its HBM fraction;
  imbalance    the dispatch-backend sweep: grouped (clearmoe_ffn_forward)
               against padded batches (clearmoe_ffn_forward_padded) at 0, 40,
               60 and 80 % load imbalance, E = 4, DeiT-Small widths, top-1 and
               top-2, 1568 and 12608 tokens;
  routers      the DeiT-Small layer with the linear, MLP and adaptive routers
               (clearmoe_ffn_forward_ex);
  deit_tiny    the DeiT-Tiny-shaped fp32 layer (1576 tokens, D = 192);
  expert_sweep the DeiT-Small shape for E = 2, 4, 6, 8 beside the dense FFN;
  ffn_stack    the FFN part of a 12-block DeiT-Small forward with 6 CLEAR-MoE
               layers (class tokens on the dense path) against 12 dense ones.
"""
import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
PROFILE_DIR = os.path.join(ROOT, "profiles")
TIME_EVERY = 8          # sampling of the dominant kernel's timed launches in short steps
MIN_TIMED = 20          # timed launches of the dominant kernel, at least
# stages whose kernels are matrix products (the router's flops are not its bound)
MFMA_STAGES = ("fc1_gelu", "basis_t", "basis_h", "res_u", "res_h", "tu_grouped", "y_grouped",
               "tu_pair", "y_pair", "dense_fc2", "fused_top1")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="only the timed steps (for profiler runs)")
    ap.add_argument("--workload", default="C3", choices=["C1", "C2", "C3"])
    ap.add_argument("--traffic-probe", action="store_true",
                    help="for counter runs: one 1 GiB device copy from a cache-cold source "
                         "(known bytes, to scale the counters), then the timed steps only")
    ap.add_argument("--dispatch-probe", action="store_true",
                    help="for counter runs: the copy of --traffic-probe, then --steps passes "
                         "of the 2^20-token dispatch workload only")
    return ap.parse_args()


KERNEL_SOURCES = {
    "route": ["route.hip"], "tile_hist": ["dispatch.hip"], "scan": ["dispatch.hip"],
    "permute": ["dispatch.hip"], "combine": ["dispatch.hip"], "combine_res": ["dispatch.hip"],
    "fused_top1": ["fused_kernel.h", "fused_body.inc", "class_ffn.h", "fused.hip", "fused_split.hip",
                   "fused_cls.hip"],
    "pair_key": ["dispatch.hip"], "residual_add": ["dispatch.hip"],
}


def source_digest(kernel=None):
    """Hash of the HIP sources a kernel is built from (its own file and the shared
    header; GEMM stages: gemm.hip), or of all of them: counters taken on other
    code are not reported."""
    h = hashlib.sha256()
    cdir = os.path.join(ROOT, "paper_2606_28516_amd", "csrc")
    if kernel is None:
        names = sorted(os.listdir(cdir))
    else:
        names = sorted(KERNEL_SOURCES.get(kernel, ["gemm.hip"]) + ["kernels.h"])
    for name in names:
        with open(os.path.join(cdir, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def stage_work(stage, cfg, b):
    """Algorithmic (flops, bytes) of one launch of a stage of the layer.
    b = bytes per stored element; h_sh and h_res are float32."""
    T, D, H, E, k, r, q = cfg.T, cfg.D, cfg.H, cfg.E, cfg.k, cfg.r, cfg.q
    A = T * k
    w = {
        "route": (2 * T * D * E, T * D * b + E * D * b + A * 8),
        "scan": (0, 8 * ((T + 255) // 256) * E),
        "permute": (0, A * 4 + A * 8),
        "fc1_gelu": (2 * T * H * D, T * D * b + H * D * b + T * H * b),
        "basis_t": (2 * T * r * H, T * H * b + r * H * b + T * r * b),
        "basis_h": (2 * T * D * r, T * r * b + D * r * b + T * D * 4),
        "res_u": (2 * A * q * H, A * H * b + E * q * H * b + A * q * b),
        "res_h": (2 * A * D * q, A * q * b + E * D * q * b + A * D * 4),
        "combine_res": (0, T * D * 4 + A * D * 4 + A * 4 + T * D * b),
        "dense_fc2": (2 * T * D * H, T * H * b + D * H * b + T * D * b),
        "tu_grouped": (2 * A * (r + q) * H, A * H * b + (r + E * q) * H * b + A * (r + q) * b),
        "y_grouped": (2 * A * D * (r + q), A * (r + q) * b + D * (r + E * q) * b + T * D * b),
        # top-2 in expert-pair order: one row per token with its two experts
        "tu_pair": (2 * T * (r + 2 * q) * H, T * H * b + (r + E * q) * H * b + T * (r + 2 * q) * b),
        "y_pair": (2 * T * D * (r + 2 * q), T * (r + 2 * q) * b + D * (r + E * q) * b + T * D * b),
        "pair_key": (0, A * 8 + T * 12),
        "tile_hist": (0, T * 4 + 4 * ((T + 63) // 64) * (E + E * (E - 1) // 2)),
        # x in, y out; W1, [Vt;Q_e] and [US|P_e] once each; b1, b2; the expert
        # index of every token and the router's tile histogram
        "fused_top1": (2 * T * (D * H + H * (r + q) + (r + q) * D),
                       2 * T * D * b + H * D * b + 2 * (r + E * q) * (H + D) * b // 2
                       + (H + D) * 4 + T * 4 + 4 * E * ((T + 63) // 64 if E <= 16 else (T + 255) // 256)),
    }
    return w.get(stage, (0, 0))


def layer_flops(cfg):
    T, D, H, E, k, r, q = cfg.T, cfg.D, cfg.H, cfg.E, cfg.k, cfg.r, cfg.q
    return 2 * T * (D * H + H * r + r * D + k * (H * q + q * D) + D * E)


def load_traffic(kernel, workload, digest):
    """Measured HBM bytes per launch from a committed counter summary, if it was
    taken on the current kernel source."""
    path = os.path.join(PROFILE_DIR, f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_digest") != digest:
        return None
    return t.get("hbm_bytes_per_launch")


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE {world}); the path shards by tokens with no exchange, see the "
              f"design notes", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_28516_amd import clearmoe as cm
    from paper_2606_28516_amd import synth

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.dispatch_probe:
        copy_probe(torch, torch.device("cuda:0"))
        bench_dispatch(cm, synth, torch, None, torch.cuda.current_stream(), args.steps, timed=False)
        print(json.dumps({"dispatch_probe": True, "steps": args.steps}), flush=True)
        return
    cfg = synth.CONFIGS[args.workload]
    L = synth.make_layer(cfg)
    core = measure_layer(cm, torch, cfg, L, args.steps, args.warmup, args.traffic_probe)
    if core is None:            # traffic probe run: nothing to report
        return
    step, d, ws, y, stream = core.pop("_step"), core.pop("_d"), core.pop("_ws"), core.pop("_y"), \
        core.pop("_stream")
    b = 4 if cfg.dtype == "f32" else 2
    ms_step = core["ms_per_step"]

    out = {
        "metric": "tokens/sec per CLEAR-MoE FFN layer + % HBM peak (dispatch) / % MFMA peak (GEMM)",
        "value": core["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded Gaussian-cluster tokens, N(0,0.02) weights, SVD-extracted basis)",
        "config": {"workload": cfg.name, "tokens": cfg.T, "D": cfg.D, "H": cfg.H, "E": cfg.E,
                   "k": cfg.k, "r": cfg.r, "q": cfg.q, "seed": cfg.seed},
        "roofline": core["roofline"],
        "step_ms": core["step_ms"],
        "layer_tflops": core["layer_tflops"],
        "stages_us": core["stages_us"],
        "wall_s": core["wall_s"],
        "source_digest": source_digest(),
    }

    if not args.no_extras:
        out["cold"] = time_cold(torch, np, step, stream, cfg)
        out["dense"] = time_dense(cm, synth, torch, np, cfg, L, d, ws, stream, args.steps,
                                  args.warmup, ms_step)
        out["products"] = bench_layer(cm, synth, torch, np, stream, None, 20, cfg=cfg, L=L,
                                      d=d, ws=ws)["stages"]
        del d, ws, y, step
        # the DeiT-Small top-1 layer (fused kernel) with its own roofline
        c2 = synth.CONFIGS["C2"]
        L2 = synth.make_layer(c2)
        small = measure_layer(cm, torch, c2, L2, max(args.steps, 100), args.warmup)
        step2, d2, ws2, _y2, _ = (small.pop(k) for k in ("_step", "_d", "_ws", "_y", "_stream"))
        small["workload"] = f"{c2.name} (T={c2.T} D={c2.D} H={c2.H} E={c2.E} k={c2.k} r={c2.r} q={c2.q} bf16)"
        small["cold"] = time_cold(torch, np, step2, stream, c2)
        small["dense"] = time_dense(cm, synth, torch, np, c2, L2, d2, ws2, stream,
                                    max(args.steps, 100), args.warmup, small["ms_per_step"])
        out["deit_small"] = small
        del d2, ws2, _y2, step2
        out["dispatch"] = bench_dispatch(cm, synth, torch, np, stream, max(10, args.steps // 10))
        out["imbalance"] = bench_imbalance(cm, synth, torch, np, stream, max(20, args.steps // 5))
        out["routers"] = bench_routers(cm, synth, torch, np, stream, L2, max(20, args.steps // 5))
        out["ffn_stack"] = bench_stack(cm, synth, torch, np, stream, L2, max(20, args.steps // 10))
        out["deit_tiny"] = bench_layer(cm, synth, torch, np, stream, "C1", 100)
        dense_ms = small["dense"]["ms_per_step"]
        sweep = {}
        for e in (2, 4, 6, 8):
            r = bench_layer(cm, synth, torch, np, stream, f"C5-E{e}", 100)
            sweep[f"E{e}"] = {"ms": r["ms"], "tokens_per_s": r["tokens_per_s"],
                              "moe_over_dense_time": r["ms"] / dense_ms,
                              "stages_us": {k: v["us"] for k, v in r["stages"].items()}}
        out["expert_sweep"] = {"workload": "DeiT-Small shape (12608 tokens, D = 384, H = 1536, r = 128, "
                                           "q = 32, bf16, top-1) for E in {2, 4, 6, 8}, uniform "
                                           "clusters, seed 4; dense = the DeiT-Small dense comparator",
                               "points": sweep}

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(L, cfg, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def time_cold(torch, np, step, stream, cfg):
    """The step with the 256 MB last-level cache flushed (512 MiB written)
    before each of 30 timed calls; median."""
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    times = []
    for _ in range(30):
        flush.fill_(1)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        step()
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    del flush
    cold = float(np.median(times))
    return {"ms_per_step": cold, "tokens_per_s": cfg.T / (cold * 1e-3)}


def time_dense(cm, synth, torch, np, cfg, L, d, ws, stream, steps, warmup, moe_ms):
    """The dense FFN of the same shape, GELU(x W1^T + b1) W2^T + b2 with the
    layer's pre-extraction fc2, through the same GEMM kernels."""
    W2 = cm.from_stored(L["W2"].astype(np.float32) if cfg.dtype == "f32"
                        else synth.to_bf16_bits(L["W2"]))
    yd = torch.empty_like(d["x"])

    def dense():
        cm.dense_ffn_forward(d["x"], d["W1"], d["b1"], W2, d["b2"], ws=ws, out=yd)

    for _ in range(warmup):
        dense()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        dense()
    e1.record(stream)
    torch.cuda.synchronize()
    dms = e0.elapsed_time(e1) / steps
    return {"ms_per_step": dms, "tokens_per_s": cfg.T / (dms * 1e-3),
            "moe_over_dense_time": moe_ms / dms,
            "tflops": 4 * cfg.T * cfg.D * cfg.H / (dms * 1e-3) / 1e12}


def copy_probe(torch, dev):
    """One device copy of exactly 1 GiB from a cache-cold source: the known
    bytes that scale the FETCH_SIZE / WRITE_SIZE counters of a counter run."""
    src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    flush.fill_(2)                  # evicts src from the 256 MB last-level cache
    torch.cuda.synchronize()
    dst.copy_(src)                  # reads and writes exactly 1 GiB
    torch.cuda.synchronize()
    del src, dst, flush


def measure_layer(cm, torch, cfg, L, steps, warmup, traffic_probe=False):
    """Warm up, find the dominant kernel from a per-stage pass, then time
    exactly `steps` layer calls between two events on the stream, with the
    dominant kernel's own dispatch writing start/end events for at least
    MIN_TIMED of its launches (every launch when the step is long, one in
    TIME_EVERY when a timed dispatch would be a visible share of the step;
    with too few steps for that, every launch)."""
    dev = torch.device("cuda:0")
    b = 4 if cfg.dtype == "f32" else 2
    d = {n: cm.from_stored(L[n]) for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg", "bg")}
    shape = cm.make_shape(cfg.T, cfg.D, cfg.E, cfg.k, cm.F32 if cfg.dtype == "f32" else cm.BF16,
                          H=cfg.H, r=cfg.r, q=cfg.q)
    ws = cm.alloc_workspace(shape)
    y = torch.empty((cfg.T, cfg.D), dtype=d["x"].dtype, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        cm.ffn_forward(d["x"], d["W1"], d["b1"], d["US"], d["Vt"], d["b2"], d["P"], d["Q"],
                       d["Wg"], d["bg"], cfg.k, ws=ws, out=y)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    if traffic_probe:
        copy_probe(torch, dev)
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        print(json.dumps({"traffic_probe": True, "workload": cfg.name, "steps": steps}), flush=True)
        return None

    # Per-stage times of a few steps (all stages timed) to find the dominant kernel.
    names = cm.stage_names()
    cm.timing_start(names, 64 * len(names))
    for _ in range(20):
        step()
    per = cm.timing_stop()
    stages = {s_: ms / n for s_, (ms, n) in per.items()}
    dominant = max(stages, key=stages.get)
    # a timed dispatch costs a few microseconds: sample one launch in
    # TIME_EVERY only when the step is short and the steps are many
    every = TIME_EVERY if sum(stages.values()) < 0.25 else 1
    every = max(1, min(every, steps // MIN_TIMED))

    cm.timing_start([dominant], max(steps, 1), every=every)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dom_ms, dom_n = cm.timing_stop()[dominant]
    ms_step = ev0.elapsed_time(ev1) / steps
    # spread of single steps (a separate pass after the timed one, an event
    # pair around each call)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(max(steps, 1))]
    for e0, e1 in pairs:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    per_step = sorted(e0.elapsed_time(e1) for e0, e1 in pairs)
    pct = {f"p{p}": per_step[min(len(per_step) - 1, round(p / 100 * (len(per_step) - 1)))]
           for p in (10, 50, 90)}

    flops, byts = stage_work(dominant, cfg, b)
    dom_avg_s = dom_ms / dom_n * 1e-3
    digest = source_digest(dominant)
    if flops > 0:
        roof = dict(bound="mfma", achieved=flops / dom_avg_s / 1e12,
                    peak=MFMA_PEAK_TFLOPS[cfg.dtype], unit="TFLOP/s")
    else:
        roof = dict(bound="hbm", achieved=byts / dom_avg_s / 1e9, peak=HBM_PEAK_GBS, unit="GB/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = load_traffic(dominant, cfg.name.split("-")[0], digest)
    roof["kernel"] = dominant
    roof["avg_launch_us"] = dom_avg_s * 1e6
    roof["timed_launches"] = dom_n
    roof["algorithmic_per_launch"] = flops if flops > 0 else byts
    if flops > 0:
        roof["attainable"] = min(roof["peak"], flops / byts * HBM_PEAK_GBS / 1e3)
        roof["frac_attainable"] = roof["achieved"] / roof["attainable"]
    return {"value": cfg.T / (ms_step * 1e-3), "ms_per_step": ms_step, "roofline": roof,
            "step_ms": pct,
            "layer_tflops": layer_flops(cfg) / (ms_step * 1e-3) / 1e12,
            "stages_us": {s_: v * 1e3 for s_, v in sorted(stages.items(), key=lambda kv: -kv[1])},
            "wall_s": wall, "_step": step, "_d": d, "_ws": ws, "_y": y, "_stream": stream}


def bench_dispatch(cm, synth, torch, np, stream, steps, timed=True):
    """Route -> dispatch (rows copied into expert order) -> gated combine on the
    2^20-token workload.  HBM fraction against compulsory bytes (x read once)
    and against the bytes this design moves (x read by route and by permute)."""
    L = synth.make_dispatch()
    c = L["cfg"]
    T, D, E, k = c["T"], c["D"], c["E"], c["k"]
    x, Wg, bg = cm.from_stored(L["x"]), cm.from_stored(L["Wg"]), cm.from_stored(L["bg"])
    del L
    s = cm.make_shape(T, D, E, k, cm.BF16)
    ws = cm.alloc_workspace(s)
    dev = x.device
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    gate = torch.empty((T, k), dtype=torch.float32, device=dev)
    counts = torch.empty(E, dtype=torch.int32, device=dev)
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
    perm = torch.empty(T * k, dtype=torch.int32, device=dev)
    inv = torch.empty(T * k, dtype=torch.int32, device=dev)
    xperm = torch.empty((T * k, D), dtype=x.dtype, device=dev)
    y = torch.empty_like(x)
    Lb = cm.lib()
    import ctypes

    sp = ctypes.byref(s)
    st = ctypes.c_void_p(stream.cuda_stream)
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731

    def run():
        rc = Lb.clearmoe_route(sp, P(x), P(Wg), P(bg), P(idx), P(gate), P(ws), ws.numel(), st)
        rc |= Lb.clearmoe_dispatch(sp, P(idx), P(ws), ws.numel(), P(counts), P(offsets), P(perm),
                                   P(inv), P(x), P(xperm), cm.DISPATCH_HIST_IN_WS, st)
        rc |= Lb.clearmoe_combine(sp, P(xperm), P(inv), P(gate), P(y), st)
        if rc:
            raise cm.ClearMoEError("dispatch workload failed")

    for _ in range(3):
        run()
    torch.cuda.synchronize()
    if not timed:                   # counter runs: the passes alone
        for _ in range(steps):
            run()
        torch.cuda.synchronize()
        return None
    # untimed steps for the step time, then timed ones for the per-kernel times
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    names = cm.stage_names()
    cm.timing_start(names, steps * len(names))
    for _ in range(steps):
        run()
    per = cm.timing_stop()
    A = T * k
    b = 2
    # x read, xperm written and read, y written, idx/gate/perm/inv written, inv/gate read
    compulsory = T * D * b + 2 * A * D * b + T * D * b + A * 24
    moved = compulsory + T * D * b
    kern = {}
    kbytes = {"route": T * D * b + A * 8, "permute": A * 4 + T * D * b + A * 8 + A * D * b,
              "combine": A * 8 + A * D * b + T * D * b}
    for s_, (t_ms, n) in per.items():
        us = t_ms / n * 1e3
        e = {"us": us}
        if s_ in kbytes:
            e["GBs"] = kbytes[s_] / (us * 1e-6) / 1e9
            e["hbm_frac"] = e["GBs"] / HBM_PEAK_GBS
        kern[s_] = e
    return {"workload": "C4-dispatch-bf16 T=2^20 D=384 E=8 k=2 zipf1.2", "ms": ms,
            "tokens_per_s": T / (ms * 1e-3),
            "hbm_frac_compulsory": compulsory / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "hbm_frac_moved": moved / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "compulsory_GB": compulsory / 1e9, "moved_GB": moved / 1e9,
            "counts": counts.cpu().tolist(), "kernels": kern}


def bench_imbalance(cm, synth, torch, np, stream, steps):
    """Grouped against padded dispatch backends under load imbalance (the
    paper's dispatch benchmark: E = 4, imbalance 0/40/60/80 %, here at the
    DeiT-Small widths on MI355X).  Imbalance p draws a share p of the tokens
    from cluster 0 on top of an even spread (synth.imbalance_mixture); the
    realised expert loads are reported with each point.  Both backends compute
    the whole layer; tokens/s is per layer call, host waits included."""
    D, H, E, r, q = 384, 1536, 4, 128, 32
    out = []
    for T in (1568, 12608):
        for p in (0.0, 0.4, 0.6, 0.8):
            cfg = synth.LayerConfig(f"imbalance-{round(100 * p)}", T=T, D=D, H=H, E=E, k=1, r=r,
                                    q=q, dtype="bf16", seed=5, n_cal=4000,
                                    mixture=synth.imbalance_mixture(E, p))
            L = synth.make_layer(cfg)
            d = {n: cm.from_stored(L[n])
                 for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg", "bg")}
            del L
            y = torch.empty((T, D), dtype=d["x"].dtype, device=d["x"].device)
            for k in (1, 2):
                shape = cm.make_shape(T, D, E, k, cm.BF16, H=H, r=r, q=q)
                ws = torch.empty(cm.padded_workspace_bytes(shape), dtype=torch.uint8,
                                 device=y.device)
                idx = torch.empty((T, k), dtype=torch.int32, device=y.device)
                row = {"tokens": T, "imbalance": p, "k": k}
                for name, fwd in (("grouped", cm.ffn_forward), ("padded", cm.ffn_forward_padded)):
                    def run():
                        fwd(d["x"], d["W1"], d["b1"], d["US"], d["Vt"], d["b2"], d["P"], d["Q"],
                            d["Wg"], d["bg"], k, ws=ws, out=y, idx_out=idx)
                    for _ in range(5):
                        run()
                    torch.cuda.synchronize()
                    ms = float("inf")
                    for _ in range(2):   # best of two passes
                        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                        e0.record(stream)
                        for _ in range(steps):
                            run()
                        e1.record(stream)
                        torch.cuda.synchronize()
                        ms = min(ms, e0.elapsed_time(e1) / steps)
                    row[name] = {"ms": ms, "tokens_per_s": T / (ms * 1e-3)}
                counts = torch.bincount(idx.flatten().long(), minlength=E).cpu().numpy()
                row["counts"] = counts.tolist()
                row["padded_rows_over_assignments"] = E * int(counts.max()) / (T * k)
                row["padded_over_grouped_time"] = row["padded"]["ms"] / row["grouped"]["ms"]
                out.append(row)
                del ws, idx
            del d, y
    return {"workload": "DeiT-Small widths D=384 H=1536 r=128 q=32 bf16, E=4, seed 5",
            "steps": steps, "points": out}


def bench_routers(cm, synth, torch, np, stream, L, steps):
    """The same DeiT-Small-shaped layer with the paper's three routers
    (Sec. III Phase 4, Table C5): linear top-1, MLP top-1 (hidden d/6 = 64)
    and adaptive (linear scores, top-1 escalated to top-2 below the confidence
    threshold tau = 0.9: a token whose largest softmax probability is below
    0.9 takes two experts, about 30 % of this workload's tokens).  Per
    variant: ms per layer call, tokens/s, the router kernel's time and the
    share of tokens on two experts."""
    cfg = L["cfg"]
    d = {n: cm.from_stored(L[n]) for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q")}
    Lm = synth.with_mlp_router(L, seed=1)
    keep = {"Wg": cm.from_stored(L["Wg"]), "bg": cm.from_stored(L["bg"]),
            "Wo": cm.from_stored(Lm["Wg"]), "bo": cm.from_stored(Lm["bg"]),
            "Wh": cm.from_stored(Lm["router"]["Wh"]), "bh": cm.from_stored(Lm["router"]["bh"])}
    tau = 0.9
    variants = [
        ("linear", cm.make_router(keep["Wg"], keep["bg"]), 1),
        ("mlp", cm.make_router(keep["Wo"], keep["bo"], keep["Wh"], keep["bh"]), 1),
        ("adaptive", cm.make_router(keep["Wg"], keep["bg"], adaptive=True, tau=tau), 2),
    ]
    out = {"workload": f"{cfg.name} (T={cfg.T} D={cfg.D} H={cfg.H} E={cfg.E} r={cfg.r} "
                       f"q={cfg.q} bf16)", "mlp_hidden": int(Lm["router"]["Wh"].shape[0]),
           "adaptive_tau": tau, "steps": steps, "variants": {}}
    dev = d["x"].device
    for name, router, k in variants:
        shape = cm.make_shape(cfg.T, cfg.D, cfg.E, k, cm.BF16, H=cfg.H, r=cfg.r, q=cfg.q)
        ws = cm.alloc_workspace(shape)
        y = torch.empty((cfg.T, cfg.D), dtype=d["x"].dtype, device=dev)
        idx = torch.empty((cfg.T, k), dtype=torch.int32, device=dev)

        def run():
            cm.ffn_forward_ex(d["x"], d["W1"], d["b1"], d["US"], d["Vt"], d["b2"], d["P"],
                              d["Q"], router, k, ws=ws, out=y, idx_out=idx)
        for _ in range(5):
            run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        cm.timing_start(["route"], steps)
        for _ in range(steps):
            run()
        r_ms, r_n = cm.timing_stop()["route"]
        two = float((idx[:, 1] >= 0).float().mean()) if k == 2 else 0.0
        out["variants"][name] = {"ms": ms, "tokens_per_s": cfg.T / (ms * 1e-3),
                                 "route_us": r_ms / r_n * 1e3, "share_top2": two}
        del ws, y, idx
    return out


def bench_layer(cm, synth, torch, np, stream, workload, steps, cfg=None, L=None, d=None,
                ws=None):
    """One layer of another configuration (a named workload, or cfg): step
    time from an untimed pass, then every stage timed in a second pass; MFMA
    rate of each product.  L, d and ws may be passed in when they exist."""
    cfg = cfg if cfg is not None else synth.CONFIGS[workload]
    if d is None:
        L = synth.make_layer(cfg) if L is None else L
        d = {n: cm.from_stored(L[n])
             for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg", "bg")}
    if ws is None:
        shape = cm.make_shape(cfg.T, cfg.D, cfg.E, cfg.k,
                              cm.F32 if cfg.dtype == "f32" else cm.BF16, H=cfg.H, r=cfg.r, q=cfg.q)
        ws = cm.alloc_workspace(shape)
    y = torch.empty_like(d["x"])

    def step():
        cm.ffn_forward(d["x"], d["W1"], d["b1"], d["US"], d["Vt"], d["b2"], d["P"], d["Q"],
                       d["Wg"], d["bg"], cfg.k, ws=ws, out=y)

    for _ in range(3):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    names = cm.stage_names()
    cm.timing_start(names, steps * len(names))
    for _ in range(steps):
        step()
    per = cm.timing_stop()
    b = 4 if cfg.dtype == "f32" else 2
    peak = MFMA_PEAK_TFLOPS[cfg.dtype]
    stages = {}
    for s_, (t_ms, n) in sorted(per.items(), key=lambda kv: -kv[1][0]):
        us = t_ms / n * 1e3
        flops = stage_work(s_, cfg, b)[0] if s_ in MFMA_STAGES else 0
        e = {"us": us}
        if flops:
            e["tflops"] = flops / (us * 1e-6) / 1e12
            e["mfma_frac"] = e["tflops"] / peak
            # against the attainable rate min(peak, AI x HBM) of its
            # algorithmic flops and bytes
            byts = stage_work(s_, cfg, b)[1]
            attain = min(peak, flops / byts * HBM_PEAK_GBS / 1e3)
            e["attainable_tflops"] = attain
            e["attainable_frac"] = e["tflops"] / attain
        stages[s_] = e
    del ws, y, d
    return {"workload": f"{cfg.name} (T={cfg.T} D={cfg.D} H={cfg.H} E={cfg.E} k={cfg.k} "
                        f"r={cfg.r} q={cfg.q} {cfg.dtype})",
            "ms": ms, "tokens_per_s": cfg.T / (ms * 1e-3),
            "layer_tflops": layer_flops(cfg) / (ms * 1e-3) / 1e12, "stages": stages, "steps": steps}


def bench_stack(cm, synth, torch, np, stream, L, steps):
    """The FFN part of a DeiT-Small forward as one chain (clearmoe_stack_forward):
    12 blocks with their own weights, each adding its input back (x + f(x));
    six are CLEAR-MoE (Sec. III Phase 2 keeps the best-scoring L/2; here
    blocks 6..11, the order does not change the timing) with each image's
    class token on the dense path (Table C6), six stay dense.  Compared with
    the chain of 12 dense blocks through the same kernels: the FFN-only
    analogue of the paper's model-level CLEAR-MoE / dense latency ratio
    (Table III).  Attention and layer norms are not part of this path."""
    cfg = L["cfg"]
    x = cm.from_stored(L["x"])
    keep, moe_stack, dense_stack = [], [], []
    for l in range(12):
        Ll = synth.make_layer(dataclasses.replace(cfg, name=f"block{l}", T=1, seed=100 + l,
                                                  n_cal=4000))
        W2 = cm.from_stored(synth.to_bf16_bits(Ll["W2"]))
        d = {n: cm.from_stored(Ll[n]) for n in ("W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg", "bg")}
        d["W2"] = W2
        keep.append(d)
        dense = cm.make_stack_layer(d["W1"], d["b1"], d["b2"], W2=W2)
        dense_stack.append(dense)
        if l >= 6:
            router = cm.make_router(d["Wg"], d["bg"], dense_stride=197, W2=W2)
            moe_stack.append(cm.make_stack_layer(d["W1"], d["b1"], d["b2"], d["US"], d["Vt"],
                                                 d["P"], d["Q"], router, k=cfg.k, W2=W2))
        else:
            moe_stack.append(dense)
    shape = cm.stack_shape(x, cfg.H, cfg.E, cfg.r, cfg.q)
    ws = torch.empty(cm.stack_workspace_bytes(shape, moe_stack), dtype=torch.uint8,
                     device=x.device)
    y = torch.empty_like(x)

    def timed(layers):
        for _ in range(3):
            cm.stack_forward(x, layers, cfg.H, cfg.E, cfg.r, cfg.q, ws=ws, out=y)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            cm.stack_forward(x, layers, cfg.H, cfg.E, cfg.r, cfg.q, ws=ws, out=y)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    # three interleaved passes of each, the best of each kept (clock and
    # cache state drift between passes hits both alike)
    mixed, all_dense = float("inf"), float("inf")
    for _ in range(3):
        mixed = min(mixed, timed(moe_stack))
        all_dense = min(all_dense, timed(dense_stack))
    del keep
    return {"workload": f"12 chained FFN blocks (x + f(x)) at {cfg.name} (T={cfg.T}), blocks 6..11 "
                        f"CLEAR-MoE top-{cfg.k} with class tokens on the dense path, 0..5 dense; "
                        f"own weights per block", "ms": mixed,
            "tokens_per_s": cfg.T / (mixed * 1e-3), "dense_ms": all_dense,
            "moe_over_dense_time": mixed / all_dense, "steps": steps}


def cpu_model():
    """The host CPU's model name and the threads this process may use."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return name, len(os.sched_getaffinity(0))


def _oracle_rate(oracle, np, L, cfg, blk, min_seconds):
    """Tokens per second of the oracle's layer on consecutive row blocks of
    the workload until at least min_seconds of CPU work have run."""
    done, t_used, start = 0, 0.0, 0
    while t_used < min_seconds:
        rows = np.arange(start, min(cfg.T, start + blk))
        t0 = time.perf_counter()
        oracle.ffn_forward_layer(L, rows=rows)
        t_used += time.perf_counter() - t0
        done += rows.size
        start = (start + blk) % cfg.T
    return done, t_used


def cpu_baseline(L, cfg, min_seconds):
    """The CPU oracle, as it stands, on the same workload's tokens: on every
    host thread the process may use (OpenMP over tokens) for at least
    min_seconds, and on one thread (the analogue of the paper's serial CPU
    row) for at least half that."""
    import numpy as np

    import oracle

    oracle.lib()
    model, visible = cpu_model()
    threads = oracle.num_threads()          # OpenMP's own count (OMP_NUM_THREADS where set)
    done, t_used = _oracle_rate(oracle, np, L, cfg, 2048, min_seconds)
    oracle.set_num_threads(1)
    done1, t1 = _oracle_rate(oracle, np, L, cfg, 128, 0.5 * min_seconds)
    oracle.set_num_threads(threads)
    return {"value": done / t_used, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": model, "host_threads_visible": visible,
            "sample": f"{done} tokens of {cfg.name} in blocks of 2048, {t_used:.1f} s, fp64 "
                      f"plain loops, OpenMP over tokens on {threads} threads",
            "serial": {"value": done1 / t1, "unit": "tokens/s", "cores": 1,
                       "sample": f"{done1} tokens in blocks of 128, {t1:.1f} s, one thread"}}


if __name__ == "__main__":
    main()
