#!/usr/bin/env python3
"""Throughput of the MoE-layer hot path on one MI355X.

One step = the whole layer (route -> permute -> grouped SwiGLU FFN [-> shared
expert] -> combine) over one synthetic expert batch whose inputs are already
resident in HBM.  The default workload is the Mixtral-shaped layer: 4096
tokens, hidden 4096, 8 experts, top-2, FFN dim 14336, bf16, near-uniform
routing.  Prints ONE JSON line on stdout; progress goes to stderr.

Per-kernel durations come from the library's own HIP-event profiler, recorded
on the launch stream inside the timed region.  The roofline figure is for the
dominant kernel, GEMM-1 (gate/up projections + SwiGLU): algorithmic flops
4*H*F*R per launch over its average launch duration, against the 2.5 PFLOP/s
dense bf16 MFMA peak.  The CPU baseline times the fp64 oracle on a bounded
sample of tokens of the same workload on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
METRIC = "MoE layer tokens/s + grouped-GEMM TFLOP/s (% bf16 MFMA peak) at 1 MI355X"

# Tokens of each workload the oracle processes for the CPU baseline (10-30 s of host work).
CPU_SAMPLE = {"tiny": 256, "mixtral4k": 4096, "mixtral32k_zipf": 4096, "deepseek": 2048,
              "memconstrained": 4096}


def gemm_source_sha256() -> str:
    """sha256 of the grouped-GEMM source (ffn.hip, then the common.h it includes)
    with comments removed and whitespace collapsed, so that only code changes
    invalidate counters taken on it."""
    import hashlib
    import re
    csrc = os.path.join(ROOT, "paper_2606_21712_amd", "csrc")
    h = hashlib.sha256()
    for name in ("ffn.hip", "common.h"):
        with open(os.path.join(csrc, name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)      # block comments
        text = re.sub(r"//[^\n]*", " ", text)                    # line comments
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per GEMM-1 launch from the committed counter summary, or None when
    the summary is for another workload or the grouped-GEMM source changed since
    (the hash covers ffn.hip followed by the common.h it includes)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"ffn_gemm1_gate_up_{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.split(":")[0] in ("source_sha256", "gemm1_traffic_bytes_per_launch"):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("source_sha256") != gemm_source_sha256():
        return None
    return float(fields["gemm1_traffic_bytes_per_launch"])


GEMM1 = "ffn_gemm1_gate_up"


def per_kernel(recs, nsteps):
    """Average duration per kernel name over the recorded launches.  The routed
    launches come first in each step; with a shared expert the second launch of a
    name in a step belongs to it."""
    per = {}
    for name, t in recs:
        per.setdefault(name, []).append(t)
    kernels = {}
    for name, ts in per.items():
        n_per_step = max(1, len(ts) // nsteps)
        for j in range(n_per_step):
            sub = ts[j::n_per_step]
            key = name if j == 0 else f"{name}.shared"
            kernels[key] = dict(avg_us=1e3 * float(np.mean(sub)), launches=len(sub))
    return kernels


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def to_dev(a, torch):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to("cuda").view(torch.bfloat16)
    return torch.from_numpy(a).to("cuda")


def cpu_baseline(I, tokens, min_seconds: float = 10.0, max_passes: int = 8):
    """Time the fp64 oracle (as it stands) on `tokens` of the workload, repeating the
    pass until about min_seconds of CPU work have been timed."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    c = I.cfg
    sh = (I.ws_gate, I.ws_up, I.ws_down) if c.Fs else (None, None, None)
    y, dt, passes = None, 0.0, 0
    while passes < max_passes and (passes == 0 or dt < min_seconds):
        t0 = time.perf_counter()
        _, _, yp, _ = oracle.token_outputs(tokens, I.x, I.logits, c.k, I.w_gate, I.w_up, I.w_down,
                                           c.renormalize, *sh)
        dt += time.perf_counter() - t0
        passes += 1
        if y is None:
            y = yp
    return dict(value=passes * len(tokens) / dt, unit="tokens/s", cores=int(threads), kind="oracle",
                sample=f"{len(tokens)} of {c.T} tokens through the whole layer "
                       f"(fp64 numpy, route + per-expert SwiGLU + combine), {passes} passes, "
                       f"{dt:.1f} s"), y


def copy_calibration(nbytes: int):
    """A plain copy of known size: HBM bytes counted by FETCH_SIZE / WRITE_SIZE for it
    give the scale factor applied to the same counters of the MoE kernels."""
    import torch
    src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    dst.copy_(src)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1)
    print(json.dumps({"copy_bytes": nbytes, "ms": ms, "GBps_read_plus_write": 2 * nbytes / ms / 1e6}))


def stream_copy_gbps(nbytes: int = 1 << 30, reps: int = 5) -> float:
    """Practical HBM rate on this GPU: read + write bytes of a plain device copy of
    nbytes (torch's copy kernel), median of reps, run outside any timed region."""
    import torch
    src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    rates = []
    for _ in range(reps):
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        dst.copy_(src)
        ev1.record()
        torch.cuda.synchronize()
        rates.append(2 * nbytes / ev0.elapsed_time(ev1) / 1e6)
    del src, dst
    return float(np.median(rates))


def route_probe(reps: int = 10):
    """Bandwidth of moe_route alone at T = 2^20 tokens (E = 64: 268 MB of fp32
    logits, more than the 256 MB Infinity Cache), cold (a 1 GiB scratch buffer is
    written before each rep, flushing L2 and the Infinity Cache) and warm (back to
    back).  One JSON line per (E, k)."""
    import torch

    import paper_2606_21712_amd as moe
    T = 1 << 20
    copy_gbs = stream_copy_gbps()
    scratch = torch.empty(1 << 29, dtype=torch.float16, device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    for E, k in ((64, 4), (64, 8), (8, 2)):
        logits = torch.randn((T, E), generator=gen, device="cuda", dtype=torch.float32)
        ids = torch.empty((T, k), dtype=torch.int32, device="cuda")
        w = torch.empty((T, k), dtype=torch.float32, device="cuda")
        for _ in range(3):
            moe.moe_route(logits, k, topk_ids=ids, topk_weights=w)
        torch.cuda.synchronize()
        res = {}
        for mode in ("cold", "warm"):
            ts = []
            for _ in range(reps):
                if mode == "cold":
                    scratch.fill_(1.0)
                ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                ev0.record()
                moe.moe_route(logits, k, topk_ids=ids, topk_weights=w)
                ev1.record()
                torch.cuda.synchronize()
                ts.append(ev0.elapsed_time(ev1) * 1e3)
            us = float(np.median(ts))
            gbs = (T * E * 4 + T * k * 8) / (us * 1e-6) / 1e9
            res[mode] = dict(us=round(us, 2), GBps=round(gbs, 1), frac_hbm=round(gbs / PEAK_HBM_GBS, 3),
                             frac_copy=round(gbs / copy_gbs, 3))
        print(json.dumps({"probe": "moe_route", "tokens": T, "experts": E, "top_k": k,
                          "bytes": T * E * 4 + T * k * 8, "stream_copy_GBps": round(copy_gbs, 1), **res}),
              flush=True)
        del logits, ids, w


PEAK_FP8_TFLOPS = 5000.0        # MI355X dense fp8 MFMA


def mxfp8_bench(config: str, steps: int, warmup: int):
    """The layer with MXFP8 expert GEMMs on one workload: one JSON line (a separate
    measurement; the bf16 line is the headline).  Weights are quantized once, outside
    the timed region; inside it every step routes, permutes, quantizes x, runs both
    MXFP8 GEMMs and combines."""
    import torch

    import moegen
    import paper_2606_21712_amd as moe
    c = moegen.CONFIGS[config]
    log(f"mxfp8: generating {c.name}")
    I = moegen.make_inputs(c)
    x, logits = to_dev(I.x, torch), to_dev(I.logits, torch)
    wq = [moe.quantize_weights_mxfp8(to_dev(w, torch)) for w in (I.w_gate, I.w_up, I.w_down)]
    wqs = [moe.quantize_weights_mxfp8(to_dev(w, torch)) for w in (I.ws_gate, I.ws_up, I.ws_down)] if c.Fs \
        else [None, None, None]
    layer = moe.MoELayerMXFP8(c.T, c.H, c.E, c.k, c.F, c.Fs)
    stream = torch.cuda.current_stream()

    def step():
        layer.run(x, logits, *wq, *wqs, renormalize=c.renormalize, stream=stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # timed region with only GEMM-1 bracketed, then a pass timing every kernel
    moe.profiler_start(steps * 2 + 8)
    moe.profiler_select(GEMM1)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    moe.profiler_stop()
    ms = ev0.elapsed_time(ev1) / steps
    timed_recs = moe.profiler_records()
    moe.profiler_select(None)
    moe.profiler_start(steps * 16 + 16)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    moe.profiler_stop()
    kernels = per_kernel(moe.profiler_records(), steps)
    kernels.update(per_kernel(timed_recs, steps))
    kernels = {k: v["avg_us"] for k, v in kernels.items()}
    g1 = kernels["ffn_gemm1_gate_up"]
    gemm1_flops = 4.0 * c.H * c.F * c.R
    ffn_us = sum(v for k, v in kernels.items() if k.startswith("ffn_"))
    ffn_tflops = c.flops() / (ffn_us * 1e-6) / 1e12
    out = {
        "metric": "MoE layer tokens/s with MXFP8 expert GEMMs + grouped-GEMM TFLOP/s (% fp8 MFMA peak)",
        "value": round(c.T / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": True,
        "dtype": "mxfp8 (e4m3 codes, e8m0 scale per 32; fp32 accumulation; bf16 x, y)",
        "data": "synthetic (seeded generator; random-init expert weights, quantized once)",
        "config": {"workload": c.name, "tokens": c.T, "hidden": c.H, "experts": c.E, "top_k": c.k,
                   "ffn_dim": c.F, "shared_ffn_dim": c.Fs},
        "ffn_tflops": round(ffn_tflops, 1), "ffn_frac_fp8_peak": round(ffn_tflops / PEAK_FP8_TFLOPS, 4),
        "roofline": {"kernel": "ffn_gemm1_gate_up (mxfp8)", "bound": "mfma",
                     "achieved": round(gemm1_flops / (g1 * 1e-6) / 1e12, 1), "peak": PEAK_FP8_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gemm1_flops / (g1 * 1e-6) / 1e12 / PEAK_FP8_TFLOPS, 4),
                     "flops_per_launch": gemm1_flops},
        "kernels_us": {k: round(v, 2) for k, v in kernels.items()},
    }
    print(json.dumps(out), flush=True)


def router_probe(reps: int = 10):
    """moe_router_topk (router GEMM fused with the gate) on the layer shapes: time,
    bytes read (token rows + router matrix) per second, cold (L2 and Infinity Cache
    flushed before each rep).  One JSON line per shape."""
    import torch

    import moegen
    import paper_2606_21712_amd as moe
    copy_gbs = stream_copy_gbps()
    scratch = torch.empty(1 << 29, dtype=torch.float16, device="cuda")
    for name in ("mixtral4k", "deepseek", "memconstrained"):
        c = moegen.CONFIGS[name]
        I = moegen.make_inputs(c, with_weights=False)
        x = to_dev(I.x, torch)
        w = to_dev(I.extra["w_router"], torch)
        ids = torch.empty((c.T, c.k), dtype=torch.int32, device="cuda")
        wt = torch.empty((c.T, c.k), dtype=torch.float32, device="cuda")
        for _ in range(3):
            moe.moe_router_topk(x, w, c.k, topk_ids=ids, topk_weights=wt)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            scratch.fill_(1.0)
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ev0.record()
            moe.moe_router_topk(x, w, c.k, topk_ids=ids, topk_weights=wt)
            ev1.record()
            torch.cuda.synchronize()
            ts.append(ev0.elapsed_time(ev1) * 1e3)
        us = float(np.median(ts))
        nbytes = c.T * c.H * 2 + c.E * c.H * 2 + c.T * c.k * 8
        gbs = nbytes / (us * 1e-6) / 1e9
        print(json.dumps({"probe": "moe_router_topk", "workload": name, "tokens": c.T, "hidden": c.H,
                          "experts": c.E, "top_k": c.k, "us": round(us, 2), "bytes": nbytes,
                          "GBps": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 3),
                          "frac_copy": round(gbs / copy_gbs, 3), "stream_copy_GBps": round(copy_gbs, 1),
                          "tflops": round(2.0 * c.T * c.H * c.E / (us * 1e-6) / 1e12, 2)}), flush=True)
        del x, w, ids, wt


SWEEP_SHAPES = {
    # layer shape -> (workload whose weights and routing recipe it uses, largest T)
    "mixtral": ("mixtral4k", 65536),
    "deepseek": ("deepseek", 32768),
    "memconstrained": ("memconstrained", 131072),
}


def expert_batch_sweep(shape: str, steps: int, warmup: int):
    """Module-level roofline of the MoE layer: time one layer over expert batches of
    T = 256 .. T_max tokens (the leading T tokens of one seeded batch, so every
    smaller batch is a prefix of the larger ones) and report tokens/s and grouped
    FFN TFLOP/s per size.  The saturation batch is the smallest T whose FFN
    throughput reaches 90% of the largest measured."""
    import torch

    import moegen
    import paper_2606_21712_amd as moe

    name, tmax = SWEEP_SHAPES[shape]
    base = moegen.CONFIGS[name]
    cfg = base.scaled(T=tmax, routing="router") if base.routing != "router" else base.scaled(T=tmax)
    log(f"sweep {shape}: generating T={cfg.T} H={cfg.H} E={cfg.E} k={cfg.k} F={cfg.F} Fs={cfg.Fs}")
    I = moegen.make_inputs(cfg)
    x, logits = to_dev(I.x, torch), to_dev(I.logits, torch)
    wg, wu, wd = to_dev(I.w_gate, torch), to_dev(I.w_up, torch), to_dev(I.w_down, torch)
    shared = (to_dev(I.ws_gate, torch), to_dev(I.ws_up, torch), to_dev(I.ws_down, torch)) if cfg.Fs \
        else (None, None, None)
    rows = []
    T = 256
    while T <= tmax:
        layer = moe.MoELayer(T, cfg.H, cfg.E, cfg.k, cfg.F, cfg.Fs)
        xs, ls = x[:T].contiguous(), logits[:T].contiguous()

        def step():
            layer.run(xs, ls, wg, wu, wd, *shared, renormalize=cfg.renormalize)

        for _ in range(warmup):
            step()
        # the layer timed without the profiler, then a pass timing every kernel
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record()
        for _ in range(steps):
            step()
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / steps
        moe.profiler_start(steps * 16 + 16)
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        moe.profiler_stop()
        ffn_ms = sum(t for n, t in moe.profiler_records() if n.startswith("ffn_")) / steps
        flops = 6.0 * cfg.H * cfg.F * T * cfg.k + 6.0 * cfg.H * cfg.Fs * T
        row = {"tokens": T, "ms_per_layer": round(ms, 4), "tokens_per_s": round(T / ms * 1e3, 1),
               "ffn_ms": round(ffn_ms, 4), "ffn_tflops": round(flops / ffn_ms / 1e9, 1),
               "tokens_per_expert": T * cfg.k / cfg.E}
        rows.append(row)
        print(json.dumps({"sweep": shape, **row}), flush=True)
        del layer
        T *= 2
    peak = max(r["ffn_tflops"] for r in rows)
    sat = next(r["tokens"] for r in rows if r["ffn_tflops"] >= 0.9 * peak)
    print(json.dumps({"sweep": shape, "summary": True, "peak_ffn_tflops": peak,
                      "saturation_tokens_90pct": sat,
                      "saturation_tokens_per_expert": sat * cfg.k / cfg.E}), flush=True)


def main():
    import moegen

    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="mixtral4k", choices=sorted(moegen.CONFIGS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gather", action="store_true",
                    help="materialize x_perm in moe_permute instead of gathering rows in the grouped FFN")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES (HBM counter calibration)")
    ap.add_argument("--sweep", choices=["mixtral", "deepseek", "memconstrained"], default=None,
                    help="expert-batch sweep of one layer shape: one JSON line per batch size")
    ap.add_argument("--mxfp8", action="store_true",
                    help="time the layer with MXFP8 expert GEMMs on --config (a separate JSON line)")
    ap.add_argument("--router-probe", action="store_true",
                    help="only time moe_router_topk (router GEMM + gate) on the layer shapes")
    ap.add_argument("--route-probe", action="store_true",
                    help="only time moe_route at 2^20 tokens (bandwidth probe), cold and warm")
    args = ap.parse_args()
    if args.copy_calibration:
        return copy_calibration(args.copy_calibration)
    if args.route_probe:
        return route_probe()
    if args.router_probe:
        return router_probe()
    if args.mxfp8:
        return mxfp8_bench(args.config, args.steps, args.warmup)
    if args.sweep:
        return expert_batch_sweep(args.sweep, args.steps, args.warmup)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the MoE-layer hot path is built and timed on a "
              "single MI355X (no collectives or sharding); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2606_21712_amd as moe

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    moe.lib()                                        # fail loudly if the library is missing

    cfg = moegen.CONFIGS[args.config]
    c = cfg
    t0 = time.perf_counter()
    log(f"generating inputs for {c.name}: T={c.T} H={c.H} E={c.E} k={c.k} F={c.F} Fs={c.Fs} {c.dtype}")
    I = moegen.make_inputs(cfg)
    log(f"inputs ready in {time.perf_counter() - t0:.1f} s; copying to the GPU")
    dt = torch.float32 if c.dtype == "f32" else torch.bfloat16
    x, logits = to_dev(I.x, torch), to_dev(I.logits, torch)
    wg, wu, wd = to_dev(I.w_gate, torch), to_dev(I.w_up, torch), to_dev(I.w_down, torch)
    shared = (to_dev(I.ws_gate, torch), to_dev(I.ws_up, torch), to_dev(I.ws_down, torch)) if c.Fs \
        else (None, None, None)
    layer = moe.MoELayer(c.T, c.H, c.E, c.k, c.F, c.Fs, dtype=dt, gather=not args.no_gather)
    stream = torch.cuda.current_stream()

    def step():
        layer.run(x, logits, wg, wu, wd, *shared, renormalize=c.renormalize, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps); timing {args.steps} steps")

    # Timed region: only GEMM-1 (the roofline kernel) is bracketed by HIP events, so
    # the other launches run exactly as in production.
    moe.profiler_start(args.steps * 2 + 8)
    moe.profiler_select(GEMM1)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    moe.profiler_stop()
    ms = ev0.elapsed_time(ev1) / args.steps
    timed_recs = moe.profiler_records()
    log(f"timed: {ms:.3f} ms/step")
    # Per-kernel times of the other kernels: a second pass with every launch bracketed.
    moe.profiler_select(None)
    moe.profiler_start(args.steps * 16 + 16)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    moe.profiler_stop()
    kernels = per_kernel(moe.profiler_records(), args.steps)
    kernels.update(per_kernel(timed_recs, args.steps))          # GEMM-1 from the timed region

    R = c.R
    gemm1_flops = 4.0 * c.H * c.F * R
    g1 = kernels.get("ffn_gemm1_gate_up", {}).get("avg_us")
    ffn_us = sum(kernels[k]["avg_us"] for k in kernels if k.startswith("ffn_"))
    peak = PEAK_F32_TFLOPS if c.dtype == "f32" else PEAK_BF16_TFLOPS
    achieved = gemm1_flops / (g1 * 1e-6) / 1e12 if g1 else None
    ffn_tflops = c.flops() / (ffn_us * 1e-6) / 1e12 if ffn_us else None

    b = 4 if c.dtype == "f32" else 2
    bytes_alg = {
        "route": c.T * c.E * 4 + c.T * c.k * 8,
        # ids read + dest_rows and sorted_token_ids written (+ x read and x_perm written
        # when the rows are materialized rather than gathered by the grouped FFN)
        "permute": 3 * R * 4 + (0 if not args.no_gather else c.T * c.H * b + R * c.H * b),
        "combine": R * c.H * b + c.T * c.H * b * (2 if c.Fs else 1) + c.T * c.k * 8,
    }
    perm_us = sum(kernels[k]["avg_us"] for k in kernels if k.startswith("permute_"))
    copy_gbs = stream_copy_gbps()
    bw = {"stream_copy_GBps": round(copy_gbs, 1)}
    for name, us in (("route", kernels.get("route", {}).get("avg_us")), ("permute", perm_us),
                     ("combine", kernels.get("combine", {}).get("avg_us"))):
        if us:
            gbs = bytes_alg[name] / (us * 1e-6) / 1e9
            bw[name] = dict(us=round(us, 2), GBps=round(gbs, 1), frac_hbm=round(gbs / PEAK_HBM_GBS, 3),
                            frac_copy=round(gbs / copy_gbs, 3))

    out = {
        "metric": METRIC,
        "value": round(c.T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if c.dtype == "f32" else "bf16",
        "data": "synthetic (seeded generator; random-init expert weights)",
        "config": {"workload": c.name, "tokens": c.T, "hidden": c.H, "experts": c.E, "top_k": c.k,
                   "ffn_dim": c.F, "shared_ffn_dim": c.Fs, "routing": c.routing, "seed": c.seed,
                   "path": "permute maps + gather-fused grouped FFN" if not args.no_gather
                   else "permute with x_perm + grouped FFN"},
        "ffn_tflops": round(ffn_tflops, 1) if ffn_tflops else None,
        "ffn_frac_peak": round(ffn_tflops / peak, 4) if ffn_tflops else None,
        "roofline": {
            "kernel": "ffn_gemm1_gate_up",
            "bound": "mfma",
            "achieved": round(achieved, 1) if achieved else None,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4) if achieved else None,
            "traffic": measured_traffic(c.name),
            "flops_per_launch": gemm1_flops,
        },
        "kernels_us": {k: round(v["avg_us"], 2) for k, v in kernels.items()},
        "bandwidth": bw,
    }

    if not args.no_cpu_baseline:
        n = min(CPU_SAMPLE.get(c.name, 128), c.T)
        tokens = np.random.default_rng(1234).choice(c.T, size=n, replace=False)
        log(f"CPU baseline: oracle on {n} tokens")
        base, y_or = cpu_baseline(I, tokens)
        out["cpu_baseline"] = base
        yg = layer.y.float().cpu().numpy()[tokens].astype(np.float64)
        out["sample_check"] = {"tokens": int(n),
                               "max_rel_err": float(np.abs(yg - y_or).max() / np.abs(y_or).max())}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
