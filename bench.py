#!/usr/bin/env python3
"""Throughput of the MoE-layer hot path on one MI355X.

One step = the whole layer (route -> permute -> grouped SwiGLU FFN [-> shared
expert] -> combine) over one synthetic expert batch whose inputs are already
resident in HBM.  The default workload is the large memory-constrained expert
batch: 131072 tokens, hidden 4096, 64 experts, top-4, FFN dim 4096, bf16, with
lognormal expert loads whose three smallest experts hold 1, 17 and 31 rows.
Prints ONE JSON line on stdout; progress goes to stderr.

Per-kernel durations come from the library's own HIP-event profiler, recorded
on the launch stream inside the timed region.  The roofline figure is for the
dominant kernel, GEMM-1 (gate/up projections + SwiGLU): algorithmic flops
4*H*F*R per launch over its average launch duration, against the 2.5 PFLOP/s
dense bf16 MFMA peak.  Route, permute and combine are then timed call by call,
cold (a 1 GiB buffer read and written before each call, flushing L2 and the
256 MB Infinity Cache) and warm, as median / min / max over repetitions.  The
CPU baseline times the fp64 oracle on a bounded sample of tokens of the same
workload on the host cores.

Other modes: --profile-run (a short run for rocprofv3 counter passes),
--summarize DIR (tables from rocprofv3 output: kernel times, MFMA busy, clock,
HBM bytes against the algorithmic bytes), --sweep (expert-batch sweep with a
fitted runtime model), --mxfp8, --route-probe, --router-probe.
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


def gemm_source_sha256(mx: bool = False) -> str:
    """sha256 of the grouped-GEMM source (ffn.hip, or ffn_fp8.hip for the MXFP8
    GEMMs, then the common.h it includes) with comments removed and whitespace
    collapsed, so that only code changes invalidate counters taken on it."""
    import hashlib
    import re
    csrc = os.path.join(ROOT, "paper_2606_21712_amd", "csrc")
    h = hashlib.sha256()
    for name in ("ffn_fp8.hip" if mx else "ffn.hip", "common.h"):
        with open(os.path.join(csrc, name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)      # block comments
        text = re.sub(r"//[^\n]*", " ", text)                    # line comments
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def measured_traffic(workload: str):
    """L2-egress bytes (FETCH_SIZE + WRITE_SIZE, calibrated) per GEMM-1 launch from the
    committed rocprofv3 summary of the workload, or None when there is none or the
    grouped-GEMM source changed since the counters were taken (the hash covers
    ffn.hip followed by the common.h it includes)."""
    for name in (f"moe_layer_{workload}_rocprof.md", f"ffn_gemm1_gate_up_{workload}_hbm_traffic.md"):
        path = os.path.join(ROOT, "profiles", name)
        if not os.path.exists(path):
            continue
        fields = {}
        for line in open(path):
            if ":" in line and line.split(":")[0] in ("source_sha256", "gemm1_traffic_bytes_per_launch"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        if "gemm1_traffic_bytes_per_launch" not in fields:
            continue
        if fields.get("source_sha256") != gemm_source_sha256():
            return None
        return float(fields["gemm1_traffic_bytes_per_launch"])
    return None


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
                       f"{dt:.1f} s", blas=_blas_name(), cpu=_cpu_model()), y


def _blas_name() -> str:
    """numpy's BLAS library and version, for the CPU baseline's record."""
    try:
        blas = np.show_config(mode="dicts").get("Build Dependencies", {}).get("blas", {})
        return f"{blas.get('name', '?')} {blas.get('version', '')}".strip()
    except Exception:                                  # older numpy: no dict mode
        return "unknown"


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


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


def dense_ceiling(cname: str, reps: int = 5):
    """The vendor GEMM on the same work, for context: torch.matmul (hipBLASLt) run
    expert by expert over the workload's own group sizes (the routing and grouping
    of this library's route and permute on the workload's logits), bf16 in, fp32
    accumulation, bf16 out, with contiguous pre-transposed weights and the rows of
    each group contiguous (x_perm), so the library gets its easiest layout.  Both
    projections are timed (the gate and up weights as one [H, 2F] matrix per expert;
    the down projection on a random h), without the SwiGLU between them; then one
    dense GEMM of each projection's total size (M = R) as an upper bound.  Weights and
    h are random normal with the workload's scale (the values only matter for the
    board's power draw).  Median over reps of the whole loop, HIP events."""
    import torch

    import moegen
    import paper_2606_21712_amd as moe

    c = moegen.CONFIGS[cname]
    assert c.dtype == "bf16", "bf16 workloads only"
    T, H, E, k, F, R = c.T, c.H, c.E, c.k, c.F, c.R
    log(f"dense ceiling {cname}: generating T={T} H={H} E={E} k={k} F={F}")
    I = moegen.make_inputs(c, with_weights=False)
    x, logits = to_dev(I.x, torch), to_dev(I.logits, torch)
    ids = torch.empty((T, k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, k), dtype=torch.float32, device="cuda")
    moe.moe_route(logits, k, c.renormalize, ids, w)
    perm = moe.moe_permute(ids, x, E)
    torch.cuda.synchronize()
    offs = perm["offsets"].cpu().tolist()
    x_perm = perm["x_perm"]
    g = torch.Generator(device="cuda").manual_seed(c.seed)
    w_gu = (torch.randn((E, H, 2 * F), generator=g, device="cuda") / H ** 0.5).to(torch.bfloat16)
    w_d = (torch.randn((E, F, H), generator=g, device="cuda") / F ** 0.5).to(torch.bfloat16)
    h = torch.randn((R, F), generator=g, device="cuda").to(torch.bfloat16)
    gu = torch.empty((R, 2 * F), dtype=torch.bfloat16, device="cuda")
    y = torch.empty((R, H), dtype=torch.bfloat16, device="cuda")
    groups = [(e, offs[e], offs[e + 1]) for e in range(E) if offs[e + 1] > offs[e]]

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    def gate_up():
        for e, a, b in groups:
            torch.matmul(x_perm[a:b], w_gu[e], out=gu[a:b])

    def down():
        for e, a, b in groups:
            torch.matmul(h[a:b], w_d[e], out=y[a:b])

    t1, t2 = timed(gate_up), timed(down)
    t1d = timed(lambda: torch.matmul(x_perm, w_gu[0], out=gu))
    t2d = timed(lambda: torch.matmul(h, w_d[0], out=y))
    del w_gu, w_d, h, gu
    # this library's grouped FFN (gather path) on the same routing, in the same process
    wg = (torch.randn((E, F, H), generator=g, device="cuda") / H ** 0.5).to(torch.bfloat16)
    wu = (torch.randn((E, F, H), generator=g, device="cuda") / H ** 0.5).to(torch.bfloat16)
    wd = (torch.randn((E, H, F), generator=g, device="cuda") / F ** 0.5).to(torch.bfloat16)
    ws = torch.empty(moe.moe_grouped_ffn_workspace_bytes(R, E, H, F, torch.bfloat16), dtype=torch.uint8,
                     device="cuda")

    def ours():
        moe.moe_grouped_ffn_gather(x, perm["sorted_token_ids"], perm["offsets"], wg, wu, wd, y_perm=y, ws=ws)

    ours()
    torch.cuda.synchronize()
    moe.profiler_start(reps * 8 + 8)
    for _ in range(reps):
        ours()
    torch.cuda.synchronize()
    moe.profiler_stop()
    rec = {}
    for n, ms in moe.profiler_records():
        rec.setdefault(n, []).append(ms)
    o1 = float(np.median(rec["ffn_gemm1_gate_up"]))
    o2 = float(np.median(rec["ffn_gemm2_down"])) + float(np.median(rec.get("ffn_tail_reduce", [0.0])))
    f1, f2 = 4.0 * H * F * R, 2.0 * H * F * R
    print(json.dumps({"dense_ceiling": cname, "library": "torch.matmul (hipBLASLt), bf16",
                      "experts_run": len(groups), "reps": reps,
                      "this_library": {"gate_up_swiglu_gather_ms": round(o1, 3),
                                       "gate_up_tflops": round(f1 / o1 / 1e9, 1),
                                       "down_ms": round(o2, 3), "down_tflops": round(f2 / o2 / 1e9, 1),
                                       "ffn_tflops": round((f1 + f2) / (o1 + o2) / 1e9, 1)},
                      "per_expert": {"gate_up_ms": round(t1, 3), "gate_up_tflops": round(f1 / t1 / 1e9, 1),
                                     "down_ms": round(t2, 3), "down_tflops": round(f2 / t2 / 1e9, 1),
                                     "ffn_tflops": round((f1 + f2) / (t1 + t2) / 1e9, 1)},
                      "one_dense_gemm": {"gate_up_ms": round(t1d, 3), "gate_up_tflops": round(f1 / t1d / 1e9, 1),
                                         "down_ms": round(t2d, 3), "down_tflops": round(f2 / t2d / 1e9, 1)}}),
          flush=True)


def dense_ceiling_fp8(cname: str, reps: int = 5):
    """The MXFP8 counterpart of dense_ceiling: this library's MXFP8 grouped FFN
    (gather path; the token rows quantized once, not timed here) beside the vendor
    fp8 GEMM, torch._scaled_mm (hipBLASLt) with OCP E4M3 operands and one fp32 scale
    per tensor (a coarser scaling than MX blocks, so a generous ceiling), expert by
    expert over the same groups and as one dense GEMM of each projection's total
    size.  Operands are random normal at the workload's scale."""
    import torch

    import moegen
    import paper_2606_21712_amd as moe

    c = moegen.CONFIGS[cname]
    T, H, E, k, F, R = c.T, c.H, c.E, c.k, c.F, c.R
    log(f"fp8 dense ceiling {cname}: generating T={T} H={H} E={E} k={k} F={F}")
    I = moegen.make_inputs(c, with_weights=False)
    x, logits = to_dev(I.x, torch), to_dev(I.logits, torch)
    ids = torch.empty((T, k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, k), dtype=torch.float32, device="cuda")
    moe.moe_route(logits, k, c.renormalize, ids, w)
    perm = moe.moe_permute(ids, x, E)
    torch.cuda.synchronize()
    offs = perm["offsets"].cpu().tolist()
    groups = [(e, offs[e], offs[e + 1]) for e in range(E) if offs[e + 1] > offs[e]]
    g = torch.Generator(device="cuda").manual_seed(c.seed)

    def rnd(shape, std):
        return (torch.randn(shape, generator=g, device="cuda") * std).to(torch.bfloat16)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    f1, f2 = 4.0 * H * F * R, 2.0 * H * F * R
    out = {"dense_ceiling_fp8": cname, "experts_run": len(groups), "reps": reps}
    # this library
    wq_g = moe.quantize_weights_mxfp8(rnd((E, F, H), H ** -0.5))
    wq_u = moe.quantize_weights_mxfp8(rnd((E, F, H), H ** -0.5))
    wq_d = moe.quantize_weights_mxfp8(rnd((E, H, F), F ** -0.5))
    xq = moe.moe_quantize_mxfp8(x)
    y = torch.empty((R, H), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(moe.moe_grouped_ffn_mxfp8_workspace_bytes(R, E, H, F), dtype=torch.uint8, device="cuda")

    def ours():
        moe.moe_grouped_ffn_mxfp8_gather(xq, perm["sorted_token_ids"], perm["offsets"], wq_g, wq_u, wq_d,
                                         y_perm=y, ws=ws)

    ours()
    torch.cuda.synchronize()
    moe.profiler_start(reps * 8 + 8)
    for _ in range(reps):
        ours()
    torch.cuda.synchronize()
    moe.profiler_stop()
    rec = {}
    for n, ms in moe.profiler_records():
        rec.setdefault(n, []).append(ms)
    o1 = float(np.median(rec["ffn_gemm1_gate_up"]))
    o2 = float(np.median(rec["ffn_gemm2_down"])) + float(np.median(rec.get("ffn_tail_reduce", [0.0])))
    out["this_library_mxfp8"] = {"gate_up_swiglu_gather_ms": round(o1, 3), "gate_up_tflops": round(f1 / o1 / 1e9, 1),
                                 "down_ms": round(o2, 3), "down_tflops": round(f2 / o2 / 1e9, 1),
                                 "ffn_tflops": round((f1 + f2) / (o1 + o2) / 1e9, 1)}
    del wq_g, wq_u, wq_d, xq, ws
    # the vendor GEMM: A row-major [M, K], B column-major [K, N] (the weights' own K-contiguous rows)
    f8 = torch.float8_e4m3fn
    one = torch.ones((), dtype=torch.float32, device="cuda")
    a1 = perm["x_perm"].to(f8)
    w1 = rnd((E, 2 * F, H), H ** -0.5).to(f8)
    a2 = rnd((R, F), 1.0).to(f8)
    w2 = rnd((E, H, F), F ** -0.5).to(f8)
    gu = torch.empty((R, 2 * F), dtype=torch.bfloat16, device="cuda")
    try:
        def gate_up():
            for e, a, b in groups:
                gu[a:b] = torch._scaled_mm(a1[a:b], w1[e].t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16)

        def down():
            for e, a, b in groups:
                y[a:b] = torch._scaled_mm(a2[a:b], w2[e].t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16)

        t1, t2 = timed(gate_up), timed(down)
        t1d = timed(lambda: torch._scaled_mm(a1, w1[0].t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16))
        t2d = timed(lambda: torch._scaled_mm(a2, w2[0].t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16))
        out["library"] = "torch._scaled_mm (hipBLASLt), E4M3, per-tensor scales"
        out["per_expert"] = {"gate_up_ms": round(t1, 3), "gate_up_tflops": round(f1 / t1 / 1e9, 1),
                             "down_ms": round(t2, 3), "down_tflops": round(f2 / t2 / 1e9, 1),
                             "ffn_tflops": round((f1 + f2) / (t1 + t2) / 1e9, 1)}
        out["one_dense_gemm"] = {"gate_up_ms": round(t1d, 3), "gate_up_tflops": round(f1 / t1d / 1e9, 1),
                                 "down_ms": round(t2d, 3), "down_tflops": round(f2 / t2d / 1e9, 1)}
    except (RuntimeError, TypeError) as err:
        out["library_error"] = str(err)[:300]
    print(json.dumps(out), flush=True)


def mfma_ceiling(reps: int = 3):
    """What the matrix cores sustain on this board with no memory traffic: the
    register-only probe of libmoe_probe.so (a measurement tool built beside the
    library, not part of the MoE path) for bf16 and MX-scaled E4M3 MFMAs, with
    constant operands and with operands redrawn as they run.  Under the board's
    power limit the second is the ceiling a GEMM on real data can approach.
    Median over reps of one launch, HIP events; 2048 workgroups of 4 wavefronts."""
    import ctypes

    import torch
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2606_21712_amd", "libmoe_probe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    fn = lib.moe_probe_mfma_rate
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    blocks, waves = 2048, 4
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    rows = []
    for fp8 in (0, 1):
        iters = 8000 if fp8 else 16000                        # multiples of 4
        flop_per_mfma = 131072 if fp8 else 32768
        peak = PEAK_FP8_TFLOPS if fp8 else PEAK_BF16_TFLOPS
        for rnd in (0, 1):
            def call():
                rc = fn(fp8, rnd, blocks, iters, out.data_ptr(), stream.cuda_stream)
                if rc != 0:
                    raise RuntimeError(f"moe_probe_mfma_rate returned {rc}")
            call()
            torch.cuda.synchronize()
            assert bool(torch.isfinite(out).all()), "probe accumulators not finite"
            ts = []
            for _ in range(reps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                call()
                e1.record(stream)
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            ms = float(np.median(ts))
            tflops = blocks * waves * iters * 8 * flop_per_mfma / (ms * 1e-3) / 1e12
            rows.append({"mfma": "v_mfma_scale_f32_32x32x64_f8f6f4 (E4M3)" if fp8 else "v_mfma_f32_32x32x16_bf16",
                         "operands": "redrawn" if rnd else "constant", "ms": round(ms, 3),
                         "tflops": round(tflops, 1), "frac_of_peak": round(tflops / peak, 4)})
            log(f"mfma ceiling: {rows[-1]}")
    print(json.dumps({"mfma_ceiling": rows, "workgroups": blocks, "wavefronts_per_workgroup": waves}), flush=True)


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


def mxfp8_bench(config: str, steps: int, warmup: int, profile_run: bool = False):
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

    if profile_run:
        # what the counter passes see: one warmup step, then two steps
        for i in range(3):
            log(f"mxfp8 profile run: layer step {i + 1} of 3")
            step()
            torch.cuda.synchronize()
        print(json.dumps({"profile_run": c.name, "mxfp8": True, "steps": 3}), flush=True)
        return

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
    "memconstrained_lognormal": ("memconstrained", 131072),
}


def fit_ffn_model(rows, weight_bytes: float):
    """Fit t_ffn(T) = t0 + max(weight_bytes / BW, flops(T) / P) to the measured
    grouped-FFN times (least squares on the relative residuals): a fixed cost, the
    expert weights streamed once at bandwidth BW, and the flops at rate P, the
    larger of the two bounding each batch (the roofline of one grouped FFN).
    Returns the parameters, the batch where the two bounds meet and each size's
    residual."""
    from scipy.optimize import least_squares
    t = np.array([r["ffn_ms"] * 1e-3 for r in rows])
    fl = np.array([r["flops"] for r in rows])

    def model(q):
        t0, bw, pf = np.exp(q)
        return t0 + np.maximum(weight_bytes / bw, fl / pf)

    q0 = np.log([1e-5, 5e12, 1.2e15])
    res = least_squares(lambda q: model(q) / t - 1.0, q0)
    t0, bw, pf = np.exp(res.x)
    pred = model(res.x)
    ridge_flops = weight_bytes / bw * pf
    return dict(t0_us=round(t0 * 1e6, 2), weight_GBps=round(bw / 1e9, 1), tflops=round(pf / 1e12, 1),
                ridge_flops=ridge_flops,
                residual_pct=[round(100 * (p / m - 1.0), 2) for p, m in zip(pred, t)],
                max_abs_residual_pct=round(100 * float(np.max(np.abs(pred / t - 1.0))), 2))


def stream_probe(reps: int = 7):
    """How fast 256-row panels stream from HBM one 128-byte k column at a time (the
    way a grouped-GEMM tile reads its weight panel), against the row pitch K, with
    every panel starting at column 0 and with panel p starting at column 7 p mod
    (K / 128): the panel-streaming probe of libmoe_probe.so over 1 GiB of panels,
    256 persistent workgroups, median of reps launches (HIP events).  One JSON line
    per (K, order)."""
    import ctypes

    import torch
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2606_21712_amd", "libmoe_probe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built (run __graft_entry__.build())")
    fn = ctypes.CDLL(path).moe_probe_stream_panels
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_void_p]
    total = 1 << 30
    w = torch.ones(total, dtype=torch.uint8, device="cuda")
    ctr = torch.zeros(1, dtype=torch.int32, device="cuda")
    blocks = 256
    out = torch.empty(blocks * 512, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    for K in (4096, 6144, 7168, 8192, 12288, 14336, 16384, 28672):
        panels = total // (256 * K)
        row = {"stream_probe": "panels", "row_bytes": K, "panels": panels}
        for rot in (0, 1):
            ts = []
            for _ in range(reps):
                ctr.zero_()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                rc = fn(w.data_ptr(), panels, K, rot, blocks, ctr.data_ptr(), out.data_ptr(), stream.cuda_stream)
                e1.record(stream)
                torch.cuda.synchronize()
                if rc != 0:
                    raise RuntimeError(f"moe_probe_stream_panels returned {rc}")
                ts.append(e0.elapsed_time(e1))
            assert int(ctr.item()) == panels + blocks, "panel counter"
            ms = float(np.median(ts))
            row["rotated_TBps" if rot else "column0_TBps"] = round(panels * 256 * K / (ms * 1e-3) / 1e12, 2)
        print(json.dumps(row), flush=True)
    # the other direction: 16-byte nontemporal stores alone over the same 1 GiB
    wfn = ctypes.CDLL(path).moe_probe_write
    wfn.restype = ctypes.c_int
    wfn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p]
    for wblocks in (2048, 8192):
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            rc = wfn(w.data_ptr(), total, wblocks, stream.cuda_stream)
            e1.record(stream)
            torch.cuda.synchronize()
            if rc != 0:
                raise RuntimeError(f"moe_probe_write returned {rc}")
            ts.append(e0.elapsed_time(e1))
        ms = float(np.median(ts))
        print(json.dumps({"stream_probe": "write", "bytes": total, "blocks": wblocks,
                          "TBps": round(total / (ms * 1e-3) / 1e12, 2)}), flush=True)


def graph_probe(steps: int, warmup: int):
    """Small expert batches, where launches rather than the kernels set the pace: one
    layer step issued call by call (eager: the Python binding's calls, each a kernel
    launch or two) against the same step captured once as a HIP graph (LayerGraph)
    and replayed, T = 256 .. 4096 tokens on the Mixtral and DeepSeek shapes (router
    logits, gather path).  Per size: ms per step back to back over `steps` steps,
    both ways, and the sum of the kernels' own times (the library's profiler, eager
    steps).  One JSON line per size."""
    import torch

    import moegen
    import paper_2606_21712_amd as moe

    for name in ("mixtral4k", "deepseek"):
        base = moegen.CONFIGS[name]
        cfg = base.scaled(T=4096)
        log(f"graph probe {name}: generating T={cfg.T} H={cfg.H} E={cfg.E} k={cfg.k} F={cfg.F} Fs={cfg.Fs}")
        I = moegen.make_inputs(cfg)
        x_all, l_all = to_dev(I.x, torch), to_dev(I.logits, torch)
        W = [to_dev(a, torch) for a in (I.w_gate, I.w_up, I.w_down)]
        W += [to_dev(a, torch) for a in (I.ws_gate, I.ws_up, I.ws_down)] if cfg.Fs else [None, None, None]
        T = 256
        while T <= cfg.T:
            layer = moe.MoELayer(T, cfg.H, cfg.E, cfg.k, cfg.F, cfg.Fs, gather=True)
            x, lg = x_all[:T].contiguous(), l_all[:T].contiguous()

            def eager():
                layer.run(x, lg, *W, renormalize=cfg.renormalize)

            g = moe.LayerGraph(layer, x, lg, *W, renormalize=cfg.renormalize)
            out = {}
            for mode, fn in (("eager", eager), ("graph", g.replay)):
                for _ in range(warmup):
                    fn()
                torch.cuda.synchronize()
                ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                ev0.record()
                for _ in range(steps):
                    fn()
                ev1.record()
                torch.cuda.synchronize()
                out[mode] = ev0.elapsed_time(ev1) / steps
            moe.profiler_start(steps * 16 + 16)
            for _ in range(steps):
                eager()
            torch.cuda.synchronize()
            moe.profiler_stop()
            kern = sum(t for _, t in moe.profiler_records()) / steps
            print(json.dumps({"graph_probe": name, "tokens": T, "eager_ms": round(out["eager"], 4),
                              "graph_ms": round(out["graph"], 4), "kernels_ms": round(kern, 4),
                              "speedup": round(out["eager"] / out["graph"], 3),
                              "graph_tokens_per_s": round(T / out["graph"] * 1e3, 1)}), flush=True)
            del g, layer
            T *= 2


def expert_batch_sweep(shape: str, steps: int, warmup: int):
    """Module-level roofline of the MoE layer: time one layer over expert batches of
    T = 256 .. T_max tokens and report tokens/s and grouped-FFN TFLOP/s per size,
    then fit the grouped FFN's runtime model (fit_ffn_model).  Router-logit shapes
    use the leading T tokens of one seeded batch (every smaller batch is a prefix of
    the larger ones).  memconstrained_lognormal keeps the workload's own routing at
    every T: exact per-expert counts from 64 lognormal(0, 1) draws, scaled to T * k
    assignments, the three smallest experts pinned to 1, 17 and 31 rows (an expert
    above T rows, possible only at the smallest T, is capped at T and its excess
    moved to the next largest).
    The saturation batch is the smallest T whose FFN throughput reaches 90% of the
    largest measured."""
    import torch

    import moegen
    import paper_2606_21712_amd as moe

    name, tmax = SWEEP_SHAPES[shape]
    base = moegen.CONFIGS[name]
    lognormal = shape == "memconstrained_lognormal"
    cfg = base.scaled(T=tmax) if lognormal or base.routing == "router" else base.scaled(T=tmax, routing="router")
    log(f"sweep {shape}: generating T={cfg.T} H={cfg.H} E={cfg.E} k={cfg.k} F={cfg.F} Fs={cfg.Fs}")
    I = moegen.make_inputs(cfg)
    x = to_dev(I.x, torch)
    logits_all = to_dev(I.logits, torch)
    wg, wu, wd = to_dev(I.w_gate, torch), to_dev(I.w_up, torch), to_dev(I.w_down, torch)
    shared = (to_dev(I.ws_gate, torch), to_dev(I.ws_up, torch), to_dev(I.ws_down, torch)) if cfg.Fs \
        else (None, None, None)
    w_r = moegen.router_matrix(cfg) if lognormal else None
    rows = []
    T = 256
    while T <= tmax:
        layer = moe.MoELayer(T, cfg.H, cfg.E, cfg.k, cfg.F, cfg.Fs, gather=True)
        xs = x[:T].contiguous()
        if lognormal:
            # the workload's routing recipe at this T (generator only: counts, sets, margin logits)
            rng = np.random.default_rng(np.random.SeedSequence([cfg.seed, T]))
            target = moegen.cap_counts(
                moegen.lognormal_counts(rng, cfg.E, T * cfg.k, cfg.lognormal_sigma, cfg.pinned_small), T)
            chosen, _ = moegen.exact_count_assignment(target, T, cfg.k, rng)
            ls = to_dev(moegen.margin_logits(I.x[:T], w_r, chosen, cfg.margin), torch)
            counts = np.sort(np.bincount(chosen.ravel(), minlength=cfg.E))
        else:
            ls = logits_all[:T].contiguous()
            counts = None

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
               "tokens_per_expert": T * cfg.k / cfg.E, "flops": flops}
        if counts is not None:
            row["smallest_groups"] = counts[:3].tolist()
            row["largest_group"] = int(counts[-1])
        rows.append(row)
        print(json.dumps({"sweep": shape, **row}), flush=True)
        del layer
        T *= 2
    peak = max(r["ffn_tflops"] for r in rows)
    sat = next(r["tokens"] for r in rows if r["ffn_tflops"] >= 0.9 * peak)
    weight_bytes = 3.0 * cfg.E * cfg.H * cfg.F * 2 + 3.0 * cfg.H * cfg.Fs * 2
    fit = fit_ffn_model(rows, weight_bytes)
    ridge_T = fit.pop("ridge_flops") / (6.0 * cfg.H * (cfg.F * cfg.k + cfg.Fs))
    print(json.dumps({"sweep": shape, "summary": True, "peak_ffn_tflops": peak,
                      "saturation_tokens_90pct": sat,
                      "saturation_tokens_per_expert": sat * cfg.k / cfg.E,
                      "model": "t_ffn(T) = t0 + max(weight_bytes / BW, flops(T) / P)",
                      "weight_bytes": weight_bytes, **fit,
                      "ridge_tokens": round(ridge_T, 1),
                      "ridge_tokens_per_expert": round(ridge_T * cfg.k / cfg.E, 1)}), flush=True)


# --------------------------------------------------------------------------- algorithmic work per kernel
def algorithmic_work(c, role: str, gather: bool = True, mx: bool = False):
    """(flops, bytes) one launch of a kernel of the layer must do at the least on
    workload c: every operand read once, every result written once, no padding.
    role is a kernel label from kernel_label() (".shared" for the shared expert).
    mx: the MXFP8 layer (GEMM operands as one-byte codes plus a one-byte scale per
    32 along k; x, y and y_perm stay bf16)."""
    b = 4 if c.dtype == "f32" else 2
    T, H, E, k, F, Fs, R = c.T, c.H, c.E, c.k, c.F, c.Fs, c.R
    if mx:
        q = 1 + 1 / 32                                   # bytes per element: code + its share of a scale
        base = role.split(".")[0]
        shared = role.endswith(".shared")
        if base == "quantize_rows":
            return 0.0, T * H * 2 + T * H * q
        if base == "gemm1":
            if shared:
                return 4.0 * H * Fs * T, 2 * Fs * H * q + T * H * q + T * Fs * q
            return 4.0 * H * F * R, 2 * E * F * H * q + T * H * q + R * 4 + R * F * q
        if base == "gemm2":
            if shared:
                return 2.0 * H * Fs * T, Fs * H * q + T * Fs * q + T * H * 2
            return 2.0 * H * F * R, E * H * F * q + R * F * q + R * H * 2
    units = (R + 1023) // 1024
    shared = role.endswith(".shared")
    base = role.split(".")[0]
    if base == "route":
        return 0.0, T * E * 4 + T * k * 8
    if base == "permute_count":
        return 0.0, R * 4 + units * E * 4
    if base == "permute_scan":
        return 0.0, 2 * units * E * 4 + E * 4
    if base == "permute_rank":
        return 0.0, R * 4 + units * E * 4 + E * 4 + (E + 1) * 4 + 2 * R * 4
    if base in ("permute_small", "permute_maps"):
        return 0.0, R * 4 + E * 4 + (E + 1) * 4 + 2 * R * 4
    if base == "permute_copy":
        return 0.0, T * H * b + R * H * b + R * 4
    if base == "combine":
        return 0.0, R * H * b + T * H * b * (2 if Fs else 1) + T * k * 8
    if base == "gemm1":
        if shared:
            return 4.0 * H * Fs * T, 2 * Fs * H * b + T * H * b + T * Fs * b
        rows_in = T * H * b + R * 4 if gather else R * H * b
        return 4.0 * H * F * R, 2 * E * F * H * b + rows_in + R * F * b
    if base == "gemm2":
        if shared:
            return 2.0 * H * Fs * T, Fs * H * b + T * Fs * b + T * H * b
        return 2.0 * H * F * R, E * H * F * b + R * F * b + R * H * b
    return 0.0, 0


def kernel_label(name: str) -> str:
    """Short label of a kernel from its demangled name (rocprofv3 traces)."""
    import re
    m = re.search(r"(\w+)_kernel(<[^()]*>)?\(", name)
    if not m:
        return name.split("(")[0].strip()
    base, tmpl = m.group(1), m.group(2) or ""
    if base == "grouped_gemm_bf16" or base == "grouped_gemm_f32" or base == "grouped_gemm_fp8":
        return "gemm1" if tmpl.startswith("<true") else "gemm2"
    return base


# --------------------------------------------------------------------------- cold / warm timing
def time_calls(calls, stream, reps: int = 20):
    """Median / min / max duration of each call, cold and warm.  calls = [(name, fn,
    algorithmic bytes)].  Cold: a 1 GiB buffer is read and written (on the same
    stream) right before each timed call, which evicts the call's operands from the
    L2s and the 256 MB Infinity Cache; warm: the call runs again right after
    itself.  HIP events on the launch stream bracket each call."""
    import torch
    scratch = torch.zeros(1 << 28, dtype=torch.float32, device="cuda")     # 1 GiB
    out = {}
    for name, fn, nbytes in calls:
        res = {}
        for mode in ("cold", "warm"):
            fn()
            ts = []
            for _ in range(reps):
                if mode == "cold":
                    scratch.add_(1.0)
                ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                ev0.record(stream)
                fn()
                ev1.record(stream)
                torch.cuda.synchronize()
                ts.append(ev0.elapsed_time(ev1) * 1e3)
            med = float(np.median(ts))
            gbs = nbytes / (med * 1e-6) / 1e9
            res[mode] = dict(median_us=round(med, 2), min_us=round(float(np.min(ts)), 2),
                             max_us=round(float(np.max(ts)), 2), GBps=round(gbs, 1),
                             frac_hbm=round(gbs / PEAK_HBM_GBS, 4))
        out[name] = dict(bytes=int(nbytes), reps=reps, **res)
    del scratch
    return out


# --------------------------------------------------------------------------- rocprofv3 summaries
# What the profile passes collect (one rocprofv3 --pmc run each; a run may hold at
# most 8 SQ, 4 TCC, 2 GRBM counters).
PMC_PASSES = {
    "sq": "SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_WAVE_CYCLES "
          "SQ_WAIT_ANY SQ_WAIT_INST_LDS SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE",
    "sq8": "SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES SQ_INSTS_VALU_MFMA_MOPS_F8 SQ_INSTS_VALU_MFMA_MOPS_F6F4 "
           "SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_LDS SQ_INSTS_LDS GRBM_GUI_ACTIVE",
    "lds": "SQ_LDS_IDX_ACTIVE SQ_LDS_DATA_FIFO_FULL SQ_LDS_CMD_FIFO_FULL SQ_INSTS_LDS_LOAD_BANDWIDTH "
           "SQ_INSTS_LDS_STORE_BANDWIDTH SQ_WAIT_INST_ANY SQ_ACTIVE_INST_MISC SQ_WAVE_CYCLES GRBM_GUI_ACTIVE",
    "vmem": "SQ_VMEM_TA_ADDR_FIFO_FULL SQ_VMEM_TA_CMD_FIFO_FULL "
            "SQ_ACTIVE_INST_VMEM SQ_WAVE_CYCLES TA_TA_BUSY TA_ADDR_STALLED_BY_TC_CYCLES TD_TD_BUSY TD_TC_STALL "
            "TCP_TCC_READ_REQ TCP_TCC_READ_REQ_LATENCY TCP_PENDING_STALL_CYCLES TCP_TCR_TCP_STALL_CYCLES "
            "GRBM_GUI_ACTIVE",
    "l2": "TCC_HIT TCC_MISS TCC_EA0_RDREQ TCC_EA0_RDREQ_LEVEL GRBM_GUI_ACTIVE",
    "fetch": "FETCH_SIZE GRBM_GUI_ACTIVE",
    "write": "WRITE_SIZE GRBM_GUI_ACTIVE",
}
NUM_XCD, NUM_CU, NUM_SIMD = 8, 256, 1024
BF16_FLOP_PER_CU_CLK = 4096           # dense bf16 MFMA, gfx950


def _read_csv(path):
    import csv
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _segments(dispatches):
    """Split (dispatch_id, label, ...) records, ordered by dispatch id, into layer
    steps: a step starts at each route launch.  Within a step the second GEMM-1 or
    GEMM-2 launch is the shared expert's.  Returns [(step_index, label, record)]."""
    out, step, seen = [], -1, {}
    for rec in dispatches:
        lab = rec["label"]
        if lab == "route":
            step += 1
            seen = {}
        if lab in ("gemm1", "gemm2"):
            n = seen.get(lab, 0)
            seen[lab] = n + 1
            if n == 1:
                lab = lab + ".shared"
        out.append((step, lab, rec))
    return out


def summarize(root, c, warmup: int, steps: int, gather: bool = True, mx: bool = False):
    """Markdown tables from the rocprofv3 output under root:
    root/trace/*kernel_trace.csv (a default bench.py run: warmup, then the timed
    steps), root/<pass>/*counter_collection.csv (--profile-run under --pmc), and
    root/copy_<pass>/*counter_collection.csv (--copy-calibration BYTES under --pmc;
    the copy's size is read from root/copy_bytes.txt)."""
    import glob
    known = ("route", "permute_count", "permute_scan", "permute_rank", "permute_small", "permute_maps",
             "permute_copy", "tile_prefix", "gemm1", "gemm2", "tail_reduce", "combine", "quantize_rows")

    lines = [f"Workload {c.name}: T={c.T} H={c.H} E={c.E} k={c.k} F={c.F} Fs={c.Fs} {c.dtype}, "
             f"{'gather' if gather else 'x_perm'} path.", ""]
    # ---------------------------------------------------------------- kernel trace
    traced = {}
    for path in sorted(glob.glob(os.path.join(root, "trace", "*kernel_trace.csv"))):
        rows = []
        for r in _read_csv(path):
            lab = kernel_label(r["Kernel_Name"])
            if lab in known:
                rows.append(dict(id=int(r["Dispatch_Id"]), label=lab, name=r["Kernel_Name"],
                                 us=(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3))
        rows.sort(key=lambda r: r["id"])
        for st, lab, rec in _segments(rows):
            if warmup <= st < warmup + steps:
                traced.setdefault(lab, []).append(rec["us"])
    if traced:
        step_us = sum(float(np.mean(v)) * len(v) / steps for v in traced.values())
        lines += [f"Kernel trace (rocprofv3 --kernel-trace), the {steps} timed steps after {warmup} warmup "
                  "steps:", "",
                  "| kernel | launches | avg us | median us | min us | max us | % of step |",
                  "|---|---|---|---|---|---|---|"]
        for lab, v in sorted(traced.items(), key=lambda kv: -sum(kv[1])):
            lines.append(f"| {lab} | {len(v)} | {np.mean(v):.2f} | {np.median(v):.2f} | {np.min(v):.2f} | "
                         f"{np.max(v):.2f} | {100 * np.mean(v) * len(v) / steps / step_us:.2f} |")
        lines += ["", f"Sum of kernel averages per step: {step_us / 1e3:.3f} ms -> "
                      f"{c.T / (step_us * 1e-6) / 1e6:.3f} M tokens/s.", ""]
    bench_json = os.path.join(root, "trace", "bench.json")
    if os.path.exists(bench_json):
        line = [ln for ln in open(bench_json) if ln.startswith("{")][-1]
        bj = json.loads(line)
        lines += [f"The same run's bench.py line: {bj['ms_per_step']} ms/step, {bj['value']:.0f} tokens/s; "
                  f"its GEMM-1 (HIP events in the timed region) {bj['kernels_us'].get(GEMM1)} us, "
                  f"roofline.frac {bj['roofline']['frac']}.", ""]
    # ---------------------------------------------------------------- counters
    calib = {}
    copy_bytes_path = os.path.join(root, "copy_bytes.txt")
    copy_bytes = int(open(copy_bytes_path).read().split()[0]) if os.path.exists(copy_bytes_path) else None
    per = {}                       # label -> counter -> [values]; label -> "us" -> [durations]
    for path in sorted(glob.glob(os.path.join(root, "*", "*counter_collection.csv"))):
        pass_name = os.path.basename(os.path.dirname(path))
        by_disp = {}
        for r in _read_csv(path):
            d = by_disp.setdefault(int(r["Dispatch_Id"]), dict(id=int(r["Dispatch_Id"]), name=r["Kernel_Name"],
                                                              label=kernel_label(r["Kernel_Name"]),
                                                              counters={}))
            d["counters"][r["Counter_Name"]] = float(r["Counter_Value"])
            d["us"] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        recs = sorted(by_disp.values(), key=lambda d: d["id"])
        if pass_name.startswith("copy_"):
            for d in recs:
                if "copy" in d["name"].lower():
                    for k, v in d["counters"].items():
                        calib.setdefault(k, []).append(v)
            continue
        for st, lab, d in _segments([r for r in recs if r["label"] in known]):
            if st < 1:
                continue                          # the profile run's first step warms up
            slot = per.setdefault(lab, {})
            for k, v in d["counters"].items():
                slot.setdefault(k, []).append(v)
            slot.setdefault("us", []).append(d["us"])
    factor = {}
    for k in ("FETCH_SIZE", "WRITE_SIZE"):
        if copy_bytes and calib.get(k):
            factor[k] = copy_bytes / (float(np.median(calib[k])) * 1024.0)
    if per:
        lines += ["Counters (rocprofv3 --pmc, one pass per counter set, dispatches serialized by the "
                  "profiler; averages over the profile run's layer steps 2-3, plus its x_perm permute):", ""]
        if factor:
            lines += [f"HBM-byte calibration: a plain {copy_bytes / 2**30:.2f} GiB device copy reads "
                      f"FETCH_SIZE x {factor.get('FETCH_SIZE', float('nan')):.3f} and WRITE_SIZE x "
                      f"{factor.get('WRITE_SIZE', float('nan')):.3f} of its size; the same factors scale the "
                      "kernels' counters below.", ""]
        lines += ["Columns: duration under the counter passes; shader clock = GRBM_GUI_ACTIVE per XCD / "
                  "duration (kernels of 100 us or more); MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (cycles x "
                  "1024 SIMDs); MFMA-work cycles = counted MFMA flop (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 at 4096 flop "
                  "per CU cycle, SQ_INSTS_VALU_MFMA_MOPS_F8 + _F6F4 x 512 at 8192) / 256 CUs, over the elapsed "
                  "cycles; waiting = SQ_WAIT_ANY / "
                  "SQ_WAVE_CYCLES, LDS-issue wait = SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES; bytes = FETCH_SIZE + "
                  "WRITE_SIZE (bytes leaving or entering the L2s: Infinity Cache hits included), calibrated; "
                  "GB/s = algorithmic bytes / the traced average duration (* : kernel not in the timed "
                  "steps, duration of the counter pass).", "",
                  "| kernel | us (pmc run) | clock GHz | MFMA busy % | MFMA-work cycles / elapsed | "
                  "counted bf16 flop / algorithmic | wave-cycles waiting % | LDS-issue wait % | "
                  "L2-egress bytes | / algorithmic bytes | algorithmic GB/s | % of 8 TB/s |",
                  "|---|---|---|---|---|---|---|---|---|---|---|---|"]
        for lab in sorted(per, key=lambda l: -float(np.mean(per[l]["us"]))):
            s = per[lab]
            m = {k: float(np.mean(v)) for k, v in s.items()}
            us = m["us"]
            grbm = m.get("GRBM_GUI_ACTIVE")
            cyc = grbm / NUM_XCD if grbm else None               # elapsed cycles (per XCD)
            # the GRBM window includes the dispatch itself, so the clock is meaningful
            # for long kernels only
            clk = cyc / (us * 1e3) if cyc and us >= 100 else None
            busy = 100 * m["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * NUM_SIMD) \
                if cyc and "SQ_VALU_MFMA_BUSY_CYCLES" in m else None
            flops, nbytes = algorithmic_work(c, lab, gather, mx)
            cflop16 = m.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512
            cflop8 = (m.get("SQ_INSTS_VALU_MFMA_MOPS_F8", 0.0) + m.get("SQ_INSTS_VALU_MFMA_MOPS_F6F4", 0.0)) * 512
            cflop = cflop16 + cflop8
            work = (cflop16 / BF16_FLOP_PER_CU_CLK + cflop8 / (2 * BF16_FLOP_PER_CU_CLK)) / NUM_CU / cyc \
                if cyc and cflop else None
            wait = 100 * m["SQ_WAIT_ANY"] / m["SQ_WAVE_CYCLES"] \
                if m.get("SQ_WAVE_CYCLES") and "SQ_WAIT_ANY" in m else None
            lwait = 100 * m["SQ_WAIT_INST_LDS"] / m["SQ_WAVE_CYCLES"] \
                if m.get("SQ_WAVE_CYCLES") and "SQ_WAIT_INST_LDS" in m else None
            hbm = None
            if "FETCH_SIZE" in m and "WRITE_SIZE" in m and factor:
                hbm = m["FETCH_SIZE"] * 1024 * factor["FETCH_SIZE"] + m["WRITE_SIZE"] * 1024 * factor["WRITE_SIZE"]
            t_us = float(np.mean(traced[lab])) if lab in traced else None
            mark = "" if t_us else " *"
            gbs = nbytes / ((t_us or us) * 1e3) if nbytes else None

            def f(v, fmt):
                return "-" if v is None else format(v, fmt)
            lines.append(f"| {lab} | {f(us, '.1f')} | {f(clk, '.3f')} | {f(busy, '.1f')} | {f(work, '.3f')} | "
                         f"{f(cflop / flops if flops and cflop else None, '.4f')} | {f(wait, '.1f')} | "
                         f"{f(lwait, '.1f')} | {f(hbm / 1e6 if hbm else None, '.1f')} MB | "
                         f"{f(hbm / nbytes if hbm and nbytes else None, '.2f')} | {f(gbs, '.0f')}{mark} | "
                         f"{f(100 * gbs / PEAK_HBM_GBS if gbs else None, '.1f')}{mark} |")
        lines.append("")
        lds_rows = [lab for lab in per if "SQ_LDS_IDX_ACTIVE" in per[lab] and lab.startswith("gemm")]
        if lds_rows:
            lines += ["LDS of the grouped GEMMs (the `lds` pass; per compute unit and elapsed cycle): LDS active = "
                      "SQ_LDS_IDX_ACTIVE / (cycles x 256 CUs); bytes read by LDS instructions = "
                      "SQ_INSTS_LDS_LOAD_BANDWIDTH x 64 / (cycles x 256) (the operand fragments; the direct "
                      "global -> LDS loads that fill the stages are not LDS instructions); data / command FIFO "
                      "full = SQ_LDS_DATA_FIFO_FULL, SQ_LDS_CMD_FIFO_FULL / (cycles x 256); any-instruction "
                      "wait and misc (barrier, waitcnt) active = SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_MISC / "
                      "SQ_WAVE_CYCLES.", "",
                      "| kernel | LDS active % | LDS-read bytes per CU cycle | LDS-instruction store bytes "
                      "per CU cycle | data FIFO full % | command FIFO full % | wave-cycles waiting on an "
                      "instruction % | misc active % |",
                      "|---|---|---|---|---|---|---|---|"]
            for lab in sorted(lds_rows):
                m = {k: float(np.mean(v)) for k, v in per[lab].items()}
                cu_cyc = m["GRBM_GUI_ACTIVE"] / NUM_XCD * NUM_CU
                wc = m.get("SQ_WAVE_CYCLES")

                def pct(k, d):
                    return "-" if k not in m or not d else f"{100 * m[k] / d:.1f}"
                rd = m.get("SQ_INSTS_LDS_LOAD_BANDWIDTH", 0.0) * 64 / cu_cyc
                wr = m.get("SQ_INSTS_LDS_STORE_BANDWIDTH", 0.0) * 64 / cu_cyc
                lines.append(f"| {lab} | {pct('SQ_LDS_IDX_ACTIVE', cu_cyc)} | {rd:.1f} | {wr:.1f} | "
                             f"{pct('SQ_LDS_DATA_FIFO_FULL', cu_cyc)} | {pct('SQ_LDS_CMD_FIFO_FULL', cu_cyc)} | "
                             f"{pct('SQ_WAIT_INST_ANY', wc)} | {pct('SQ_ACTIVE_INST_MISC', wc)} |")
            lines.append("")
        vm_rows = [lab for lab in per if "TA_TA_BUSY" in per[lab] and lab.startswith("gemm")]
        if vm_rows:
            lines += ["Load path of the grouped GEMMs (the `vmem` pass): TA / TD busy and stalled = TA_TA_BUSY, "
                      "TA_ADDR_STALLED_BY_TC_CYCLES, TD_TD_BUSY, TD_TC_STALL / (cycles x 256 CUs); "
                      "L1 -> L2 read latency = "
                      "TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ; TA FIFO full = SQ_VMEM_TA_ADDR_FIFO_FULL + "
                      "SQ_VMEM_TA_CMD_FIFO_FULL / (cycles x 256); TCP pending / TCR stall = "
                      "TCP_PENDING_STALL_CYCLES, TCP_TCR_TCP_STALL_CYCLES / (cycles x 256).", "",
                      "| kernel | TA busy % | TA stalled by L2 % | TD busy % | TD stalled by L2 % | "
                      "L1 -> L2 read latency, cycles | TA FIFO full % | "
                      "TCP pending stall % | TCR stall % |",
                      "|---|---|---|---|---|---|---|---|---|"]
            for lab in sorted(vm_rows):
                m = {k: float(np.mean(v)) for k, v in per[lab].items()}
                cu_cyc = m["GRBM_GUI_ACTIVE"] / NUM_XCD * NUM_CU

                def pc(*ks):
                    return "-" if any(k not in m for k in ks) else f"{100 * sum(m[k] for k in ks) / cu_cyc:.1f}"

                def ratio(a, b):
                    return "-" if not m.get(b) or a not in m else f"{m[a] / m[b]:.0f}"
                lines.append(f"| {lab} | {pc('TA_TA_BUSY')} | {pc('TA_ADDR_STALLED_BY_TC_CYCLES')} | "
                             f"{pc('TD_TD_BUSY')} | {pc('TD_TC_STALL')} | "
                             f"{ratio('TCP_TCC_READ_REQ_LATENCY', 'TCP_TCC_READ_REQ')} | "
                             f"{pc('SQ_VMEM_TA_ADDR_FIFO_FULL', 'SQ_VMEM_TA_CMD_FIFO_FULL')} | "
                             f"{pc('TCP_PENDING_STALL_CYCLES')} | {pc('TCP_TCR_TCP_STALL_CYCLES')} |")
            lines.append("")
        l2_rows = [lab for lab in per if "TCC_HIT" in per[lab] and "TCC_MISS" in per[lab]]
        if l2_rows:
            lines += ["L2 (the `l2` pass): hit rate = TCC_HIT / (TCC_HIT + TCC_MISS) over all requests reaching "
                      "the L2s; reads sent past the L2 (to the Infinity Cache or HBM) per algorithmic byte = "
                      "TCC_EA0_RDREQ x 128 B / algorithmic bytes (requests of up to 128 B); their mean time in "
                      "flight = TCC_EA0_RDREQ_LEVEL / TCC_EA0_RDREQ (cycles, Little's law).", "",
                      "| kernel | L2 hit rate % | read requests past L2 x 128 B / algorithmic bytes | "
                      "mean read time past L2, cycles |",
                      "|---|---|---|---|"]
            for lab in sorted(l2_rows, key=lambda l: -float(np.mean(per[l]["us"]))):
                m = {k: float(np.mean(v)) for k, v in per[lab].items()}
                tot = m["TCC_HIT"] + m["TCC_MISS"]
                _, nbytes = algorithmic_work(c, lab, gather, mx)
                rd = m.get("TCC_EA0_RDREQ")
                past = f"{rd * 128 / nbytes:.2f}" if rd and nbytes else "-"
                lat = f"{m['TCC_EA0_RDREQ_LEVEL'] / rd:.0f}" if rd and "TCC_EA0_RDREQ_LEVEL" in m else "-"
                lines.append(f"| {lab} | {100 * m['TCC_HIT'] / tot:.1f} | {past} | {lat} |" if tot else
                             f"| {lab} | - | {past} | {lat} |")
            lines.append("")
        g = per.get("gemm1")
        if g and "FETCH_SIZE" in g and "WRITE_SIZE" in g and factor:
            hbm = float(np.mean(g["FETCH_SIZE"])) * 1024 * factor["FETCH_SIZE"] + \
                float(np.mean(g["WRITE_SIZE"])) * 1024 * factor["WRITE_SIZE"]
            lines += [f"source_sha256: {gemm_source_sha256(mx)}", f"gemm1_traffic_bytes_per_launch: {hbm:.6g}", ""]
    print("\n".join(lines))


def summarize_probe(root):
    """Counters per kernel instantiation (full template name) from the --pmc passes
    under root, for the stand-alone probes (--route-probe): duration, VALU
    instructions and the share of the SIMDs' issue cycles they fill (a wave64 VALU
    instruction holds its SIMD 4 cycles), wave-cycles spent waiting, bytes."""
    import glob
    import re
    per = {}
    for path in sorted(glob.glob(os.path.join(root, "*", "*counter_collection.csv"))):
        if os.path.basename(os.path.dirname(path)).startswith("copy_"):
            continue
        by_disp = {}
        for r in _read_csv(path):
            d = by_disp.setdefault(int(r["Dispatch_Id"]), dict(name=r["Kernel_Name"], counters={}))
            d["counters"][r["Counter_Name"]] = float(r["Counter_Value"])
            d["us"] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        for d in by_disp.values():
            m = re.search(r"(\w+_kernel<[^()]*>)", d["name"])
            if not m or not m.group(1).startswith(("route_kernel", "router_", "mfma_rate_kernel")):
                continue
            slot = per.setdefault(m.group(1), {})
            for k, v in d["counters"].items():
                slot.setdefault(k, []).append(v)
            slot.setdefault("us", []).append(d["us"])
    lines = ["| kernel | dispatches | us (pmc run) | clock GHz | MFMA busy % | VALU instr | VALU issue share % | "
             "wave-cycles waiting % | FETCH_SIZE KiB | WRITE_SIZE KiB |", "|---|---|---|---|---|---|---|---|---|---|"]
    for name, sl in per.items():
        m = {k: float(np.median(v)) for k, v in sl.items()}
        cyc = m.get("GRBM_GUI_ACTIVE", 0) / NUM_XCD
        valu = m.get("SQ_INSTS_VALU")
        share = 100 * valu * 4 / (cyc * NUM_SIMD) if valu and cyc else None
        wait = 100 * m["SQ_WAIT_ANY"] / m["SQ_WAVE_CYCLES"] if m.get("SQ_WAVE_CYCLES") and "SQ_WAIT_ANY" in m \
            else None

        def f(v, fmt):
            return "-" if v is None else format(v, fmt)
        clk = cyc / (m["us"] * 1e3) if cyc and m["us"] >= 100 else None
        busy = 100 * m["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * NUM_SIMD) if cyc and "SQ_VALU_MFMA_BUSY_CYCLES" in m \
            else None
        lines.append(f"| `{name}` | {len(sl['us'])} | {m['us']:.1f} | {f(clk, '.3f')} | {f(busy, '.1f')} | "
                     f"{f(valu, '.3g')} | {f(share, '.1f')} | "
                     f"{f(wait, '.1f')} | {f(m.get('FETCH_SIZE'), '.0f')} | {f(m.get('WRITE_SIZE'), '.0f')} |")
    print("\n".join(lines))


def summarize_dense(root):
    """Counters of the GEMM dispatches of a --dense-ceiling run (the vendor library's
    kernels beside this library's grouped ones) from the --pmc passes under root.
    Per kernel name, the dispatches within 80% of its longest (for the vendor kernel:
    the one dense GEMM of the projection's whole size, not the per-expert ones);
    medians over them."""
    import glob
    import re
    per = {}
    for path in sorted(glob.glob(os.path.join(root, "*", "*counter_collection.csv"))):
        by_disp = {}
        for r in _read_csv(path):
            n = r["Kernel_Name"]
            if "Cijk" not in n and "grouped_gemm" not in n:
                continue
            d = by_disp.setdefault(int(r["Dispatch_Id"]), dict(name=n, counters={}))
            d["counters"][r["Counter_Name"]] = d["counters"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            d["us"] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        longest = {}
        for d in by_disp.values():
            longest[d["name"]] = max(longest.get(d["name"], 0.0), d["us"])
        for d in by_disp.values():
            if d["us"] < 0.8 * longest[d["name"]]:
                continue
            m = re.search(r"MT\d+x\d+x\d+", d["name"])
            k = re.search(r"(\w+_kernel<[^()]*>)", d["name"])
            label = f"hipBLASLt {m.group(0)}" if m else (k.group(1) if k else d["name"][:60])
            slot = per.setdefault(label, {})
            for k, v in d["counters"].items():
                slot.setdefault(k, []).append(v)
            slot.setdefault("us", []).append(d["us"])
    lines = ["| kernel | dispatches | us (pmc run) | clock GHz | MFMA busy % | MFMA flop (counted) | "
             "L1->L2 read requests | mean L1->L2 latency, cycles | L1 pending-miss stall % | L2 hit % |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for name, sl in sorted(per.items(), key=lambda kv: -float(np.median(kv[1]["us"]))):
        m = {k: float(np.median(v)) for k, v in sl.items()}
        cyc = m.get("GRBM_GUI_ACTIVE", 0) / NUM_XCD

        def f(v, fmt):
            return "-" if v is None else format(v, fmt)
        # the GRBM window includes the dispatch itself: the clock is meaningful for long kernels only
        clk = cyc / (m["us"] * 1e3) if cyc and m["us"] >= 100 else None
        busy = 100 * m["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * NUM_SIMD) if cyc and "SQ_VALU_MFMA_BUSY_CYCLES" in m \
            else None
        mops = sum(m.get(k, 0.0) for k in ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F8",
                                            "SQ_INSTS_VALU_MFMA_MOPS_F6F4"))
        req = m.get("TCP_TCC_READ_REQ")
        lat = m["TCP_TCC_READ_REQ_LATENCY"] / req if req and "TCP_TCC_READ_REQ_LATENCY" in m else None
        pend = 100 * m["TCP_PENDING_STALL_CYCLES"] / (cyc * NUM_CU) if cyc and "TCP_PENDING_STALL_CYCLES" in m \
            else None
        hit = 100 * m["TCC_HIT"] / (m["TCC_HIT"] + m["TCC_MISS"]) if "TCC_HIT" in m and "TCC_MISS" in m else None
        lines.append(f"| `{name}` | {len(sl['us'])} | {m['us']:.1f} | {f(clk, '.3f')} | {f(busy, '.1f')} | "
                     f"{f(mops * 512 if mops else None, '.3e')} | {f(req, '.3e')} | {f(lat, '.0f')} | "
                     f"{f(pend, '.1f')} | {f(hit, '.1f')} |")
    print("\n".join(lines))


def main():
    import moegen

    ap = argparse.ArgumentParser(description=__doc__.split("\n")[1])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="memconstrained", choices=sorted(moegen.CONFIGS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gather", action="store_true",
                    help="materialize x_perm in moe_permute instead of gathering rows in the grouped FFN")
    ap.add_argument("--profile-run", action="store_true",
                    help="a short run for rocprofv3 counter passes: 1 warmup and 2 layer steps, then one "
                         "moe_permute that also writes x_perm; no profiler pass, no cold/warm timing, no "
                         "CPU baseline")
    ap.add_argument("--summarize", metavar="DIR", default=None,
                    help="print markdown tables from the rocprofv3 output under DIR (kernel traces and "
                         "counter passes of --profile-run / default runs of --config)")
    ap.add_argument("--probe", action="store_true",
                    help="with --summarize: counters per kernel instantiation of a --route-probe run")
    ap.add_argument("--dense", action="store_true",
                    help="with --summarize: counters of the GEMMs of a --dense-ceiling run")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="the matrix cores' rate with no memory traffic (register-only probe), bf16 and fp8")
    ap.add_argument("--dense-ceiling", action="store_true",
                    help="time torch.matmul (hipBLASLt) expert by expert on the workload's groups, for context")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES (HBM counter calibration)")
    ap.add_argument("--sweep", choices=sorted(SWEEP_SHAPES), default=None,
                    help="expert-batch sweep of one layer shape: one JSON line per batch size")
    ap.add_argument("--mxfp8", action="store_true",
                    help="time the layer with MXFP8 expert GEMMs on --config (a separate JSON line)")
    ap.add_argument("--router-probe", action="store_true",
                    help="only time moe_router_topk (router GEMM + gate) on the layer shapes")
    ap.add_argument("--stream-probe", action="store_true",
                    help="weight-panel streaming rate against the row pitch, with and without a per-panel k start")
    ap.add_argument("--graph-probe", action="store_true",
                    help="small batches: a layer step call by call against the same step replayed as a HIP graph")
    ap.add_argument("--route-probe", action="store_true",
                    help="only time moe_route at 2^20 tokens (bandwidth probe), cold and warm")
    args = ap.parse_args()
    if args.summarize and args.probe:
        return summarize_probe(args.summarize)
    if args.summarize and args.dense:
        return summarize_dense(args.summarize)
    if args.summarize:
        return summarize(args.summarize, moegen.CONFIGS[args.config], args.warmup, args.steps,
                         gather=not args.no_gather, mx=args.mxfp8)
    if args.copy_calibration:
        return copy_calibration(args.copy_calibration)
    if args.dense_ceiling:
        return dense_ceiling_fp8(args.config) if args.mxfp8 else dense_ceiling(args.config)
    if args.mfma_ceiling:
        return mfma_ceiling()
    if args.route_probe:
        return route_probe()
    if args.graph_probe:
        return graph_probe(args.steps, args.warmup)
    if args.stream_probe:
        return stream_probe()
    if args.router_probe:
        return router_probe()
    if args.mxfp8:
        return mxfp8_bench(args.config, args.steps, args.warmup, profile_run=args.profile_run)
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
    gather = not args.no_gather
    layer = moe.MoELayer(c.T, c.H, c.E, c.k, c.F, c.Fs, dtype=dt, gather=gather)
    stream = torch.cuda.current_stream()

    def step():
        layer.run(x, logits, wg, wu, wd, *shared, renormalize=c.renormalize, stream=stream)

    if args.profile_run:
        # what the counter passes see: one warmup step, two steps, then one permute
        # that writes x_perm (the copy-path kernel), each dispatch serialized by the
        # profiler
        for i in range(3):
            log(f"profile run: layer step {i + 1} of 3")
            step()
            torch.cuda.synchronize()
        xp = torch.empty((c.R, c.H), dtype=dt, device="cuda")
        out = dict(layer.perm, x_perm=xp)
        moe.moe_permute(layer.topk_ids, x, c.E, out=out, ws=layer.ws_perm, stream=stream)
        torch.cuda.synchronize()
        log("profile run: done")
        print(json.dumps({"profile_run": c.name, "steps": 3}), flush=True)
        return

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

    # Route, permute and combine call by call, cold and warm.  The buffers hold the
    # last step's intermediates, so each call sees the layer's own inputs.
    log("timing route / permute / combine call by call, cold and warm")
    b = 4 if c.dtype == "f32" else 2
    maps_bytes = R * 4 + 2 * R * 4 + c.E * 4 + (c.E + 1) * 4
    xp = torch.empty((R, c.H), dtype=dt, device="cuda")
    perm_copy = dict(layer.perm, x_perm=xp)
    perm_maps = dict(layer.perm, x_perm=None)
    calls = [
        ("route", lambda: moe.moe_route(logits, c.k, c.renormalize, layer.topk_ids, layer.topk_weights,
                                        stream=stream),
         c.T * c.E * 4 + c.T * c.k * 8),
        ("permute_maps", lambda: moe.moe_permute(layer.topk_ids, x, c.E, out=perm_maps, ws=layer.ws_perm,
                                                 stream=stream),
         maps_bytes),
        ("permute_with_x_perm", lambda: moe.moe_permute(layer.topk_ids, x, c.E, out=perm_copy, ws=layer.ws_perm,
                                                        stream=stream),
         maps_bytes + c.T * c.H * b + R * c.H * b),
        ("combine", lambda: moe.moe_combine(layer.y_perm, layer.perm["dest_rows"], layer.topk_weights,
                                            layer.y_shared, y=layer.y, stream=stream),
         R * c.H * b + c.T * c.H * b * (2 if c.Fs else 1) + c.T * c.k * 8),
    ]
    bw = time_calls(calls, stream)
    del xp, perm_copy
    step()                                               # leave y as the layer's output
    torch.cuda.synchronize()
    bw["stream_copy_GBps"] = round(stream_copy_gbps(), 1)

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
                   "path": "permute maps + gather-fused grouped FFN" if gather
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
