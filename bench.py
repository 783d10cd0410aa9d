#!/usr/bin/env python3
"""Benchmark of the fused MoE layer (gate -> top-k -> SwiGLU experts ->
weighted combine) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config N]

One step is one ``moe_forward`` call over one batch of synthetic inputs that
are already resident in HBM.  The default workload is the largest one that
fits one GPU, the fp8 block-quantised layer (T=8192, H=7168, E=256, I=2048,
top_k=8); ``--config`` selects one of the other workloads.  Prints ONE JSON
line on stdout.

Timing:
  * whole layer: HIP events on the launch stream around exactly K calls,
    bracketed by device synchronisation; host wall clock reported beside it.
    Each timed call is ``moe_forward_profiled`` with an event at its start
    (so every step's duration is known: median, p10 and p90 are reported
    beside the mean) and the two events around GEMM1, so the dominant
    kernel's per-launch duration (the roofline's denominator) is measured
    live inside the same timed region;
  * per stage: after the timed region, K further calls with events between
    all stages (a breakdown only; these events cost a few microseconds each);
  * graph: the same layer captured once in a HIP graph and replayed K times
    (how a serving loop would run it), reported beside ``value``, which
    stays the stream-launched figure;
  * traffic: HBM bytes per launch from committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE counters, only if the kernel sources still hash to the value
    they were taken at (else null);
  * cpu_baseline: the fp64 oracle on the host cores, on a bounded sample.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fused-MoE layer TFLOP/s (active FLOPs) + µs/layer; fraction of MFMA/HBM peak"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0}
W_BYTES = {"bf16": 2.0, "fp8": 1.0, "int4": 0.5, "fp8a16": 1.0, "mxfp4": 0.5, "mxfp4x8": 0.5}
DESCR = {
    1: "tiny MoE layer: T=64 H=256 E=8 I=128 top_k=2, bf16 weights, softmax top-2 renormalised",
    2: "decode-shaped MoE layer: T=16 H=4096 E=64 I=1408 top_k=6, bf16 weights, softmax top-6 renormalised",
    3: "prefill-shaped MoE layer: T=4096 H=4096 E=64 I=1408 top_k=6, bf16 weights, biased softmax top-6",
    4: "fp8 block-quantised MoE layer: T=8192 H=7168 E=256 I=2048 top_k=8, e4m3 128x128 weights, "
       "per-(token,128) e4m3 activations, sigmoid+bias top-8 x2.5",
    5: "int4 weight-only MoE layer: T=512 H=4096 E=128 I=1536 top_k=8, int4 g128 weights, "
       "Zipf(1.1)-skewed softmax top-8",
    6: "weight-only fp8 decode MoE layer: T=16 H=7168 E=256 I=2048 top_k=8, e4m3 128x128 weights, "
       "bf16 activations, sigmoid+bias top-8 x2.5",
    7: "MXFP4 decode MoE layer: T=16 H=7168 E=256 I=2048 top_k=8, OCP MX E2M1 weights with E8M0 "
       "scales per 32, bf16 activations, sigmoid+bias top-8 x2.5",
    8: "MXFP4 prefill MoE layer: T=8192 H=7168 E=256 I=2048 top_k=8, OCP MX E2M1 weights with E8M0 "
       "scales per 32, bf16 activations, sigmoid+bias top-8 x2.5",
    9: "MXFP4 x MXFP8 prefill MoE layer: T=8192 H=7168 E=256 I=2048 top_k=8, OCP MX E2M1 weights and "
       "in-layer MXFP8 (e4m3, E8M0 per 32) activations, sigmoid+bias top-8 x2.5",
    10: "int4 decode MoE layer: T=16 H=4096 E=128 I=1536 top_k=8, int4 g128 weights, "
        "Zipf(1.1)-skewed softmax top-8",
}


# sources that define the GEMM1 kernels (the roofline's dominant kernel)
GEMM_SOURCES = ("common.hpp", "launch.hpp", "lds_dma.hpp", "dispatch.hip", "gemm_bf16.hip", "gemm_tiled.hip")


def _code_only(text: str) -> str:
    """C++ source without comments and with whitespace runs collapsed, so an
    edit of comments alone does not count as a kernel change."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in sorted(os.path.join(ROOT, "paper_2607_12875_amd", "csrc", n) for n in GEMM_SOURCES):
        with open(p, encoding="utf-8") as f:
            h.update(os.path.basename(p).encode() + _code_only(f.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload_key: str, src_hash: str):
    """HBM bytes per GEMM1 launch from the committed counter summary, if the
    kernels have not changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload_key}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != src_hash:
        return None
    return rec.get("hbm_bytes_per_launch")


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch already loaded."""

    def __init__(self, n):
        self.rt = ctypes.CDLL("libamdhip64.so.7")
        self.rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.rt.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            assert self.rt.hipEventCreate(ctypes.byref(e)) == 0
            self.ev.append(e.value)

    def elapsed_ms(self, a, b):
        out = ctypes.c_float()
        assert self.rt.hipEventSynchronize(self.ev[b]) == 0
        assert self.rt.hipEventElapsedTime(ctypes.byref(out), self.ev[a], self.ev[b]) == 0
        return out.value

    def close(self):
        for e in self.ev:
            self.rt.hipEventDestroy(e)


def measure_peaks(moe, torch) -> dict:
    """Achievable peaks of this device, from the library's probes (see
    include/moe_peaks.h), each timed with HIP events over three launches on
    torch's current stream: MFMA-only loops in bf16 and fp8 (TFLOP/s), a
    2 GiB streaming read and a 2 GiB streaming copy (read + write bytes),
    GB/s; and the per-CU staging paths of the tiled GEMMs (global -> LDS
    copies from L2 and from HBM, LDS fragment reads), bytes per clock per
    CU."""
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    ev = HipEvents(2)
    ev.rt.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    out = {}

    def timed(fn, reps=3):
        fn()  # warm
        ev.rt.hipEventRecord(ev.ev[0], stream)
        for _ in range(reps):
            fn()
        ev.rt.hipEventRecord(ev.ev[1], stream)
        return ev.elapsed_ms(0, 1) / reps

    sink = torch.empty(moe.moe_peak_sink_elems(), dtype=torch.float32, device="cuda")
    iters = 4096
    for name, fp8 in (("mfma_bf16_tflops", False), ("mfma_fp8_tflops", True)):
        ms = timed(lambda: moe.moe_peak_mfma(fp8, iters, sink))
        out[name] = moe.moe_peak_mfma_flops_per_launch(fp8, iters) / (ms * 1e-3) / 1e12
    nbytes = 2 << 30
    src = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    words = torch.zeros(moe.moe_peak_sink_elems(), dtype=torch.int32, device="cuda")
    ms = timed(lambda: moe.moe_peak_read(src, words))
    out["hbm_read_gbs"] = nbytes / (ms * 1e-3) / 1e9
    ms = timed(lambda: moe.moe_peak_copy(src, dst))
    out["hbm_copy_gbs"] = 2 * nbytes / (ms * 1e-3) / 1e9
    # per-CU staging paths of the tiled GEMMs, in bytes per clock per CU at
    # the 2.4 GHz peak engine clock: global -> LDS copies by 4 or 8 issuing
    # waves (8 copies in flight each) from a 1 MiB region per XCD (L2) or a
    # 256 MiB one (HBM), and LDS fragment reads by 4 or 16 waves
    ncu = torch.cuda.get_device_properties(0).multi_processor_count

    def per_cu_clk(nb, ms_):
        return nb / (ms_ * 1e-3) / 2.4e9 / ncu

    steps = 200
    for tag, region in (("l2", 1 << 20), ("hbm", 256 << 20)):
        for waves in (4, 8):
            ms = timed(lambda: moe.moe_peak_lds_copy(src, region, waves, 8, steps))
            out[f"{tag}_to_lds_w{waves}_bytes_per_clk_cu"] = per_cu_clk(
                moe.moe_peak_lds_copy_bytes_per_launch(waves, 8, steps), ms)
    for waves in (4, 16):
        ms = timed(lambda: moe.moe_peak_lds_read(waves, 2000, words))
        out[f"lds_read_w{waves}_bytes_per_clk_cu"] = per_cu_clk(moe.moe_peak_lds_read_bytes_per_launch(waves, 2000), ms)
    ev.close()
    del src, dst, sink, words
    return out


def cpu_baseline(cfg, inputs, budget_s: float):
    """Time the fp64 oracle on the host: the whole layer when it fits the
    budget, else a token sample; returns the baseline record."""
    from oracle import moe_oracle as O
    # the oracle evaluates its experts on this many threads at once (one BLAS
    # thread each)
    cores = O.default_threads()
    tokens = None
    n_tok = cfg.T
    # the oracle dequantises every expert a token routes to: bound that work
    per_token = cfg.top_k * 3.0 * cfg.H * cfg.I
    if cfg.T * per_token > 2e9:
        n_tok = max(1, min(cfg.T, int(2e9 / per_token)))
        tokens = np.linspace(0, cfg.T - 1, n_tok).astype(np.int64)
    reps, t0 = 0, time.perf_counter()
    while True:
        O.forward(cfg, inputs, tokens=tokens)
        reps += 1
        if time.perf_counter() - t0 >= budget_s or reps >= 20:
            break
    dt = (time.perf_counter() - t0) / reps
    flops = 6.0 * n_tok * cfg.top_k * cfg.H * cfg.I
    sample = (f"{'all ' if tokens is None else ''}{n_tok} tokens of the same layer, "
              f"fp64 oracle incl. dequantisation, {reps} run(s), {dt:.2f} s each")
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": sample, "seconds_per_layer_sample": dt}


def gemm1_kernel_match(name: str) -> bool:
    """True for the GEMM1 (+SiLU*up) kernel of any format / variant."""
    decode = ("gemm_bf16_skinny<", "gemm_bf16_stream<", "gemm_w8a16_skinny<", "gemm_w4a16_skinny<")
    return (any(k in name for k in decode) and "true>" in name) or \
           ("moe_gemm_tiled<" in name and ", true," in name)


def traffic_summary(fetch_csv, write_csv, calib_fetch_csv, calib_write_csv, calib_mib):
    """HBM bytes per GEMM1 launch from rocprofv3 FETCH_SIZE / WRITE_SIZE
    counter CSVs (KiB per dispatch), each scaled by what the same counter
    reads for a plain device copy of calib_mib MiB."""
    import csv

    def per_kernel(path, match):
        vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path)) if match(r["Kernel_Name"])]
        return sum(vals) / len(vals), len(vals)

    copy = lambda n: "copyBuffer" in n  # noqa: E731
    nbytes = calib_mib * 1024 * 1024
    f_copy, _ = per_kernel(calib_fetch_csv, copy)
    w_copy, _ = per_kernel(calib_write_csv, copy)
    f_g1, n1 = per_kernel(fetch_csv, gemm1_kernel_match)
    w_g1, n2 = per_kernel(write_csv, gemm1_kernel_match)
    f_scale, w_scale = nbytes / (f_copy * 1024), nbytes / (w_copy * 1024)
    fetch, write = f_g1 * 1024 * f_scale, w_g1 * 1024 * w_scale
    return {"kernel": "gemm1 (+SiLU*up)", "fetch_size_kib_raw": f_g1, "write_size_kib_raw": w_g1,
            "dispatches": [n1, n2], "copy_calibration_mib": calib_mib,
            "copy_fetch_kib_raw": f_copy, "copy_write_kib_raw": w_copy,
            "fetch_scale": f_scale, "write_scale": w_scale,
            "hbm_fetch_bytes_per_launch": fetch, "hbm_write_bytes_per_launch": write,
            "hbm_bytes_per_launch": fetch + write, "kernel_source_hash": kernel_source_hash()}


def counter_summary(csv_paths, simd_per_cu=4):
    """Per-kernel averages per dispatch of every counter in rocprofv3
    counter-collection CSVs, plus MFMA busy as a fraction of the SIMD cycles
    (SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE * SIMDs)) when both were
    collected in the same pass."""
    import csv
    from collections import defaultdict
    vals = defaultdict(lambda: defaultdict(list))   # kernel -> counter -> per-dispatch values
    for path in csv_paths:
        rows = defaultdict(dict)                    # (kernel, dispatch) -> counter -> value
        for r in csv.DictReader(open(path)):
            key = (r["Kernel_Name"], r.get("Dispatch_Id") or r.get("Correlation_Id"))
            name = r["Counter_Name"]
            rows[key][name] = rows[key].get(name, 0.0) + float(r["Counter_Value"])
        for (kern, _), cs in rows.items():
            for name, v in cs.items():
                vals[kern][name].append(v)
    out = {}
    for kern, cs in vals.items():
        rec = {name: sum(v) / len(v) for name, v in cs.items()}
        rec["dispatches"] = max(len(v) for v in cs.values())
        if "SQ_VALU_MFMA_BUSY_CYCLES" in rec and "GRBM_GUI_ACTIVE" in rec:
            import torch
            cus = torch.cuda.get_device_properties(0).multi_processor_count if torch.cuda.is_available() else 256
            rec["mfma_busy_frac"] = rec["SQ_VALU_MFMA_BUSY_CYCLES"] / (rec["GRBM_GUI_ACTIVE"] * cus * simd_per_cu)
        out[kern] = rec
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=4, choices=sorted(DESCR))
    ap.add_argument("--router", action="store_true",
                    help="compute the logits in-layer from a router weight [E,H] (router GEMM fused "
                         "with the gate); the FLOP count stays that of the experts")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="host-time budget of the oracle baseline (0 disables it)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (the reference "
                         "kernel that scales HBM counter readings), then exit")
    ap.add_argument("--traffic-summary", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="host only: print the GEMM1 HBM-traffic record from rocprofv3 counter CSVs "
                         "(the copy ones from --copy-calibration 1024) and exit")
    ap.add_argument("--peaks", action="store_true",
                    help="only measure the device's achievable MFMA and memory peaks, print them, and exit")
    ap.add_argument("--counter-summary", nargs="+", metavar="CSV",
                    help="host only: print per-kernel counter averages (and MFMA busy fraction) from "
                         "rocprofv3 counter-collection CSVs and exit")
    args = ap.parse_args()
    if args.counter_summary:
        print(json.dumps(counter_summary(args.counter_summary), indent=1))
        return
    if args.traffic_summary:
        print(json.dumps(traffic_summary(*args.traffic_summary, 1024), indent=1))
        return
    if args.gpus != 1:
        print("bench.py: the MoE layer runs on one GPU only; sharding it across GPUs "
              "is described in the design notes, not implemented (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_12875_amd as moe
    import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}))
        return
    moe.lib()
    if args.peaks:
        print(json.dumps(measure_peaks(moe, torch)))
        return
    cfg = synth.config(args.config)
    t0 = time.perf_counter()
    inputs = synth.make_inputs(cfg)
    d = synth.to_device(inputs)
    w_router = None
    if args.router:
        w_router = synth.to_device({"w": synth.make_router_weights(cfg)})["w"]
    gen_s = time.perf_counter() - t0
    out = torch.empty((cfg.T, cfg.H), dtype=torch.float32, device="cuda")
    margs = moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, mode=cfg.mode,
                          renormalize=cfg.renormalize, routed_scale=cfg.routed_scale,
                          wfmt=cfg.wfmt, out_dtype="f32", hidden=d["hidden"],
                          logits=None if args.router else d["logits"],
                          w1=d["w1"], w2=d["w2"], w1_scale=d["w1_scale"], w2_scale=d["w2_scale"],
                          sel_bias=d["sel_bias"], out=out, w_router=w_router)
    ws = torch.empty(moe.moe_workspace_bytes(margs), dtype=torch.uint8, device="cuda")
    layout = moe.moe_workspace_layout(margs)
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        moe.moe_forward_args(margs, ws)
    torch.cuda.synchronize()

    # ---- whole layer: exactly K steps between two synchronisations; every
    # step brackets its GEMM1 launch with a pair of events of its own
    # events: 0 .. K-1 the start of each step, K the end of the last, then
    # the GEMM1 pair of each step
    K = args.steps
    ev = HipEvents(1 + 3 * K)
    rt = ev.rt
    rt.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    g1_marks = [[ev.ev[i], None, None, ev.ev[K + 1 + 2 * i], ev.ev[K + 2 + 2 * i], None, None] for i in range(K)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(K):
        moe.moe_forward_profiled(margs, ws, g1_marks[i])
    rt.hipEventRecord(ev.ev[K], ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3 / K
    ms = ev.elapsed_ms(0, K) / K
    step_us = np.array([ev.elapsed_ms(i, i + 1) * 1e3 for i in range(K)])
    g1_launch_us = [ev.elapsed_ms(K + 1 + 2 * i, K + 2 + 2 * i) * 1e3 for i in range(K)]
    ev.close()

    # ---- per-stage breakdown (after the timed region): events between stages
    sev = HipEvents(moe.NUM_STAGES + 1)
    stage_sum = np.zeros(moe.NUM_STAGES)
    for _ in range(K):
        moe.moe_forward_profiled(margs, ws, sev.ev)
        torch.cuda.synchronize()
        for i in range(moe.NUM_STAGES):
            stage_sum[i] += sev.elapsed_ms(i, i + 1)
    stage_us = {name: float(v * 1e3 / K) for name, v in zip(moe.STAGES, stage_sum)}
    sev.close()

    # ---- the same layer captured once in a HIP graph, replayed K times
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        moe.moe_forward_args(margs, ws)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        moe.moe_forward_args(margs, ws)
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    gev = HipEvents(2)
    rt.hipEventRecord(gev.ev[0], ctypes.c_void_p(stream.cuda_stream))
    for _ in range(K):
        graph.replay()
    rt.hipEventRecord(gev.ev[1], ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    graph_us = gev.elapsed_ms(0, 1) * 1e3 / K
    gev.close()
    del graph

    # routing statistics of this batch (from the layer's own workspace)
    offs = ws[layout["expert_offsets"]:layout["expert_offsets"] + 4 * (cfg.E + 1)].view(torch.int32).cpu().numpy()
    ids = ws[layout["topk_ids"]:layout["topk_ids"] + 4 * cfg.n_routed].view(torch.int32).cpu().numpy()
    counts = np.bincount(ids, minlength=cfg.E)
    n_active = int((counts > 0).sum())
    del offs

    flops = cfg.active_flops()
    wb = W_BYTES[cfg.wfmt]
    H, I, T, n = cfg.H, cfg.I, cfg.T, cfg.n_routed
    # GEMM1 per launch: W1 of every active expert (+ its scales), hidden read
    # once, the SwiGLU intermediate written once
    w1_scale_bytes = {"bf16": 0, "fp8": 2 * I * H / (128 * 128) * 4, "int4": 2 * I * H / 128 * 2,
                      "fp8a16": 2 * I * H / (128 * 128) * 4, "mxfp4": 2 * I * H / 32,
                      "mxfp4x8": 2 * I * H / 32}[cfg.wfmt]
    # bytes per element of the activation rows GEMM1 reads and of the
    # intermediate it writes (with their scales)
    act_bytes = {"bf16": 2, "fp8": 1 + 4 / 128, "int4": 2, "fp8a16": 2, "mxfp4": 2,
                 "mxfp4x8": 1 + 1 / 32}[cfg.wfmt]
    g1_bytes = n_active * (2 * I * H * wb + w1_scale_bytes) + T * H * act_bytes + n * I * act_bytes
    g1_flops = 2.0 * n * H * 2 * I
    g1_us = float(np.mean(g1_launch_us))
    # the roof that binds GEMM1: the larger of bytes / HBM peak and flops / MFMA peak
    # the matrix rate the products run at: fp8 for e4m3 activations (the
    # fp8 x fp4 instruction issues at the fp8 rate), bf16 otherwise
    mfma_peak = PEAK_TFLOPS["fp8" if cfg.wfmt in ("fp8", "mxfp4x8") else "bf16"]
    t_hbm = g1_bytes / (PEAK_HBM_GBS * 1e9)
    t_mfma = g1_flops / (mfma_peak * 1e12)
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    src_hash = kernel_source_hash()
    key = f"{synth.config(args.config).name}_gemm1"
    traffic = load_traffic(key, src_hash)
    common = {"kernel": "gemm1 (+SiLU*up)", "traffic": traffic, "launch_us": g1_us,
              "launch_us_median": float(np.median(g1_launch_us)),
              "algorithmic_bytes_per_launch": g1_bytes, "algorithmic_flops_per_launch": g1_flops,
              "roof_us": {"hbm": t_hbm * 1e6, "mfma": t_mfma * 1e6}}
    if bound == "hbm":
        achieved = g1_bytes / (g1_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, **common}
    else:
        achieved = g1_flops / (g1_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": mfma_peak,
                "unit": "TFLOP/s", "frac": achieved / mfma_peak, **common}

    # the device's achievable peaks beside the published ones the fraction uses
    peaks = measure_peaks(moe, torch)
    # (the GEMM's HBM traffic is almost all reads: the read ceiling)
    roof["peak_measured"] = peaks["hbm_read_gbs"] if bound == "hbm" else \
        peaks["mfma_fp8_tflops" if cfg.wfmt in ("fp8", "mxfp4x8") else "mfma_bf16_tflops"]
    roof["frac_of_measured_peak"] = roof["achieved"] / roof["peak_measured"]

    base = None
    if args.cpu_seconds > 0:
        base = cpu_baseline(cfg, inputs, args.cpu_seconds)

    dtype = {"bf16": "bf16", "fp8": "fp8e4m3", "int4": "bf16", "fp8a16": "bf16", "mxfp4": "bf16",
             "mxfp4x8": "mxfp8e4m3 x mxfp4e2m1"}[cfg.wfmt]
    rec = {
        "metric": METRIC,
        "value": flops / (ms * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic (seeded; recipe in synth/moe_inputs.py)",
        "config": {"workload": DESCR[args.config] + (", logits from a fused router GEMM (bf16 [E,H])" if args.router else ""), "T": T, "H": H, "E": cfg.E, "I": I,
                   "top_k": cfg.top_k, "wfmt": cfg.wfmt, "active_experts": n_active,
                   "max_rows_per_expert": int(counts.max()), "block_m": layout["block_m"]},
        "us_per_layer": ms * 1e3,
        "us_per_layer_median": float(np.median(step_us)),
        "us_per_layer_p10": float(np.percentile(step_us, 10)),
        "us_per_layer_p90": float(np.percentile(step_us, 90)),
        "wall_us_per_layer": wall_ms * 1e3,
        "graph_us_per_layer": graph_us,
        "stage_us": stage_us,
        "roofline": roof,
        "peaks_measured": peaks,
        "cpu_baseline": base,
        "kernel_source_hash": src_hash,
        "input_generation_s": gen_s,
    }
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
