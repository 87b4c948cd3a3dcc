#!/usr/bin/env python3
"""Benchmark of the fused BitLinear forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Workloads (shapes in workloads.py):
  decode_m1 (default), decode_m8, large_dec -- decode: a step is one forward
      (RMSNorm + int8 quant + VALU ternary contraction + dequant) for each of R
      distinct packed weight copies totalling >= 1 GiB, so every weight byte
      comes from HBM, issued back to back from one HIP graph.  value = HBM GB/s
      of algorithmic bytes (packed weights + x + gamma + y per call).
  glu_up, glu_down, large, tiny -- prefill: a step is one forward over all M
      tokens.  value = effective TOPS, 2*M*N*K / step time.

The JSON line carries the roofline of the dominant kernel (the contraction),
timed alone with HIP events on the stream it runs on, and the CPU oracle timed
on a bounded sample of the same workload.  The default run also reports the
GLU up-projection prefill (effective TOPS vs the int8 MFMA peak) under
"secondary".
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefill effective TOPS (2·M·N·K) vs int8 MFMA peak; decode HBM GB/s"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
INT8_PEAK_TOPS = 5000.0        # MI355X dense int8 MFMA, TOPS (5.0 POPS)
DECODE = ("decode_m1", "decode_m8", "large_dec")
ROTATE_BYTES = 1 << 30         # distinct packed weights per decode step


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="decode_m1")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    return ap.parse_args()


def check_single_gpu(args):
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        msg = ("bench.py measures one GPU only: the fused BitLinear path is built and timed on a "
               "single MI355X (no collectives, no sharding); run it with --gpus 1")
        if int(os.environ.get("RANK", "0")) == 0:
            print(msg, flush=True)
        sys.exit(2)


# ---------------------------------------------------------------------------
# byte and op counts (algorithmic)
# ---------------------------------------------------------------------------

def forward_bytes(w, x_bytes_per_elem):
    """x + gamma + packed weights + w_scale + y for one forward call."""
    return (w.M * w.K * x_bytes_per_elem + 4 * w.K + (w.K // 16) * w.N * 4 + 4 + 4 * w.M * w.N)


def contraction_bytes(w):
    """q + a_scale + q_rowsum + packed weights + w_scale + y for one contraction launch."""
    return w.M * w.K + 8 * w.M + (w.K // 16) * w.N * 4 + 4 + 4 * w.M * w.N


# ---------------------------------------------------------------------------

class Timer:
    def __init__(self, torch):
        self.torch = torch

    def time(self, fn, steps, warmup):
        torch = self.torch
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(steps):
            fn()
        end.record()
        torch.cuda.synchronize()
        return start.elapsed_time(end) / steps  # ms


def setup_common(torch, mmf, w):
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    xd, _ = workloads.make_x(w)
    if xd.dtype == np.float32:
        x = torch.from_numpy(xd).to(dev)
    else:
        x = torch.from_numpy(xd.view(np.int16)).to(dev).view(torch.bfloat16)
    gamma = None if w.gamma_kind == "ones" else torch.from_numpy(workloads.make_gamma(w)).to(dev)
    W0 = torch.from_numpy(workloads.make_w(w)).to(dev)
    Wp0, ws0 = mmf.ternarize(W0)
    del W0
    return dev, x, gamma, Wp0, ws0


def bench_decode(torch, mmf, w, args):
    dev, x, gamma, Wp0, ws0 = setup_common(torch, mmf, w)
    packed = (w.K // 16) * w.N * 4
    R = max(1, math.ceil(ROTATE_BYTES / packed))
    log(f"[bench] {w.name}: M={w.M} K={w.K} N={w.N}, {R} weight copies ({R * packed / 2**30:.2f} GiB)")
    gen = torch.Generator(device=dev)
    gen.manual_seed(240602528)
    Wps, wss = [Wp0], [ws0]
    for _ in range(R - 1):
        Wl = torch.randn((w.N, w.K), generator=gen, device=dev) * 0.02
        Wp, ws = mmf.ternarize(Wl)
        Wps.append(Wp)
        wss.append(ws)
    del Wl
    y = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    wsb = torch.empty(mmf.mmf_bitlinear_workspace_bytes(w.M, w.K), dtype=torch.uint8, device=dev)
    q = torch.empty((w.M, w.K), dtype=torch.int8, device=dev)
    a = torch.empty((w.M,), dtype=torch.float32, device=dev)
    rs = torch.empty((w.M,), dtype=torch.int32, device=dev)
    mmf.mmf_act_quant(x, gamma, q, a, rs)

    def fwd_all():
        for i in range(R):
            mmf.mmf_bitlinear_fwd_ws(x, gamma, Wps[i], wss[i], y, wsb)

    def contract_all():
        for i in range(R):
            mmf.mmf_ternary_gemm_dequant(q, a, rs, Wps[i], wss[i], y)

    graphs = {}
    for name, fn in (("fwd", fwd_all), ("contract", contract_all)):
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        graphs[name] = g
    timer = Timer(torch)
    log("[bench] timing the forward graph")
    ms_step = timer.time(graphs["fwd"].replay, args.steps, args.warmup)
    log("[bench] timing the contraction graph")
    ms_contract = timer.time(graphs["contract"].replay, args.steps, args.warmup) / R
    fb = forward_bytes(w, x.element_size())
    cb = contraction_bytes(w)
    value = R * fb / (ms_step * 1e-3) / 1e9
    achieved = cb / (ms_contract * 1e-3) / 1e9
    # hot-cache single call, for context
    ms_hot = timer.time(lambda: mmf.mmf_bitlinear_fwd_ws(x, gamma, Wp0, ws0, y, wsb),
                        max(args.steps * 10, 50), args.warmup)
    result = {
        "value": value, "unit": "GB/s", "ms_per_step": ms_step,
        "config": {"workload": w.name, "M": w.M, "K": w.K, "N": w.N, "x_dtype": w.x_dtype,
                   "weight_copies": R, "calls_per_step": R,
                   "bytes_per_call": fb, "graph": True},
        "roofline": {"bound": "hbm", "kernel": "gemv_kernel (decode contraction)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "bytes_per_launch": cb, "avg_launch_us": ms_contract * 1e3},
        "hot_cache_call_us": ms_hot * 1e3,
    }
    return result, fb


def bench_prefill(torch, mmf, w, args):
    dev, x, gamma, Wp, ws = setup_common(torch, mmf, w)
    log(f"[bench] {w.name}: M={w.M} K={w.K} N={w.N}")
    y = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    wsb = torch.empty(mmf.mmf_bitlinear_workspace_bytes(w.M, w.K), dtype=torch.uint8, device=dev)
    q = torch.empty((w.M, w.K), dtype=torch.int8, device=dev)
    a = torch.empty((w.M,), dtype=torch.float32, device=dev)
    rs = torch.empty((w.M,), dtype=torch.int32, device=dev)
    mmf.mmf_act_quant(x, gamma, q, a, rs)
    timer = Timer(torch)
    ms_step = timer.time(lambda: mmf.mmf_bitlinear_fwd_ws(x, gamma, Wp, ws, y, wsb),
                         args.steps, args.warmup)
    ms_gemm = timer.time(lambda: mmf.mmf_ternary_gemm_dequant(q, a, rs, Wp, ws, y),
                         args.steps, args.warmup)
    ms_aq = timer.time(lambda: mmf.mmf_act_quant(x, gamma, q, a, rs), args.steps, args.warmup)
    tops = w.ops / (ms_step * 1e-3) / 1e12
    gemm_tops = w.ops / (ms_gemm * 1e-3) / 1e12
    aq_bytes = w.M * w.K * x.element_size() + 4 * w.K + w.M * w.K + 8 * w.M
    result = {
        "value": tops, "unit": "TOPS", "ms_per_step": ms_step,
        "config": {"workload": w.name, "M": w.M, "K": w.K, "N": w.N, "x_dtype": w.x_dtype},
        "roofline": {"bound": "mfma", "kernel": "gemm_kernel (prefill contraction)",
                     "achieved": gemm_tops, "peak": INT8_PEAK_TOPS, "unit": "TFLOP/s",
                     "frac": gemm_tops / INT8_PEAK_TOPS, "traffic": None,
                     "ops_per_launch": w.ops, "avg_launch_us": ms_gemm * 1e3},
        "act_quant": {"avg_launch_us": ms_aq * 1e3, "bytes": aq_bytes,
                      "GB/s": aq_bytes / (ms_aq * 1e-3) / 1e9},
    }
    return result


def cpu_baseline(w, fb, seconds):
    """The oracle, as it stands, on a bounded sample of the same workload."""
    import numpy as np
    import oracle
    import workloads
    _, xf = workloads.make_x(w)
    g = None if w.gamma_kind == "ones" else workloads.make_gamma(w)
    W = workloads.make_w(w)
    t, ws = oracle.weight_quant(W)
    threads = oracle.num_threads()
    if w.name in DECODE:
        calls = 0
        t0 = time.perf_counter()
        while True:
            oracle.bitlinear_fwd(xf, g, t, ws)
            calls += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                break
        return {"value": calls * fb / el / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
                "sample": f"{calls} full forward calls (M={w.M}, K={w.K}, N={w.N}) in {el:.1f} s; "
                          "bytes counted as for the GPU (packed weights + x + gamma + y)"}
    # prefill: a row sample, timed once, grown until it takes >= 1/4 of the budget
    rows = 8
    while True:
        t0 = time.perf_counter()
        oracle.bitlinear_fwd(xf[:rows], g, t, ws)
        el = time.perf_counter() - t0
        if el >= seconds / 4 or rows >= w.M:
            break
        rows = min(w.M, rows * max(2, int(seconds / 4 / max(el, 1e-3))))
    return {"value": 2.0 * rows * w.N * w.K / el / 1e12, "unit": "TOPS", "cores": threads,
            "kind": "oracle",
            "sample": f"{rows} of {w.M} token rows (K={w.K}, N={w.N}) in {el:.1f} s"}


def main():
    args = parse()
    check_single_gpu(args)
    import torch
    import paper_2406_02528_amd as mmf
    import workloads
    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    w = workloads.WORKLOADS[args.workload]
    if w.name in DECODE:
        res, fb = bench_decode(torch, mmf, w, args)
    else:
        res = bench_prefill(torch, mmf, w, args)
        fb = forward_bytes(w, 4 if w.x_dtype == "f32" else 2)
    line = {
        "metric": METRIC, "value": res["value"], "unit": res["unit"], "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int8",
        "data": "synthetic (seeded; shapes of the paper's model widths)",
        "config": res["config"], "roofline": res["roofline"],
    }
    for k in ("hot_cache_call_us", "act_quant"):
        if k in res:
            line[k] = res[k]
    if not args.no_secondary and w.name in DECODE:
        sw = workloads.WORKLOADS["glu_up"]
        log("[bench] secondary: glu_up prefill")
        sec = bench_prefill(torch, mmf, sw, args)
        line["secondary"] = {"metric": "prefill effective TOPS", "value": sec["value"],
                             "unit": "TOPS", "ms_per_step": sec["ms_per_step"],
                             "config": sec["config"], "roofline": sec["roofline"],
                             "act_quant": sec["act_quant"]}
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        line["cpu_baseline"] = cpu_baseline(w, fb, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
