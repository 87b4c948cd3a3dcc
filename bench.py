#!/usr/bin/env python3
"""Benchmark of the fused BitLinear forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

The default run measures the largest configuration of the headline metric:
``large`` (prefill at d = 5120, M=16384, K=5120, N=27648; effective TOPS
against the int8 MFMA peak) on the JSON line's top level, ``large_dec``
(decode at d = 5120, M=1, K=5120, N=15360; HBM GB/s) under "secondary", each
with its roofline, recorded HBM traffic and CPU oracle baseline, and the
decode_m1 and glu_up workloads under "extra" (roofline and traffic only).

Workloads (shapes in workloads.py):
  decode_m1, decode_m8, large_dec -- decode: a step is one forward
      (RMSNorm + int8 quant + VALU ternary contraction + dequant) for each of R
      distinct packed weight copies totalling >= 1 GiB, so every weight byte
      comes from HBM, issued back to back from one HIP graph.  value = HBM GB/s
      of algorithmic bytes (packed weights + x + gamma + y per call).
  large (default), glu_up, glu_down, tiny -- prefill: a step is one forward
      over all M tokens, i.e. the two launches mmf_bitlinear_fwd runs for
      M > 40 (act-quant, then the int8 MFMA contraction with the dequant
      epilogue), through mmf_bitlinear_fwd_ws.  value = effective TOPS,
      2*M*N*K / step time; the roofline times the contraction launch in a loop
      of its own (mmf_ternary_gemm_dequant on the same q).
  glu_gate -- the GLU channel mixer's fused up-projections and gate on the
      glu_up shape (M=8192, K=2048, L=5632): p = SiLU(g) * u in one contraction
      over the interleaved gate|up weights.  value = effective TOPS, 2*M*2L*K.
  channel_mixer -- the whole GLU channel mixer on that shape: glu_gate, then
      the down-projection BitLinear of p (K=5632, N=2048, its own RMSNorm).
      value = effective TOPS over both contractions.
  mlgru_decode -- one token step of the MLGRU token mixer at d = 2048 (input
      projections f|c|g with their gates, the recurrence, the output
      projection with bias), state updated in place, for each of R distinct
      weight sets totalling >= 1 GiB, from one HIP graph.  value = HBM GB/s of
      algorithmic bytes per step.
  mlgru_prefill -- the MLGRU token mixer over one 2048-token sequence at
      d = 2048.  value = effective TOPS, 2*M*(3d + d)*d.
  train_d1024, train_glu_up -- one training step of the layer: the training
      forward (latent weights ternarised, rstd kept) and the backward (dx, dW,
      db, dgamma) on the paper's training setting (input size and sequence
      length 1024, 16 sequences) or the 1.3B model's GLU up-projection.
      value = effective TOPS, 3 x 2*M*N*K per step.

The JSON line carries the roofline of the dominant kernel (decode: the fused
decode kernel, the only launch of a decode forward; prefill: the contraction),
timed with HIP events on the stream it runs on inside the timed region, with
its HBM traffic per launch when profiles/traffic.json holds a counter reading
of the current kernel source, and the CPU oracle timed on a bounded sample of
the same workload.
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
GLU = ("glu_gate", "channel_mixer")
MLGRU = ("mlgru_decode", "mlgru_prefill")
TRAIN = ("train_d1024", "train_glu_up")
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
ROTATE_BYTES = 1 << 30         # distinct packed weights per decode step


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="large")
    ap.add_argument("--no-secondary", action="store_true",
                    help="only the named workload (no secondary decode leg, no extras)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--hot-cache", action="store_true",
                    help="also time one decode call on cache-resident weights (same kernel, so "
                         "it would skew the kernel's average in a profiler summary)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="finish with a few 256 MiB elementwise copies, the reference kernel "
                         "whose FETCH_SIZE / WRITE_SIZE calibrate the traffic counters")
    ap.add_argument("--record-traffic", nargs=3, metavar=("WORKLOAD", "FETCH_CSV", "WRITE_CSV"),
                    help="no GPU: turn rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE counter CSVs of a "
                         "run with --calib-copy into per-launch HBM traffic in " + "profiles/traffic.json")
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
# HBM traffic per launch, from rocprofv3 counter runs (FETCH_SIZE, WRITE_SIZE)
# ---------------------------------------------------------------------------

TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
CSRC = os.path.join(ROOT, "paper_2406_02528_amd", "csrc")
# the files whose text decides what a kernel does; a recorded traffic figure
# is used only while their digest is unchanged
KERNEL_SOURCES = {
    "decode_kernel": ("decode_impl.h", "decode_bf16.hip", "mmf_device.h"),
    "gemm_kernel": ("gemm.hip", "gemm_common.h", "mmf_device.h"),
}
CALIB_BYTES = 1 << 28          # bytes read and written by one calibration copy


def source_digest(kernel):
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def kernel_key(workload_name, kernel_name):
    """Which recorded kernel a profiled kernel name stands for, or None."""
    if workload_name in DECODE:
        # the fused instance that reads x itself (Src 0 = bf16, 1 = fp32)
        if "decode_kernel<" in kernel_name and ("Src)2" not in kernel_name):
            return "decode_kernel"
        return None
    if "gemm_kernel<" in kernel_name and "Epilogue)0" in kernel_name:
        return "gemm_kernel"
    return None


def read_counter_csv(path, counter):
    import csv
    per = {}
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            if row["Counter_Name"] != counter:
                continue
            per.setdefault(row["Kernel_Name"], []).append(float(row["Counter_Value"]))
    return per


def record_traffic(run_workload, fetch_csv, write_csv):
    """Per-launch HBM bytes of the profiled run's dominant kernels, each counter
    scaled by what it reads for a plain copy of known size (--calib-copy)."""
    fetch = read_counter_csv(fetch_csv, "FETCH_SIZE")
    write = read_counter_csv(write_csv, "WRITE_SIZE")

    def calib(per, what):
        vals = [v for k, vs in per.items() if "neg_kernel" in k for v in vs]
        if not vals:
            raise SystemExit(f"no calibration copy in the {what} run (run it with --calib-copy)")
        kib = sum(vals) / len(vals)
        return kib, CALIB_BYTES / (kib * 1024.0)

    f_kib, f_fac = calib(fetch, "FETCH_SIZE")
    w_kib, w_fac = calib(write, "WRITE_SIZE")
    try:
        with open(TRAFFIC_FILE) as f:
            doc = json.load(f)
    except FileNotFoundError:
        doc = {}
    doc["calibration"] = {
        "kernel": "torch.neg over 2^28 bytes of fp32 (reads and writes 2^28 bytes)",
        "fetch_kib": f_kib, "write_kib": w_kib, "fetch_factor": f_fac, "write_factor": w_fac}
    entries = doc.setdefault("entries", {})
    # the counter runs profile one workload each (--no-secondary)
    workloads_in_run = [run_workload]
    for name, vals in fetch.items():
        for wl in workloads_in_run:
            key = kernel_key(wl, name)
            if key is None or name not in write:
                continue
            fk = sum(vals) / len(vals)
            wk = sum(write[name]) / len(write[name])
            fb, wb = fk * 1024.0 * f_fac, wk * 1024.0 * w_fac
            entries[f"{wl}/{key}"] = {
                "kernel_name": name, "dispatches": len(vals),
                "fetch_kib": fk, "write_kib": wk,
                "fetch_bytes": fb, "write_bytes": wb, "traffic_bytes": fb + wb,
                "source_sha256": source_digest(key)}
            print(f"{wl}/{key}: {len(vals)} dispatches, fetch {fb / 1e6:.3f} MB, "
                  f"write {wb / 1e6:.3f} MB per launch")
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(doc, f, indent=1, sort_keys=True)
        f.write("\n")


def recorded_traffic(workload_name, kernel):
    """(traffic bytes per launch, detail) if recorded for the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            doc = json.load(f)
    except (FileNotFoundError, ValueError):
        return None, None
    e = doc.get("entries", {}).get(f"{workload_name}/{kernel}")
    if not e or e.get("source_sha256") != source_digest(kernel):
        return None, None
    c = doc["calibration"]
    return e["traffic_bytes"], {"fetch_bytes": e["fetch_bytes"], "write_bytes": e["write_bytes"],
                                "fetch_factor": c["fetch_factor"], "write_factor": c["write_factor"]}


def calib_copy(torch):
    """A plain elementwise copy of known size (the counter calibration kernel)."""
    src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


# ---------------------------------------------------------------------------

class Timer:
    """HIP-event timing of `steps` calls after `warmup` untimed ones.  Before
    the warm-up the same work runs for SETTLE_S seconds of wall time: after
    an idle spell the chip's clocks take ~20 launches of the largest GEMM
    (2.1 -> 1.6 ms each, ~35 ms) to reach their sustained level, which a few
    warm-up steps do not cover.  (BENCH_SETTLE_S overrides the 0.25 s, e.g.
    0 for counter-collection runs, whose per-dispatch counts do not depend on
    the clock.)"""
    SETTLE_S = float(os.environ.get("BENCH_SETTLE_S", "0.25"))

    def __init__(self, torch):
        self.torch = torch

    def time(self, fn, steps, warmup):
        import time as _time
        torch = self.torch
        t0 = _time.perf_counter()
        n = 0
        while True:
            fn()
            n += 1
            if n % 4 == 0:
                torch.cuda.synchronize()
                if _time.perf_counter() - t0 >= self.SETTLE_S:
                    break
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

    # context for the launch-bound regime: R launches of one-element torch
    # kernels (the launch floor of a graph), and R plain elementwise copies of
    # each weight copy's packed bytes (reads and writes them once)
    tiny = torch.zeros(1, dtype=torch.int32, device=dev)
    copy_buf = torch.empty_like(Wp0)

    def empty_all():
        for i in range(R):
            tiny.add_(1)

    def copy_all():
        for i in range(R):
            torch.bitwise_not(Wps[i], out=copy_buf)

    graphs = {}
    for name, fn in (("fwd", fwd_all), ("contract", contract_all), ("empty", empty_all),
                     ("copy", copy_all)):
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        graphs[name] = g
    timer = Timer(torch)
    log("[bench] timing the forward graph")
    ms_step = timer.time(graphs["fwd"].replay, args.steps, args.warmup)
    log("[bench] timing the contraction-only graph (pre-quantised q)")
    ms_contract = timer.time(graphs["contract"].replay, args.steps, args.warmup) / R
    ms_empty = timer.time(graphs["empty"].replay, args.steps, args.warmup) / R
    ms_copy = timer.time(graphs["copy"].replay, args.steps, args.warmup) / R
    fb = forward_bytes(w, x.element_size())
    cb = contraction_bytes(w)
    value = R * fb / (ms_step * 1e-3) / 1e9
    # one forward call is one launch of the fused decode kernel, so its average
    # launch duration is the step time over the R launches of the graph
    us_launch = ms_step * 1e3 / R
    achieved = fb / (us_launch * 1e-6) / 1e9
    traffic, tdetail = recorded_traffic(w.name, "decode_kernel")
    result = {
        "value": value, "unit": "GB/s", "ms_per_step": ms_step,
        "config": {"workload": w.name, "M": w.M, "K": w.K, "N": w.N, "x_dtype": w.x_dtype,
                   "weight_copies": R, "calls_per_step": R,
                   "bytes_per_call": fb, "graph": True},
        "roofline": {"bound": "hbm", "kernel": "decode_kernel (fused RMSNorm + int8 quant + "
                                               "ternary GEMV + dequant)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic, "traffic_detail": tdetail,
                     "bytes_per_launch": fb, "avg_launch_us": us_launch},
        "contraction_only": {"avg_launch_us": ms_contract * 1e3, "bytes_per_launch": cb,
                             "GB/s": cb / (ms_contract * 1e-3) / 1e9},
        "launch_floor": {"empty_kernel_us": ms_empty * 1e3,
                         "copy_packed_bytes_us": ms_copy * 1e3,
                         "note": "per launch inside the same kind of graph; torch kernels"},
    }
    if args.hot_cache:
        ms_hot = timer.time(lambda: mmf.mmf_bitlinear_fwd_ws(x, gamma, Wp0, ws0, y, wsb),
                            max(args.steps * 10, 50), args.warmup)
        result["hot_cache_call_us"] = ms_hot * 1e3
    return result, fb


def bench_prefill(torch, mmf, w, args):
    dev, x, gamma, Wp, ws = setup_common(torch, mmf, w)
    log(f"[bench] {w.name}: M={w.M} K={w.K} N={w.N}")
    y = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    wsb = torch.empty(mmf.mmf_bitlinear_workspace_bytes(w.M, w.K), dtype=torch.uint8, device=dev)
    q = torch.empty((w.M, w.K), dtype=torch.int8, device=dev)
    a = torch.empty((w.M,), dtype=torch.float32, device=dev)
    rs = torch.empty((w.M,), dtype=torch.int32, device=dev)
    timer = Timer(torch)
    # value: the forward through its entry point (M > 40: the act-quant launch,
    # then the MFMA contraction with the dequant epilogue)
    ms_step = timer.time(lambda: mmf.mmf_bitlinear_fwd_ws(x, gamma, Wp, ws, y, wsb),
                         args.steps, args.warmup)
    # the roofline: the contraction launch alone, K back-to-back launches between
    # two HIP events on the stream it runs on (events between the forward's two
    # launches would add a cache write-back per event and time that instead)
    mmf.mmf_act_quant_ex(x, gamma, q, a, rs)
    us_gemm = timer.time(lambda: mmf.mmf_ternary_gemm_dequant(q, a, rs, Wp, ws, y),
                         args.steps, args.warmup) * 1e3
    us_aq = timer.time(lambda: mmf.mmf_act_quant_ex(x, gamma, q, a, rs), args.steps, args.warmup) * 1e3
    traffic, tdetail = recorded_traffic(w.name, "gemm_kernel")
    tops = w.ops / (ms_step * 1e-3) / 1e12
    gemm_tops = w.ops / (us_gemm * 1e-6) / 1e12
    aq_bytes = w.M * w.K * x.element_size() + 4 * w.K + w.M * w.K + 8 * w.M
    result = {
        "value": tops, "unit": "TOPS", "ms_per_step": ms_step,
        "config": {"workload": w.name, "M": w.M, "K": w.K, "N": w.N, "x_dtype": w.x_dtype},
        "roofline": {"bound": "mfma", "kernel": "gemm_kernel (prefill contraction, int8 MFMA)",
                     "achieved": gemm_tops, "peak": INT8_PEAK_TOPS, "unit": "TFLOP/s",
                     "frac": gemm_tops / INT8_PEAK_TOPS, "traffic": traffic,
                     "traffic_detail": tdetail,
                     "ops_per_launch": w.ops, "avg_launch_us": us_gemm,
                     "timing": "HIP events around K back-to-back contraction launches on the "
                               "stream they run on"},
        "act_quant": {"avg_launch_us": us_aq, "bytes": aq_bytes,
                      "GB/s": aq_bytes / (us_aq * 1e-6) / 1e9},
        "launches_sum_ms": (us_gemm + us_aq) * 1e-3,
    }
    return result


def bench_glu(torch, mmf, name, args):
    """glu_gate / channel_mixer on the GLU up-projection shape."""
    import workloads
    w = workloads.WORKLOADS["glu_up"]
    L = w.N // 2
    dev, x, gamma, Wp, ws = setup_common(torch, mmf, w)
    Wgu = mmf.glu_pack(Wp[:, :L].contiguous(), Wp[:, L:].contiguous())
    del Wp
    w_scales = torch.cat([ws, ws])
    log(f"[bench] {name}: M={w.M} K={w.K} L={L}")
    p = torch.empty((w.M, L), dtype=torch.float32, device=dev)
    wsb = torch.empty(mmf.mmf_bitlinear_workspace_bytes(w.M, w.K), dtype=torch.uint8, device=dev)
    q = torch.empty((w.M, w.K), dtype=torch.int8, device=dev)
    a = torch.empty((w.M,), dtype=torch.float32, device=dev)
    rs = torch.empty((w.M,), dtype=torch.int32, device=dev)
    mmf.mmf_act_quant(x, gamma, q, a, rs)
    ops_glu = 2 * w.M * w.N * w.K
    config = {"workload": name, "M": w.M, "K": w.K, "L": L, "x_dtype": w.x_dtype}
    if name == "glu_gate":
        def step():
            mmf.mmf_glu_fwd_ws(x, gamma, Wgu, w_scales, p, wsb)
        ops = ops_glu
    else:
        wd = workloads.WORKLOADS["glu_down"]
        Wdp, wsd = mmf.ternarize(torch.from_numpy(workloads.make_w(wd)).to(dev))
        gd = torch.from_numpy(workloads.make_gamma(wd)).to(dev)
        y = torch.empty((w.M, wd.N), dtype=torch.float32, device=dev)
        wsb2 = torch.empty(mmf.mmf_bitlinear_workspace_bytes(w.M, L), dtype=torch.uint8, device=dev)

        def step():
            mmf.mmf_glu_fwd_ws(x, gamma, Wgu, w_scales, p, wsb)
            mmf.mmf_bitlinear_fwd_ws(p, gd, Wdp, wsd, y, wsb2)
        ops = ops_glu + 2 * w.M * wd.N * L
        config.update({"N_down": wd.N})
    timer = Timer(torch)
    ms_step = timer.time(step, args.steps, args.warmup)
    ms_gemm = timer.time(lambda: mmf.mmf_ternary_gemm_glu(q, a, rs, Wgu, w_scales, p),
                         args.steps, args.warmup)
    gemm_tops = ops_glu / (ms_gemm * 1e-3) / 1e12
    return {
        "value": ops / (ms_step * 1e-3) / 1e12, "unit": "TOPS", "ms_per_step": ms_step,
        "config": config,
        "roofline": {"bound": "mfma", "kernel": "gemm_kernel with the GLU epilogue "
                                                 "(gate|up contraction + SiLU(g) * u)",
                     "achieved": gemm_tops, "peak": INT8_PEAK_TOPS, "unit": "TFLOP/s",
                     "frac": gemm_tops / INT8_PEAK_TOPS, "traffic": None,
                     "ops_per_launch": ops_glu, "avg_launch_us": ms_gemm * 1e3},
    }, ops


def mlgru_bytes(B, T, d):
    """Algorithmic bytes of one MLGRU mixer call: (projection, recurrence,
    output projection).  Projection: x (bf16), gamma, packed f|c|g weights,
    w_scales, biases, lower bound, fcg written.  Recurrence: fcg read, state
    read and written, o' written.  Output projection: o' read, gamma_o,
    packed W_o, w_scale, b_o, o written."""
    M = B * T
    proj = M * d * 2 + 4 * d + (d // 16) * 3 * d * 4 + 12 + 4 * 3 * d + 4 * d + 4 * M * 3 * d
    scan = 4 * M * 3 * d + 2 * 4 * B * d + 4 * M * d
    oproj = 4 * M * d + 4 * d + (d // 16) * d * 4 + 4 + 4 * d + 4 * M * d
    return proj, scan, oproj


def mlgru_setup(torch, mmf, w, copies=1):
    """Device inputs of an MLGRU workload; `copies` distinct weight sets (the
    first the seeded one, the others drawn on the device)."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    inp = workloads.make_mlgru(w)
    T_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    x = torch.from_numpy(inp["x_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
    sets = []
    gen = torch.Generator(device=dev)
    gen.manual_seed(240602528)
    for i in range(copies):
        if i == 0:
            Wf, Wo = T_(inp["W_fcg"]), T_(inp["W_o"])
        else:
            Wf = torch.randn((3 * w.d, w.d), generator=gen, device=dev) * 0.02
            Wo = torch.randn((w.d, w.d), generator=gen, device=dev) * 0.02
        Wfp, wsf = mmf.ternarize(Wf)
        Wop, wso = mmf.ternarize(Wo)
        sets.append((Wfp, torch.cat([wsf, wsf, wsf]), Wop, wso))
        del Wf, Wo
    return {"dev": dev, "x": x, "gamma": T_(inp["gamma"]), "gamma_o": T_(inp["gamma_o"]),
            "bias": T_(inp["bias"]), "b_o": T_(inp["b_o"]), "lb": T_(inp["lb"]),
            "h": T_(inp["h0"]), "sets": sets}


def bench_mlgru(torch, mmf, name, args):
    import workloads
    w = workloads.MLGRU_WORKLOADS[name]
    M, d = w.M, w.d
    pb, sb, ob = mlgru_bytes(w.B, w.T, d)
    timer = Timer(torch)
    if name == "mlgru_decode":
        R = max(1, math.ceil(ROTATE_BYTES / ((d // 16) * 4 * d * 4)))
        log(f"[bench] {name}: B={w.B} T={w.T} d={d}, {R} weight sets")
        st = mlgru_setup(torch, mmf, w, R)
    else:
        R = 1
        log(f"[bench] {name}: B={w.B} T={w.T} d={d}")
        st = mlgru_setup(torch, mmf, w, 1)
    dev, x, h = st["dev"], st["x"], st["h"]
    o = torch.empty((M, d), dtype=torch.float32, device=dev)
    wsb = torch.empty(mmf.mmf_mlgru_workspace_bytes(w.B, w.T, d), dtype=torch.uint8, device=dev)
    fcg = torch.empty((M, 3 * d), dtype=torch.float32, device=dev)
    op = torch.empty((M, d), dtype=torch.float32, device=dev)
    h_out = torch.empty_like(h)
    pws = torch.empty(mmf.mmf_mlgru_proj_workspace_bytes(M, d, d), dtype=torch.uint8, device=dev)
    sws = torch.empty(max(1, mmf.mmf_mlgru_scan_workspace_bytes(w.B, w.T, d)), dtype=torch.uint8,
                      device=dev)
    sws_arg = sws if mmf.mmf_mlgru_scan_workspace_bytes(w.B, w.T, d) else None

    # the state alternates between two arrays (the decode step then runs the
    # recurrence inside the output projection); a prefill carries it in place
    h_alt = h.clone()

    def mixer(i):
        Wfp, wsf, Wop, wso = st["sets"][i]
        h_in, h_new = (h, h_alt) if (w.T == 1 and i % 2 == 0) else ((h_alt, h) if w.T == 1 else (h, h))
        mmf.mmf_mlgru_fwd(x, w.B, w.T, st["gamma"], Wfp, wsf, st["bias"], st["lb"], h_in, h_new,
                          st["gamma_o"], Wop, wso, st["b_o"], o, wsb)

    def proj(i):
        Wfp, wsf, _, _ = st["sets"][i]
        mmf.mmf_mlgru_proj(x, st["gamma"], Wfp, wsf, st["bias"], st["lb"], fcg, pws)

    def scan(i):
        mmf.mmf_mlgru_scan(fcg, w.B, w.T, h, op, h_out, sws_arg)

    def oproj(i):
        _, _, Wop, wso = st["sets"][i]
        mmf.mmf_bitlinear_fwd_bias(op, st["gamma_o"], Wop, wso, st["b_o"], o)

    proj(0)
    scan(0)
    torch.cuda.synchronize()
    stages = {}
    if name == "mlgru_decode":
        graphs = {}
        for key, fn in (("mixer", mixer), ("proj", proj), ("scan", scan), ("oproj", oproj)):
            for i in range(R):
                fn(i)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(R):
                    fn(i)
            graphs[key] = g
        log("[bench] timing the mixer graph")
        ms_step = timer.time(graphs["mixer"].replay, args.steps, args.warmup)
        for key in ("proj", "scan", "oproj"):
            stages[key] = timer.time(graphs[key].replay, args.steps, args.warmup) * 1e3 / R
        step_bytes = pb + sb + ob
        value = R * step_bytes / (ms_step * 1e-3) / 1e9
        us_proj = stages["proj"]
        achieved = pb / (us_proj * 1e-6) / 1e9
        roof = {"bound": "hbm", "kernel": "decode_kernel with the MLGRU gate epilogue "
                                          "(f|c|g projection + bias + sigmoid/SiLU)",
                "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                "bytes_per_launch": pb, "avg_launch_us": us_proj}
        res = {"value": value, "unit": "GB/s", "ms_per_step": ms_step}
        extra = {"token_steps_per_graph": R, "us_per_token_step": ms_step * 1e3 / R,
                 "bytes_per_token_step": step_bytes}
    else:
        q = torch.empty((M, d), dtype=torch.int8, device=dev)
        a = torch.empty((M,), dtype=torch.float32, device=dev)
        rsum = torch.empty((M,), dtype=torch.int32, device=dev)
        mmf.mmf_act_quant(x, st["gamma"], q, a, rsum)
        Wfp, wsf, _, _ = st["sets"][0]
        ms_step = timer.time(lambda: mixer(0), args.steps, args.warmup)
        ms_gemm = timer.time(lambda: mmf.mmf_mlgru_proj_q(q, a, rsum, Wfp, wsf, st["bias"],
                                                          st["lb"], fcg), args.steps, args.warmup)
        for key, fn in (("proj", proj), ("scan", scan), ("oproj", oproj)):
            stages[key] = timer.time(lambda: fn(0), args.steps, args.warmup) * 1e3
        ops_proj = 2 * M * 3 * d * d
        gemm_tops = ops_proj / (ms_gemm * 1e-3) / 1e12
        res = {"value": w.ops / (ms_step * 1e-3) / 1e12, "unit": "TOPS", "ms_per_step": ms_step}
        roof = {"bound": "mfma", "kernel": "gemm_kernel with the MLGRU gate epilogue "
                                           "(f|c|g contraction + bias + sigmoid/SiLU)",
                "achieved": gemm_tops, "peak": INT8_PEAK_TOPS, "unit": "TFLOP/s",
                "frac": gemm_tops / INT8_PEAK_TOPS, "traffic": None,
                "ops_per_launch": ops_proj, "avg_launch_us": ms_gemm * 1e3}
        extra = {"tokens_per_s": M / (ms_step * 1e-3)}
    res["config"] = {"workload": name, "B": w.B, "T": w.T, "d": d, "x_dtype": "bf16", **extra}
    res["roofline"] = roof
    res["stages"] = {
        "proj_us": stages["proj"], "scan_us": stages["scan"], "oproj_us": stages["oproj"],
        "scan_bytes": sb, "scan_GB/s": sb / (stages["scan"] * 1e-6) / 1e9,
        "scan_frac_hbm": sb / (stages["scan"] * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "note": "per call, each stage timed alone (decode: inside a graph of R calls)"}
    return res, (pb + sb + ob)


def cpu_baseline_mlgru(name, step_bytes, seconds):
    """The oracle's whole mixer: decode, repeated token steps of the same
    workload (GB/s with the GPU's byte count); prefill, a prefix of the
    sequence grown until it fills a quarter of the budget (effective TOPS)."""
    import oracle
    import workloads
    w = workloads.MLGRU_WORKLOADS[name]
    inp = workloads.make_mlgru(w)
    t, ws = oracle.weight_quant(inp["W_fcg"])
    t_o, ws_o = oracle.weight_quant(inp["W_o"])

    def run(T):
        return oracle.mlgru_fwd(inp["x_f32"][:w.B * T], w.B, T, inp["gamma"], t, [ws] * 3,
                                inp["bias"], inp["lb"], inp["h0"], inp["gamma_o"], t_o, ws_o,
                                inp["b_o"])

    if name == "mlgru_decode":
        calls = 0
        t0 = time.perf_counter()
        while True:
            run(1)
            calls += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                break
        return {"value": calls * step_bytes / el / 1e9, "unit": "GB/s", "cores": oracle.num_threads(),
                "kind": "oracle",
                "sample": f"{calls} token steps (B={w.B}, d={w.d}) in {el:.1f} s; bytes counted as "
                          "for the GPU"}
    T = 8
    while True:
        t0 = time.perf_counter()
        run(T)
        el = time.perf_counter() - t0
        if el >= seconds / 4 or T >= w.T:
            break
        T = min(w.T, T * max(2, int(seconds / 4 / max(el, 1e-3))))
    return {"value": 2.0 * w.B * T * 4 * w.d * w.d / el / 1e12, "unit": "TOPS",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"the first {T} of {w.T} tokens (B={w.B}, d={w.d}) in {el:.1f} s"}


def bench_train(torch, mmf, name, args):
    import numpy as np
    import workloads
    w = workloads.TRAIN_WORKLOADS[name]
    M, K, N = w.M, w.K, w.N
    log(f"[bench] {name}: M={M} K={K} N={N}")
    inp = workloads.make_train(w)
    dev = torch.device("cuda:0")
    T_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    x = torch.from_numpy(inp["x_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
    dO = torch.from_numpy(inp["dO_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
    gamma, W = T_(inp["gamma"]), T_(inp["W"])
    del inp
    y = torch.empty((M, N), dtype=torch.float32, device=dev)
    Wp = torch.empty((K // 16, N), dtype=torch.int32, device=dev)
    ws = torch.empty((1,), dtype=torch.float32, device=dev)
    q = torch.empty((M, K), dtype=torch.int8, device=dev)
    a = torch.empty((M,), dtype=torch.float32, device=dev)
    r = torch.empty((M,), dtype=torch.float32, device=dev)
    dx = torch.empty((M, K), dtype=torch.float32, device=dev)
    dW = torch.empty((N, K), dtype=torch.float32, device=dev)
    db = torch.empty((N,), dtype=torch.float32, device=dev)
    dg = torch.empty((K,), dtype=torch.float32, device=dev)
    wsf = torch.empty(mmf.mmf_bitlinear_train_workspace_bytes(M, K, N), dtype=torch.uint8, device=dev)
    wsb = torch.empty(mmf.mmf_bitlinear_bwd_workspace_bytes(M, K, N), dtype=torch.uint8, device=dev)

    def fwd():
        mmf.mmf_bitlinear_train_fwd(x, gamma, W, None, y, Wp, ws, q, a, r, wsf)

    def bwd():
        mmf.mmf_bitlinear_bwd(dO, x, gamma, r, q, a, Wp, ws, dx, dW, db, dg, wsb)

    def step():
        fwd()
        bwd()

    timer = Timer(torch)
    ms_step = timer.time(step, args.steps, args.warmup)
    ms_fwd = timer.time(fwd, args.steps, args.warmup)
    ms_bwd = timer.time(bwd, args.steps, args.warmup)
    mnk2 = 2.0 * M * N * K
    bwd_tflops = 2 * mnk2 / (ms_bwd * 1e-3) / 1e12
    return {
        "value": w.ops / (ms_step * 1e-3) / 1e12, "unit": "TOPS", "ms_per_step": ms_step,
        "config": {"workload": name, "M": M, "K": K, "N": N, "x_dtype": "bf16", "dO_dtype": "bf16",
                   "fwd_us": ms_fwd * 1e3, "bwd_us": ms_bwd * 1e3},
        "roofline": {"bound": "mfma", "kernel": "backward: the dY and dW bf16 MFMA kernels (fp32 "
                                                "accumulation; codes and q expanded in the kernels) "
                                                "with the code re-pack, the RMSNorm-backward finish "
                                                "and the column sums, timed as one call",
                     "achieved": bwd_tflops, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": bwd_tflops / BF16_PEAK_TFLOPS, "traffic": None,
                     "flops_per_launch": 2 * mnk2, "avg_launch_us": ms_bwd * 1e3},
        "forward": {"avg_call_us": ms_fwd * 1e3, "int8_TOPS": mnk2 / (ms_fwd * 1e-3) / 1e12,
                    "note": "ternarisation of the latent weights + act-quant + int8 MFMA contraction"},
    }


def cpu_baseline_train(name, seconds):
    """The oracle's training forward and backward on a sample of token rows
    over all K and N, in effective TOPS (3 x 2 rows N K)."""
    import oracle
    import workloads
    w = workloads.TRAIN_WORKLOADS[name]
    inp = workloads.make_train(w)
    dO = workloads.bf16_bits_to_f32(inp["dO_bits"])
    rows = 4
    while True:
        t0 = time.perf_counter()
        f = oracle.bitlinear_train_fwd(inp["x_f32"][:rows], inp["gamma"], inp["W"])
        oracle.bitlinear_bwd(dO[:rows], inp["x_f32"][:rows], inp["gamma"], f["rstd"], f["q"],
                             f["a_scale"], f["t"], f["w_scale"])
        el = time.perf_counter() - t0
        if el >= seconds / 4 or rows >= w.M:
            break
        rows = min(w.M, rows * max(2, int(seconds / 4 / max(el, 1e-3))))
    return {"value": 6.0 * rows * w.N * w.K / el / 1e12, "unit": "TOPS", "cores": oracle.num_threads(),
            "kind": "oracle", "sample": f"{rows} of {w.M} token rows (K={w.K}, N={w.N}), forward and "
                                        f"backward, in {el:.1f} s"}


def cpu_baseline_glu(name, seconds):
    """The oracle (two BitLinears, the gate; for channel_mixer also the down
    projection) on a sample of token rows, in effective TOPS."""
    import oracle
    import workloads
    w = workloads.WORKLOADS["glu_up"]
    L = w.N // 2
    _, xf = workloads.make_x(w)
    g = workloads.make_gamma(w)
    t, ws = oracle.weight_quant(workloads.make_w(w))
    t_g, t_u = t[:L], t[L:]
    down = None
    if name == "channel_mixer":
        wd = workloads.WORKLOADS["glu_down"]
        td, wsd = oracle.weight_quant(workloads.make_w(wd))
        down = (td, wsd, workloads.make_gamma(wd), wd.N)
    rows = 4
    while True:
        t0 = time.perf_counter()
        pr = oracle.glu_fwd(xf[:rows], g, t_g, ws, t_u, ws)["p"]
        if down is not None:
            oracle.bitlinear_fwd(pr, down[2], down[0], down[1])
        el = time.perf_counter() - t0
        if el >= seconds / 4 or rows >= w.M:
            break
        rows = min(w.M, rows * max(2, int(seconds / 4 / max(el, 1e-3))))
    ops = 2.0 * rows * w.N * w.K + (2.0 * rows * down[3] * L if down else 0.0)
    return {"value": ops / el / 1e12, "unit": "TOPS", "cores": oracle.num_threads(),
            "kind": "oracle", "sample": f"{rows} of {w.M} token rows in {el:.1f} s"}


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
    # prefill: a row sample over all N, timed once, grown (from the rate of the
    # previous sample) until one sample takes at least half the budget
    rows = 8
    while True:
        t0 = time.perf_counter()
        oracle.bitlinear_fwd(xf[:rows], g, t, ws)
        el = time.perf_counter() - t0
        if el >= seconds / 2 or rows >= w.M:
            break
        rows = min(w.M, max(2 * rows, int(rows * 0.8 * seconds / max(el, 1e-3))))
    return {"value": 2.0 * rows * w.N * w.K / el / 1e12, "unit": "TOPS", "cores": threads,
            "kind": "oracle",
            "sample": f"{rows} of {w.M} token rows (K={w.K}, N={w.N}) in {el:.1f} s"}


def main():
    args = parse()
    if args.record_traffic:
        record_traffic(*args.record_traffic)
        return
    check_single_gpu(args)
    import torch
    import paper_2406_02528_amd as mmf
    import workloads
    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    w = None if args.workload in GLU + MLGRU + TRAIN else workloads.WORKLOADS[args.workload]
    if args.workload in MLGRU:
        res, fb = bench_mlgru(torch, mmf, args.workload, args)
    elif args.workload in TRAIN:
        res, fb = bench_train(torch, mmf, args.workload, args), None
    elif w is None:
        res, _ = bench_glu(torch, mmf, args.workload, args)
        fb = None
    elif w.name in DECODE:
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
    for k in ("hot_cache_call_us", "act_quant", "contraction_only", "launch_floor", "stages", "forward",
              "launches_sum_ms"):
        if k in res:
            line[k] = res[k]
    headline = args.workload == "large" and not args.no_secondary
    if headline:
        # the metric's decode half on the same configuration family (d = 5120)
        dw = workloads.WORKLOADS["large_dec"]
        log("[bench] secondary: large_dec decode")
        torch.cuda.empty_cache()
        sec, sec_fb = bench_decode(torch, mmf, dw, args)
        line["secondary"] = {"metric": "decode HBM GB/s", **{k: sec[k] for k in (
            "value", "unit", "ms_per_step", "config", "roofline", "contraction_only", "launch_floor")}}
        torch.cuda.empty_cache()
        extra = {}
        for name in ("decode_m1", "glu_up"):
            ew = workloads.WORKLOADS[name]
            log(f"[bench] extra: {name}")
            if name in DECODE:
                er, _ = bench_decode(torch, mmf, ew, args)
            else:
                er = bench_prefill(torch, mmf, ew, args)
            extra[name] = {k: er[k] for k in ("value", "unit", "ms_per_step", "config", "roofline")}
            torch.cuda.empty_cache()
        line["extra"] = extra
    if args.calib_copy:
        log("[bench] calibration copy")
        calib_copy(torch)
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        if args.workload in MLGRU:
            line["cpu_baseline"] = cpu_baseline_mlgru(args.workload, fb, args.cpu_seconds)
        elif args.workload in TRAIN:
            line["cpu_baseline"] = cpu_baseline_train(args.workload, args.cpu_seconds)
        elif w is None:
            line["cpu_baseline"] = cpu_baseline_glu(args.workload, args.cpu_seconds)
        else:
            line["cpu_baseline"] = cpu_baseline(w, fb, args.cpu_seconds)
        if headline:
            line["secondary"]["cpu_baseline"] = cpu_baseline(workloads.WORKLOADS["large_dec"], sec_fb,
                                                             args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
