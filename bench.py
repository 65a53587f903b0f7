#!/usr/bin/env python3
"""Benchmark of the KroQuant online activation quantizer on one MI355X.

One step = one kq_quantize_packed call (Kronecker block transform (A (x) B)
with A 4x4, B 8x8 shared by every block, then MXFP4) over the
FLUX.1-schnell-shaped activation X bf16 [4608, 3072] (Student-t(3), 0.5%
outlier channels x50).  The packed call is the K1 variant of the paper: the
materialised K = A (x) B (split for the matrix cores) is produced once per
layer by kq_pack_factors, outside the timed region, like the layer's weights;
the transform itself runs on every activation inside it.  The on-the-fly
variant (K2, kq_quantize) and the fixed-order VALU variant are timed too.

* Inputs are resident in HBM before the timed region.  The step rotates over
  enough distinct input/output buffer sets that their footprint exceeds twice
  the 256 MB last-level (MALL) cache, so every step streams from HBM.
* Time: after W warmup steps, exactly K back-to-back steps are captured into a
  HIP graph (outside the timed region) behind W more warmup launches and
  between two stamps of the device's 100 MHz real-time counter
  (kq_timestamp); the graph is replayed once between synchronizations and the
  stamp difference times exactly the K launches (HIP events around the whole
  replay, which also hold the fixed cost of launching a graph, are reported
  beside it); value = algorithmic bytes (2 B bf16 in +
  0.5 B codes + 1/32 B scale per element) / time per step.  One Python-side
  launch through ctypes costs about as much host time as the whole kernel
  (~7 us), so the same K launches from the Python loop are reported beside it
  (eager_python) rather than as the value.
* The comparators (SmoothQuant, Hadamard-32, plain MXFP4) run on identical
  inputs with the same protocol; their times go in the same JSON line.
* The outputs of the timed configuration are checked against the CPU oracle.
* The oracle itself is timed on this host as a reported CPU baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "quantizer GB/s and % HBM peak (bf16→MXFP4), M×d=4608×3072; vs SmoothQuant time"
WORKLOAD = "flux_4608x3072"
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E peak, GB/s
MALL_BYTES = 256 * 1024 * 1024   # MI355X Infinity Cache
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_flux_4608x3072.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2607_21446_amd", "csrc", f)
                  for f in ("kq_kernels.hip", "kq_kernels.h", "kq_api.hip")]


def algorithmic_bytes(M, d):
    return 2 * M * d + M * d // 2 + M * d // 32


def kernel_source_hash():
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # defaults: about 20 ms of warmup, enough for the clocks to settle after
    # the host-side setup (a 100-step warmup times ~9% slow), then 1000 steps
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=2000)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--only", choices=["kroquant", "kroquant_onthefly", "kroquant_lu", "kroquant_exact", "smoothquant",
                                       "hadamard32", "mxfp4", "stream_floor", "copy", "calib", "gemm", "gemm_vendor"],
                    help="run only this kernel for --steps launches (for profiler runs); prints no JSON "
                         "(calib: only the calibration timing, printed as JSON; gemm: the W4A4 product of the "
                         "headline activation with a 3072 x 3072 weight; gemm_vendor: that product with a bf16 "
                         "output, then the vendor's MXFP4 GEMM on the same operands)")
    ap.add_argument("--summarize-pmc", metavar="DIR",
                    help="turn the FETCH_SIZE / WRITE_SIZE counter runs under DIR (DIR/<kernel>/p3, p4 from "
                         "rocprofv3 --pmc, kernels 'kroquant' and 'copy') into the traffic record read by the "
                         "roofline field; needs no GPU")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="summarize a rocprofv3 --kernel-trace run under DIR (per kernel and grid: calls and duration "
                         "statistics, and for every group of at least 4000 launches the windows of dispatches "
                         "2001-3000 and 3001-4000, the headline's first and timed graph replays); needs no GPU")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true")
    ap.add_argument("--no-gemm", action="store_true", help="skip the W4A4 MXFP4 GEMM consumer timing")
    ap.add_argument("--no-calib", action="store_true", help="skip the layer-wise calibration timing")
    ap.add_argument("--calib-samples", type=int, default=128,
                    help="calibration samples of 4608 tokens for the calibration timing")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload table (every DiT shape, the one-GPU shard and the large per-block "
                         "stress shape; KroQuant variants and comparators)")
    ap.add_argument("--configs", default=",".join(CONFIG_WORKLOADS),
                    help="comma-separated workloads of the table (default: all)")
    ap.add_argument("--no-table2", action="store_true",
                    help="skip the paper's Table 2 (power-of-two d: Q4, Scale, K1, K2, FWHT) and Table 4 (production "
                         "shapes: Q4, Scale, K1, K2) comparisons")
    return ap.parse_args()


KERNEL_NAMES = {"kroquant": "kron_mfma_unit_kernel", "copy": "copyBuffer", "stream_floor": "stream_floor_kernel"}
COPY_BYTES = 1 << 28  # the --only copy kernel moves 256 MiB in and 256 MiB out


def _counter_median(root, kernel, counter):
    import csv
    import glob
    import statistics
    vals = []
    for f in glob.glob(os.path.join(root, kernel, "p*", "*counter_collection.csv")):
        with open(f) as fh:
            for row in csv.DictReader(fh):
                if row["Counter_Name"] == counter and KERNEL_NAMES[kernel] in row["Kernel_Name"]:
                    vals.append(float(row["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} samples for {kernel} under {root}")
    return statistics.median(vals), len(vals)


def summarize_pmc(root, workload):
    """HBM traffic of one hot-path launch: FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch) of the kernel, each divided by what the same counter reads per
    byte for a plain 256 MiB copy."""
    k_fetch, n1 = _counter_median(root, "kroquant", "FETCH_SIZE")
    k_write, n2 = _counter_median(root, "kroquant", "WRITE_SIZE")
    c_fetch, _ = _counter_median(root, "copy", "FETCH_SIZE")
    c_write, _ = _counter_median(root, "copy", "WRITE_SIZE")
    f_read = c_fetch * 1024 / COPY_BYTES   # counter bytes per real byte read
    f_write = c_write * 1024 / COPY_BYTES  # counter bytes per real byte written
    read_b = k_fetch * 1024 / f_read
    write_b = k_write * 1024 / f_write
    from synth import WORKLOADS
    _, M, d = WORKLOADS[workload][:3]
    rec = {"workload": workload, "kernel": KERNEL_NAMES["kroquant"], "kernel_source_hash": kernel_source_hash(),
           "fetch_kib_per_dispatch": k_fetch, "write_kib_per_dispatch": k_write, "dispatches": min(n1, n2),
           "copy_fetch_factor": f_read, "copy_write_factor": f_write,
           "hbm_read_bytes_per_launch": read_b, "hbm_write_bytes_per_launch": write_b,
           "hbm_bytes_per_launch": read_b + write_b, "algorithmic_bytes": algorithmic_bytes(M, d)}
    if os.path.isdir(os.path.join(root, "stream_floor")):
        # the traffic-only kernel on the same workload, for comparison
        s_fetch, _ = _counter_median(root, "stream_floor", "FETCH_SIZE")
        s_write, _ = _counter_median(root, "stream_floor", "WRITE_SIZE")
        rec["stream_floor_hbm_bytes_per_launch"] = s_fetch * 1024 / f_read + s_write * 1024 / f_write
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec, indent=1))


def summarize_trace(root, warmup, steps):
    """Kernel durations from a rocprofv3 kernel trace, grouped by kernel name
    and grid size, in launch order (markdown on stdout)."""
    import csv
    import glob
    import statistics
    rows = []
    for f in glob.glob(os.path.join(root, "**", "*kernel_trace.csv"), recursive=True):
        with open(f) as fh:
            rows.extend(csv.DictReader(fh))
    if not rows:
        raise SystemExit(f"no kernel trace under {root}")
    gcol = [c for c in rows[0] if c.startswith("Grid_Size")]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    groups = {}
    for r in rows:
        key = (r["Kernel_Name"], "x".join(r[c] for c in gcol))
        groups.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0)

    def stats(v):
        s = sorted(v)
        q = lambda p: s[min(len(s) - 1, int(p * len(s)))]
        return f"{statistics.mean(v):.3f} | {statistics.median(v):.3f} | {q(0.1):.3f} | {q(0.9):.3f}"

    print(f"{len(rows)} dispatches\n")
    print("| kernel | grid (work-items) | calls | mean us | median us | p10 | p90 |\n|---|---|---|---|---|---|---|")
    for (k, grid), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{k}` | {grid} | {len(v)} | {stats(v)} |")
    # launch order of a timed measurement: W eager warmup launches, then the graph (W warmup launches, the K
    # timed ones) replayed twice -- an untimed upload, then the timed replay
    W, K = warmup, steps
    wins = ((2 * W + 1, 2 * W + K, "upload replay"), (3 * W + K + 1, 3 * W + 2 * K, "timed replay"))
    print(f"\nwindows (launch order within a kernel and grid; W = {W}, K = {K}):\n")
    for (k, grid), v in groups.items():
        if len(v) >= 3 * W + 2 * K:
            for a, b, what in wins:
                print(f"- `{k}` grid {grid}, launches {a}-{b} ({what}): mean | median | p10 | p90 = "
                      f"{stats(v[a - 1:b])} us")


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc, args.workload)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.warmup, args.steps)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this quantizer benchmark runs on exactly one GPU (--gpus 1); the quantizer "
              "has no cross-GPU step, and runs on more than one GPU are not supported", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2607_21446_amd as kq
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    kq.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.only == "copy":
        # plain copy of a known size (256 MiB read + 256 MiB written), for counter calibration; nothing
        # else is dispatched in this mode, so every copy kernel the profiler sees is this one
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"ran copy x{args.steps}", flush=True)
        return
    if args.only == "calib":
        stream = torch.cuda.current_stream()
        print(json.dumps(calib_timing(kq, synth, dev, stream, stream.cuda_stream, args.calib_samples)), flush=True)
        return

    w = synth.workload(args.workload)
    M, d = w.X.shape
    nbytes = algorithmic_bytes(M, d)
    set_bytes = nbytes
    nsets = max(2, int(np.ceil(2 * MALL_BYTES / set_bytes)) + 1)

    X0 = torch.from_numpy(w.X.view(np.int16)).view(torch.bfloat16).to(dev)
    A = torch.from_numpy(w.A).to(dev)
    B = torch.from_numpy(w.B).to(dev)
    mult = torch.from_numpy(w.mult).to(dev)
    Xs = [X0.clone() for _ in range(nsets)]
    Cs = [torch.empty((M, d // 2), dtype=torch.uint8, device=dev) for _ in range(nsets)]
    Ss = [torch.empty((M, d // 32), dtype=torch.uint8, device=dev) for _ in range(nsets)]
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream

    kpack = kq.pack_factors(A, B, stream=sptr)  # offline, once per layer
    lu = torch.from_numpy(synth.lu_params(1, seed=7)).to(dev)  # K2-form factors (15 parameters)

    def run_kq(i):
        kq.quantize_packed(Xs[i], A, B, kpack, codes=Cs[i], scales=Ss[i])

    def run_k2(i):
        kq.quantize(Xs[i], A, B, codes=Cs[i], scales=Ss[i])

    def run_kx(i):
        kq.quantize_exact(Xs[i], A, B, codes=Cs[i], scales=Ss[i])

    def run_lu(i):
        kq.quantize_lu(Xs[i], lu, 4, codes=Cs[i], scales=Ss[i])

    def run_sq(i):
        kq.smoothquant(Xs[i], mult, codes=Cs[i], scales=Ss[i])

    def run_h32(i):
        kq.hadamard32(Xs[i], codes=Cs[i], scales=Ss[i])

    def run_q4(i):
        kq.mxfp4(Xs[i], codes=Cs[i], scales=Ss[i])

    def run_floor(i):
        kq.stream_floor(Xs[i], out16=Cs[i], out1=Ss[i])

    runs = {"kroquant": run_kq, "kroquant_onthefly": run_k2, "kroquant_lu": run_lu, "kroquant_exact": run_kx,
            "smoothquant": run_sq,
            "hadamard32": run_h32, "mxfp4": run_q4, "stream_floor": run_floor}

    if args.only in ("gemm", "gemm_vendor"):
        A_, B_ = synth.factors(4, 8, 1, seed=5)
        Wg = synth.activations(3072, d, "normal", seed=3072, chan_frac=0.0)
        Wgd = torch.from_numpy(Wg.view(np.int16)).view(torch.bfloat16).to(dev)
        _, wc, wsc = kq.weight_transform(Wgd, torch.from_numpy(A_), torch.from_numpy(B_))
        run_kq(0)
        if args.only == "gemm":
            Cg = torch.empty((M, 3072), dtype=torch.float32, device=dev)
            for i in range(args.steps):
                kq.mxfp4_gemm(Cs[0], Ss[0], wc, wsc, C=Cg, stream=sptr)
        else:
            # the bf16-output product, then the vendor's MXFP4 GEMM on the same codes and scales
            C16 = torch.empty((M, 3072), dtype=torch.bfloat16, device=dev)
            for i in range(args.steps):
                kq.mxfp4_gemm(Cs[0], Ss[0], wc, wsc, C=C16, stream=sptr)
            a, b = Cs[0].view(torch.float4_e2m1fn_x2), wc.view(torch.float4_e2m1fn_x2)
            sa, sb = Ss[0].view(torch.float8_e8m0fnu), wsc.view(torch.float8_e8m0fnu)
            with torch.cuda.stream(stream):
                for i in range(args.steps):
                    torch._scaled_mm(a, b.t(), scale_a=sa, scale_b=sb, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        print(f"ran {args.only} x{args.steps} ({M} x 3072 x {d})", flush=True)
        return
    if args.only:
        if args.only in ("copy", "calib"):
            raise AssertionError("handled before the workload setup")
        else:
            fn = runs[args.only]
            for i in range(args.steps):
                fn(i % nsets)
        torch.cuda.synchronize()
        print(f"ran {args.only} x{args.steps} on {args.workload}", flush=True)
        return

    def timed_eager(fn, steps, warmup, rotate=True):
        """K launches from the Python loop (each a ctypes call, ~7 us of host
        time), HIP events on the launch stream around them."""
        for i in range(warmup):
            fn(i % nsets if rotate else 0)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for i in range(steps):
            fn(i % nsets if rotate else 0)
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return e0.elapsed_time(e1) / steps, wall

    stamps = torch.zeros(2, dtype=torch.int64, device=dev)
    replay_us = {}

    def timed(fn, steps, warmup, rotate=True, name=None):
        """K launches captured into a HIP graph, behind W warmup launches and
        between two device stamps of the 100 MHz real-time counter
        (kq_timestamp).  The graph is captured first, then the W warmup steps
        run eagerly, the graph is replayed once untimed (the first replay
        uploads it) and once more, timed, all queued back to back with one
        torch.cuda.synchronize() at the end, so the GPU does not idle between
        the warmup and the timed launches.  The time per step is the stamp
        difference of the second replay over K: exactly the K back-to-back
        launches, without the host's per-call cost and without the fixed cost
        of launching the graph (which, spread over a short K, would read as a
        slower step).  HIP events around the timed replay (its warmup launches
        and the graph launch included) are kept beside it in `replay_us`."""
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(warmup):
                fn((steps + i) % nsets if rotate else 0)
            kq.timestamp(stamps, 0)
            for i in range(steps):
                fn(i % nsets if rotate else 0)
            kq.timestamp(stamps, 1)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        for i in range(warmup):
            fn(i % nsets if rotate else 0)
        g.replay()  # untimed: the first replay uploads the graph
        e0.record(stream)
        t0 = time.perf_counter()  # host wall clock from queueing the timed replay to its end
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        del g
        t = stamps.cpu().numpy()
        ms = (int(t[1]) - int(t[0])) / kq.TIMESTAMP_HZ * 1e3 / steps
        if name:
            replay_us[name] = round(e0.elapsed_time(e1) * 1e3 / (steps + warmup), 3)
        return ms, wall

    def per_launch(fn, n=200):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for i, (a, b) in enumerate(evs):
            a.record(stream)
            fn(i % nsets)
            b.record(stream)
        torch.cuda.synchronize()
        t = np.array([a.elapsed_time(b) for a, b in evs]) * 1e3
        return {"median_us": round(float(np.median(t)), 3), "p10_us": round(float(np.percentile(t, 10)), 3),
                "p90_us": round(float(np.percentile(t, 90)), 3)}

    # the single-launch ceiling of this traffic (about 50 ms, reported below), then the other shapes and
    # workloads, this one last with its KroQuant kernels last (several seconds of every quantizer): the hot
    # path is timed right after the GPU has run it, at the clocks it runs at inside a model's step, not in
    # the clock transient that follows memory-only work on some boxes
    ceiling = launch_sweep(kq, Xs, Cs, Ss, nsets, int(min(2000, max(30, 20e9 // nbytes))), nbytes, stream)
    table2 = None if args.no_table2 else table2_shapes(kq, synth, dev, stream, sptr)
    table4 = None if args.no_table2 else table2_shapes(kq, synth, dev, stream, sptr, shapes=TABLE4_SHAPES, fwht=False)
    wl_cache = {WORKLOAD: w}
    configs = None if args.no_configs else config_table(kq, synth, dev, stream, names=args.configs.split(","),
                                                        cache=wl_cache, last=args.workload)
    # timed region: exactly K steps of the hot path, after W warmup steps
    ms_kq, wall_kq = timed(run_kq, args.steps, args.warmup, name="kroquant")
    us_kq = ms_kq * 1e3
    ms_kq_eager, _ = timed_eager(run_kq, args.steps, args.warmup)
    gbs = nbytes / (ms_kq * 1e-3) / 1e9

    comparators = {}
    for name in ("kroquant_onthefly", "kroquant_lu", "kroquant_exact", "smoothquant", "hadamard32", "mxfp4",
                 "stream_floor"):
        ms, _ = timed(runs[name], args.steps, args.warmup, name=name)
        comparators[name + "_us"] = round(ms * 1e3, 3)
        comparators[name + "_gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
    ms_floor_eager, _ = timed_eager(run_floor, args.steps, args.warmup)
    ms_warm, _ = timed(run_kq, args.steps, args.warmup, rotate=False)
    # the vendor's device-to-device copy moving the same HBM bytes as one step
    # (half of them read, half written), with the same rotation
    half = nbytes // 2
    copy_src = [Xs[i].view(torch.uint8).reshape(-1)[:half] for i in range(nsets)]
    copy_dst = [torch.empty(half, dtype=torch.uint8, device=dev) for _ in range(nsets)]

    def run_copy(i):
        copy_dst[i].copy_(copy_src[i])

    ms_copy, _ = timed(run_copy, args.steps, args.warmup)
    del copy_dst
    gemm = None if args.no_gemm else gemm_timing(kq, synth, dev, stream, sptr, Cs[0], Ss[0], M, d)
    calib = None if args.no_calib else calib_timing(kq, synth, dev, stream, sptr, args.calib_samples)
    dist = per_launch(run_kq)

    parity = "skipped"
    if not args.no_parity:
        parity = check_parity(w, run_kq, run_k2, run_kx, Cs, Ss)
    quality = quantization_error(kq, Xs[0], A, B, kpack, mult)

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("kernel_source_hash") == kernel_source_hash() and tr.get("workload") == args.workload:
            traffic = tr.get("hbm_bytes_per_launch")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, nbytes, wl_cache, synth)

    line = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_kq, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "M": M, "d": d, "a": int(w.meta["a"]), "b": int(w.meta["b"]),
                   "nfac": int(w.meta["nfac"]), "dist": w.meta["dist"], "input": "bf16",
                   "output": "MXFP4 (E2M1 codes + E8M0 scales)",
                   "mall": f"cold: {nsets} rotating buffer sets, {nsets * set_bytes / 1e6:.0f} MB"},
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "kernel_us": round(us_kq, 3),
        "kroquant_vs_smoothquant": round(comparators["smoothquant_us"] / us_kq, 3),
        "traffic_floor": {"us": comparators["stream_floor_us"], "gbs": comparators["stream_floor_gbs"],
                          "frac_of_peak": round(comparators["stream_floor_gbs"] / HBM_PEAK_GBS, 4),
                          "hot_path_frac_of_floor": round(comparators["stream_floor_us"] / us_kq, 4),
                          "what": "kq_stream_floor: the same loads, stores and launch shape with no arithmetic"},
        "single_launch_ceiling": ceiling,
        "hot_path_frac_of_ceiling": round(ceiling["us"] / us_kq, 4),
        "vendor_copy": {"us": round(ms_copy * 1e3, 3), "gbs": round(2 * half / (ms_copy * 1e-3) / 1e9, 1),
                        "frac_of_peak": round(2 * half / (ms_copy * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                        "what": "torch copy_ (device to device) of half the step's bytes: the same HBM traffic "
                                "as one step, same graph replay and rotation"},
        "paper_context": "other hardware, context only: on an MI350 the paper reports its fused quantizer kernel "
                         "up to 14% faster than its SmoothQuant kernel (abstract; Table 4 lists up to 1.31x)",
        "path": "kq_quantize_packed: matrix cores (v_mfma_f32_32x32x16_bf16, 3-term bf16 split of the "
                "materialised A(x)B packed offline)",
        "comparators": comparators,
        "timing": "value: the K launches captured into a HIP graph (before the timed region) behind the W warmup "
                  "launches and between two kq_timestamp stamps of the 100 MHz device counter; the W warmup steps "
                  "run eagerly, then the graph is replayed once untimed and once timed, queued back to back (no "
                  "idle GPU before the timed launches); time per step = stamp difference of the timed replay / K. "
                  "replay_events_us_per_launch: HIP events around the timed replay (its W warmup steps and the "
                  "graph launch included) / (W + K); eager_python: the same K launches from the Python loop "
                  "(ctypes call per step)",
        "replay_events_us_per_launch": replay_us,
        "eager_python": {"kroquant_us": round(ms_kq_eager * 1e3, 3), "stream_floor_us": round(ms_floor_eager * 1e3, 3)},
        "per_launch_events": dist,
        "warm_single_buffer": {"us": round(ms_warm * 1e3, 3), "gbs": round(nbytes / (ms_warm * 1e-3) / 1e9, 1)},
        "wall_s_timed_region": round(wall_kq, 4),
        "parity": parity,
        "quantization_error": quality,
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic},
        "cpu_baseline": cpu,
        "configs": configs,
        "table2_pow2_d": table2,
        "table4_production": table4,
        "w4a4_gemm": gemm,
        "calibration": calib,
    }
    print(json.dumps(line), flush=True)


# Every workload of the paper's shapes that the benchmark times (name -> how it is built):
# the DiT activation shapes, the shard one GPU holds when FLUX's 12288-wide MLP input is split
# eight ways along d (tensor parallelism; the quantizer has no cross-GPU step), and the large
# per-block stress shape in both factor splits.
CONFIG_WORKLOADS = ["tiny_256x1152", "pixart_8192x1152", "pixart_8192x4608", "sana_4096x2240", "sana_4096x5600",
                    "flux_4608x3072", "flux_4608x12288", "shard_4608x1536", "large_18432x12288",
                    "large_18432x12288_2x16"]


def _config_inputs(name, synth, dev, cache):
    """(X on the device, A, B, lu, mult, per_block, description) of one table workload."""
    import torch
    if name.startswith("large"):
        a, b = (2, 16) if name.endswith("2x16") else (4, 8)
        M, d = 18432, 12288
        nb = d // 32
        if "large_X" not in cache:
            cache["large_X"] = synth.activations_device(M, d, seed=100, device=dev)
        X = cache["large_X"]
        A, B = synth.factors(a, b, nb, seed=4)
        lu = synth.lu_params(nb, seed=8)
        amax = X.abs().amax(0).float()
        mult = torch.where(amax > 0, amax.rsqrt(), torch.ones_like(amax))
        return X, A, B, lu, mult, True, (f"Student-t(3), 0.5% channels x50, drawn on the device; {nb} factor "
                                         f"pairs ({a}x{a} (x) {b}x{b}) and {nb} LU sets, one per 32-column block")
    if name == "shard_4608x1536":
        w = cache.get("flux_4608x12288") or synth.workload("flux_4608x12288")
        cache["flux_4608x12288"] = w
        Xh = np.ascontiguousarray(w.X[:, :1536])
        desc = "columns 0..1535 of flux_4608x12288 (its share of one GPU when d is split 8 ways)"
        A, B, mult = w.A, w.B, synth.smoothquant_multipliers(Xh)
    else:
        w = cache.get(name) or synth.workload(name)
        cache[name] = w
        Xh, A, B, mult = w.X, w.A, w.B, w.mult
        desc = f"{w.meta['dist']}, seed {w.meta['seed']}"
    X = torch.from_numpy(Xh.view(np.int16)).view(torch.bfloat16).to(dev)
    return X, A, B, synth.lu_params(1, seed=7), torch.from_numpy(mult).to(dev), False, desc


def _graph_us(fn, nsets, steps, stream):
    """Per-launch time of `steps` launches of fn(i % nsets) captured once into
    a HIP graph between two kq_timestamp stamps of the 100 MHz device counter:
    3 untimed replays, then the median of 3 replays of (stamp difference) /
    steps -- the launches alone, without the fixed cost of launching the
    graph."""
    import torch
    import paper_2607_21446_amd as kq
    stamps = torch.zeros(2, dtype=torch.int64, device="cuda")
    for i in range(nsets):  # eager pass over every set
        fn(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kq.timestamp(stamps, 0)
        for i in range(steps):
            fn(i % nsets)
        kq.timestamp(stamps, 1)
    for _ in range(3):  # untimed: upload, then clocks settle
        g.replay()
    torch.cuda.synchronize()
    ts = []
    for _ in range(3):
        g.replay()
        torch.cuda.synchronize()
        t = stamps.cpu().numpy()
        ts.append((int(t[1]) - int(t[0])) / kq.TIMESTAMP_HZ * 1e6 / steps)
    del g
    return float(np.median(ts))


# Launch shapes of the traffic-only probe: (waves per workgroup, 64-block units per wave, workgroups;
# 0 = one pass over the units, else a grid-stride loop)
PROBE_SHAPES = [(1, 1, 0), (2, 1, 0), (4, 1, 0), (8, 1, 0), (16, 1, 0), (1, 2, 0), (1, 4, 0), (2, 4, 0),
                (1, 1, 2048), (1, 1, 4096), (4, 1, 1024), (16, 1, 256)]


def launch_sweep(kq, Xs, Cs, Ss, nsets, steps, nbytes, stream):
    """The quantizers' traffic (kq_stream_probe) in every launch shape of
    PROBE_SHAPES, and kq_stream_floor (one wave, one unit, the quantizers'
    own shape): what one launch of these bytes reaches on this chip."""
    sweep = {"kq_stream_floor": round(_graph_us(lambda i: kq.stream_floor(Xs[i], out16=Cs[i], out1=Ss[i]), nsets,
                                                steps, stream), 3)}
    for w, u, g in PROBE_SHAPES:
        us = _graph_us(lambda i: kq.stream_probe(Xs[i], w, u, g, out16=Cs[i], out1=Ss[i]), nsets, steps, stream)
        sweep[f"waves{w}_units{u}_" + (f"stride{g}" if g else "onepass")] = round(us, 3)
    best = min(sweep, key=sweep.get)
    gbs = nbytes / sweep[best] * 1e-3
    return {"us": sweep[best], "gbs": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4), "shape": best,
            "sweep_us": sweep,
            "what": "kq_stream_probe: the quantizers' bytes (2 B read, 17/32 B written per element) in each launch "
                    "shape listed, and kq_stream_floor; the best one is the single-launch ceiling of this traffic"}


def config_table(kq, synth, dev, stream, names=CONFIG_WORKLOADS, graph_bytes=20e9, cache=None, last=None):
    """Every workload of CONFIG_WORKLOADS: KroQuant (packed K1, on-the-fly K2
    from A and B, LU-form K2 from the 15 parameters), SmoothQuant, Hadamard-32,
    plain MXFP4 and the traffic-only kernel on identical inputs.  Each kernel's
    launches (about graph_bytes of traffic, 30 to 2000 launches) are captured
    once into a HIP graph over enough rotating buffer sets to exceed twice the
    MALL, and the time per launch is read from device stamps around them.
    The workload `last` is timed last, and in every row the KroQuant kernels
    come after the comparators, the packed call last."""
    import torch
    cache = {} if cache is None else cache
    names = [n for n in names if n != last] + [n for n in names if n == last]
    out = {}
    for name in names:
        X0, A, B, lu, mult, per_block, desc = _config_inputs(name, synth, dev, cache)
        M, d = X0.shape
        nbytes = algorithmic_bytes(M, d)
        nsets = 2 if per_block else max(2, int(np.ceil(2 * MALL_BYTES / nbytes)) + 1)
        Xs = [X0] + [X0.clone() for _ in range(nsets - 1)]
        Cs = [torch.empty((M, d // 2), dtype=torch.uint8, device=dev) for _ in range(nsets)]
        Ss = [torch.empty((M, d // 32), dtype=torch.uint8, device=dev) for _ in range(nsets)]
        Ad, Bd = torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev)
        lud = torch.from_numpy(lu).to(dev)
        kpack = kq.pack_factors(Ad, Bd)
        fns = {
            "smoothquant": lambda i: kq.smoothquant(Xs[i], mult, codes=Cs[i], scales=Ss[i]),
            "hadamard32": lambda i: kq.hadamard32(Xs[i], codes=Cs[i], scales=Ss[i]),
            "mxfp4": lambda i: kq.mxfp4(Xs[i], codes=Cs[i], scales=Ss[i]),
            "stream_floor": lambda i: kq.stream_floor(Xs[i], out16=Cs[i], out1=Ss[i]),
            "kroquant_lu": lambda i: kq.quantize_lu(Xs[i], lud, A.shape[-1], codes=Cs[i], scales=Ss[i]),
            "kroquant_onthefly": lambda i: kq.quantize(Xs[i], Ad, Bd, codes=Cs[i], scales=Ss[i]),
            "kroquant_packed": lambda i: kq.quantize_packed(Xs[i], Ad, Bd, kpack, codes=Cs[i], scales=Ss[i]),
        }
        steps = int(min(2000, max(30, graph_bytes // nbytes)))
        row = {"M": M, "d": d, "a": int(A.shape[-1]), "b": int(B.shape[-1]), "nfac": int(A.shape[0]),
               "input": desc, "algorithmic_bytes": nbytes, "steps": steps,
               "mall": f"cold: {nsets} rotating buffer sets, {nsets * nbytes / 1e6:.0f} MB"}
        for kname, fn in fns.items():
            us = _graph_us(fn, nsets, steps, stream)
            gbs = nbytes / us * 1e-3
            row[kname] = {"us": round(us, 3), "gbs": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4)}
        sq = row["smoothquant"]["us"]
        for k in ("kroquant_packed", "kroquant_onthefly", "kroquant_lu"):
            row[k]["vs_smoothquant"] = round(sq / row[k]["us"], 3)
        row["hadamard32"]["vs_smoothquant"] = round(sq / row["hadamard32"]["us"], 3)
        if name == "flux_4608x12288":
            row["single_launch_ceiling"] = launch_sweep(kq, Xs, Cs, Ss, nsets, steps, nbytes, stream)
        out[name] = row
        del Xs, Cs, Ss, X0, kpack
        torch.cuda.empty_cache()
    cache.pop("large_X", None)
    torch.cuda.empty_cache()
    out["timing"] = ("per kernel: a HIP graph of `steps` launches over MALL-cold rotating buffer sets between two "
                     "kq_timestamp stamps, replayed 3 times untimed, then the median of 3 replays of the stamp "
                     "difference / steps; vs_smoothquant = SmoothQuant time / this kernel's time")
    return out


TABLE2_SHAPES = [(4096, 1024), (4096, 4096), (4096, 16384), (512, 4096), (512, 16384)]


# The paper's Table 4 production shapes (FLUX.1 / PixArt-Sigma layers), with the paper's own Scale/K1 and
# Scale/K2 on an MI350 (fp16 activations, Triton) as context: not a target for this machine.
TABLE4_SHAPES = [(512, 3072), (512, 12288), (4096, 1152), (4096, 3072), (4096, 3456), (4096, 4096), (4096, 4608),
                 (4096, 12288)]
TABLE4_PAPER_RATIOS = {(512, 3072): (1.18, 1.02), (512, 12288): (1.12, 0.86), (4096, 1152): (1.31, 0.96),
                       (4096, 3072): (1.10, 0.91), (4096, 3456): (1.14, 0.95), (4096, 4096): (1.10, 0.95),
                       (4096, 4608): (1.08, 0.94), (4096, 12288): (0.99, 0.94)}


def table2_shapes(kq, synth, dev, stream, sptr, steps=500, shapes=None, fwht=True):
    """The paper's power-of-two-d comparison (Sec. 4.4, Table 2): Q4, Scale
    (SmoothQuant), K1 (kq_quantize_packed), K2 (kq_quantize_lu, 15 parameters
    decoded on chip) and the full-row FWHT; with `shapes` = TABLE4_SHAPES and
    fwht=False, the production shapes of Table 4 (Q4, Scale, K1, K2, and the
    paper's own MI350 ratios beside ours as context).  Several of these kernels
    take less time than one Python-side launch, so each kernel's `steps`
    launches (MALL-cold rotation over buffer sets) are captured once into a HIP
    graph between two device stamps and the graph is replayed (_graph_us)."""
    import torch
    A, B = synth.factors(4, 8, 1, seed=5)
    Ad, Bd = torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev)
    lu = torch.from_numpy(synth.lu_params(1, seed=7)).to(dev)
    kpack = kq.pack_factors(Ad, Bd, stream=sptr)
    torch.cuda.synchronize()
    out = {}
    for m, d in (shapes or TABLE2_SHAPES):
        X = synth.activations(m, d, "student_t3", seed=m + d, chan_frac=0.005, chan_factor=50.0)
        mult = torch.from_numpy(synth.smoothquant_multipliers(X)).to(dev)
        nbytes = algorithmic_bytes(m, d)
        nsets = max(2, int(np.ceil(2 * MALL_BYTES / nbytes)) + 1)
        X0 = torch.from_numpy(X.view(np.int16)).view(torch.bfloat16).to(dev)
        Xs = [X0.clone() for _ in range(nsets)]
        Cs = [torch.empty((m, d // 2), dtype=torch.uint8, device=dev) for _ in range(nsets)]
        Ss = [torch.empty((m, d // 32), dtype=torch.uint8, device=dev) for _ in range(nsets)]
        # stream=None: launch on the current stream, which is the capture stream inside the graph
        fns = {
            "q4": lambda i: kq.mxfp4(Xs[i], codes=Cs[i], scales=Ss[i]),
            "scale": lambda i: kq.smoothquant(Xs[i], mult, codes=Cs[i], scales=Ss[i]),
            "k1": lambda i: kq.quantize_packed(Xs[i], Ad, Bd, kpack, codes=Cs[i], scales=Ss[i]),
            "k2": lambda i: kq.quantize_lu(Xs[i], lu, 4, codes=Cs[i], scales=Ss[i]),
        }
        if fwht:
            fns["fwht"] = lambda i: kq.fwht(Xs[i], codes=Cs[i], scales=Ss[i])
        row = {}
        for name, fn in fns.items():
            row[name + "_us"] = round(_graph_us(fn, nsets, steps, stream), 3)
        row["k1_gbs"] = round(nbytes / row["k1_us"] * 1e-3, 1)
        row["scale_over_k1"] = round(row["scale_us"] / row["k1_us"], 3)
        row["scale_over_k2"] = round(row["scale_us"] / row["k2_us"], 3)
        if fwht:
            row["fwht_over_k2"] = round(row["fwht_us"] / row["k2_us"], 3)
        if (m, d) in TABLE4_PAPER_RATIOS:
            row["paper_mi350_scale_over_k1"], row["paper_mi350_scale_over_k2"] = TABLE4_PAPER_RATIOS[(m, d)]
        out[f"{m}x{d}"] = row
        del Xs, Cs, Ss, X0
        torch.cuda.empty_cache()
    out["timing"] = ("HIP graph of 500 launches per kernel between two kq_timestamp stamps, median of 3 replays; "
                     "MALL-cold rotation")
    return out


BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak of the MI355X
FP4_PEAK_TFLOPS = 10100.0  # MI355X dense MXFP4 matrix-core peak, TFLOP/s


def gemm_timing(kq, synth, dev, stream, sptr, xc, xs, M, K, steps=100):
    """The W4A4 product that consumes the quantizer output (kq_mxfp4_gemm):
    the headline activation's MXFP4 codes times an MXFP4 weight from
    kq_weight_transform (synthetic weights, N = 3072 and 12288), fp32 output,
    and the same product rounded to bf16 (kq_mxfp4_gemm_bf16)."""
    import torch
    out = {}
    A, B = synth.factors(4, 8, 1, seed=5)
    for N in (3072, 12288):
        W = synth.activations(N, K, "normal", seed=N, chan_frac=0.0)
        Wd = torch.from_numpy(W.view(np.int16)).view(torch.bfloat16).to(dev)
        _, wc, ws = kq.weight_transform(Wd, torch.from_numpy(A), torch.from_numpy(B))
        C = torch.empty((M, N), dtype=torch.float32, device=dev)
        for _ in range(10):
            kq.mxfp4_gemm(xc, xs, wc, ws, C=C, stream=sptr)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            kq.mxfp4_gemm(xc, xs, wc, ws, C=C, stream=sptr)
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / steps * 1e3
        tf = 2.0 * M * N * K / us * 1e-6
        row = {"us": round(us, 2), "tflops": round(tf, 1), "frac_fp4_peak": round(tf / FP4_PEAK_TFLOPS, 4)}
        # the same product with the output rounded to bf16 (kq_mxfp4_gemm_bf16): half the C bytes
        C16 = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        for _ in range(10):
            kq.mxfp4_gemm(xc, xs, wc, ws, C=C16, stream=sptr)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            kq.mxfp4_gemm(xc, xs, wc, ws, C=C16, stream=sptr)
        e1.record(stream)
        torch.cuda.synchronize()
        us16 = e0.elapsed_time(e1) / steps * 1e3
        tf16 = 2.0 * M * N * K / us16 * 1e-6
        row["bf16_output"] = {"us": round(us16, 2), "tflops": round(tf16, 1),
                              "frac_fp4_peak": round(tf16 / FP4_PEAK_TFLOPS, 4)}
        row["vendor_scaled_mm"] = vendor_gemm(xc, xs, wc, ws, C, stream, steps)
        out[f"{M}x{N}x{K}"] = row
        del W, Wd, wc, ws, C, C16
    out["peak_tflops"] = FP4_PEAK_TFLOPS
    return out


def vendor_gemm(xc, xs, wc, ws, C, stream, steps):
    """The same MXFP4 product through the vendor's library (torch._scaled_mm
    on E2M1 codes with E8M0 scales per 32-element block, bf16 output), timed
    as kq_mxfp4_gemm; a comparator, never used by the library.  `max_rel_diff`
    is max |vendor - C| / max |C| against kq_mxfp4_gemm's fp32 C."""
    import torch
    M, N, K = xc.shape[0], wc.shape[0], 2 * xc.shape[1]
    a, b = xc.view(torch.float4_e2m1fn_x2), wc.view(torch.float4_e2m1fn_x2)
    sa, sb = xs.view(torch.float8_e8m0fnu), ws.view(torch.float8_e8m0fnu)
    try:
        with torch.cuda.stream(stream):
            def run():
                return torch._scaled_mm(a, b.t(), scale_a=sa, scale_b=sb, out_dtype=torch.bfloat16)
            ref = run()
            for _ in range(9):
                run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(steps):
                run()
            e1.record(stream)
        torch.cuda.synchronize()
    except (RuntimeError, TypeError, AttributeError) as e:
        return {"error": repr(e)[:200]}
    us = e0.elapsed_time(e1) / steps * 1e3
    tf = 2.0 * M * N * K / us * 1e-6
    diff = float((ref.float() - C).abs().max() / C.abs().max())
    return {"us": round(us, 2), "tflops": round(tf, 1), "frac_fp4_peak": round(tf / FP4_PEAK_TFLOPS, 4),
            "max_rel_diff": round(diff, 6)}


def calib_timing(kq, synth, dev, stream, sptr, samples, steps=5, warmup=2):
    """Layer-wise calibration (Sec. 3.3) of one FLUX.1 linear layer: `samples`
    calibration activations of 4608 tokens (d = 3072, the Student-t(3) recipe
    drawn on the device), a synthetic 3072 x 3072 weight, one LU parameter set
    per 32-column block (96 x 15 parameters), Hadamard start.  Times (HIP
    events on the launch stream) kq_calib_reference, kq_calib_step with the
    Adam update, and the paper's whole optimisation: kq_calibrate with 100
    steps (lambda evaluation, 100 updates, final evaluation), whose first and
    last objective values are reported."""
    import torch
    d = o = 3072
    R = samples * 4608
    nfac = d // 32
    X = synth.activations_device(R, d, seed=samples, device=dev)
    W = torch.from_numpy(synth.weights(o, d, seed=1).view(np.int16)).view(torch.bfloat16).to(dev)
    Yneg = torch.empty((R, o), dtype=torch.float32, device=dev)
    ws = kq.calib_workspace(R, o, d, 4, nfac, dev)
    lu = kq.hadamard_lu(nfac, dev)
    lam = torch.zeros(2, dtype=torch.float32, device=dev)
    m = torch.zeros(nfac * 15, dtype=torch.float32, device=dev)
    v = torch.zeros_like(m)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    st = stream
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record(st)
    kq.calib_reference(X, W, Yneg, stream=sptr)
    e1.record(st)
    losses, _ = kq.calib_step(X, W, Yneg, lu, lam, workspace=ws, stream=sptr)
    torch.cuda.synchronize()
    ms_ref = e0.elapsed_time(e1)
    L0 = losses.cpu().numpy()
    lam.copy_(torch.tensor([L0[0] / L0[1], L0[0] / L0[2]], dtype=torch.float32))  # automatic lambdas
    for t in range(1, warmup + 1):
        kq.calib_step(X, W, Yneg, lu, lam, workspace=ws, adam=(m, v, t, 1e-2), stream=sptr)
    torch.cuda.synchronize()
    e0.record(st)
    for t in range(warmup + 1, warmup + steps + 1):
        losses, _ = kq.calib_step(X, W, Yneg, lu, lam, workspace=ws, adam=(m, v, t, 1e-2), stream=sptr)
    e1.record(st)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    # the paper's whole per-layer optimisation from the Hadamard start: kq_calibrate, 100 Adam steps of lr 1e-2
    lu_full = kq.hadamard_lu(nfac, dev)
    torch.cuda.synchronize()
    e0.record(st)
    _, rows = kq.calibrate(X, W, lu=lu_full, steps=100, lr=1e-2, Yneg=Yneg, workspace=ws, stream=sptr)
    e1.record(st)
    torch.cuda.synchronize()
    ms_full = e0.elapsed_time(e1)
    rows = rows.cpu().numpy()
    back = 2 * 2.0 * R * o * d     # the two backward products, algorithmic flops
    fwd = 2.0 * R * o * d          # the W4A4 product of the forward pass
    out = {
        "workload": f"FLUX.1 layer: {samples} samples x 4608 tokens, d = o = 3072, per-block LU ({nfac} x 15)",
        "rows": R, "steps": steps, "warmup": warmup,
        "ms_per_step": round(ms, 3),
        "ms_reference": round(ms_ref, 3),
        "s_per_layer_100_steps": round((ms_ref + ms_full) / 1e3, 3),
        "kq_calibrate_100_steps_ms": round(ms_full, 1),
        "L_out_hadamard_start": float(rows[0, 0]),
        "L_out_after_100_steps": float(rows[-1, 0]),
        "L_start_with_lambdas": float(rows[1, 3]),
        "L_after_100_steps": float(rows[-1, 3]),
        "lambdas": [float(rows[0, 0] / rows[0, 1]), float(rows[0, 0] / rows[0, 2])],
        "flops_per_step": {"backward": back, "forward_w4a4": fwd},
        "backward_tflops_whole_step": round(back / (ms * 1e-3) / 1e12, 1),
        "backward_dtype": "bf16 (residual as two bf16 terms), fp32 accumulation",
        "peak_bf16_tflops": BF16_PEAK_TFLOPS,
    }
    del X, W, Yneg, ws
    torch.cuda.empty_cache()
    return out


E2M1_MAGNITUDES = (0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0)


def quantization_error(kq, X, A, B, kpack, mult):
    """The quality side metric (not a target): ||deq(Q(y)) - y||_F / ||y||_F
    for each method's own transformed values y (Sec. 3.1's activation loss
    L_A) on the headline input -- KroQuant (its random near-identity factors
    are not calibrated, so it is not expected to win here), SmoothQuant,
    Hadamard-32 and plain MXFP4.  Dequantization (E2M1 magnitude x 2^(s-127))
    and the norms are torch ops on the device, in fp64."""
    import torch
    mags = torch.tensor(E2M1_MAGNITUDES, dtype=torch.float64, device=X.device)

    def rel(codes, scales, y):
        c = codes.to(torch.int64)
        nib = torch.stack((c & 15, c >> 4), dim=-1).reshape(codes.shape[0], -1)  # element 2i in the low nibble
        v = mags[nib & 7] * torch.where(nib >= 8, -1.0, 1.0)
        scale = torch.exp2(scales.to(torch.float64) - 127.0).repeat_interleave(32, dim=1)
        y64 = y.to(torch.float64)
        return round(float(torch.linalg.norm(v * scale - y64) / torch.linalg.norm(y64)), 6)

    out = {}
    c, s, y = kq.quantize_packed(X, A, B, kpack, want_y=True)
    out["kroquant"] = rel(c, s, y)
    c, s, y = kq.smoothquant(X, mult, want_y=True)
    out["smoothquant"] = rel(c, s, y)
    c, s, y = kq.hadamard32(X, want_y=True)
    out["hadamard32"] = rel(c, s, y)
    c, s = kq.mxfp4(X)
    out["mxfp4"] = rel(c, s, X.to(torch.float32))
    out["what"] = ("||deq(Q(y)) - y||_F / ||y||_F on the headline input, y each method's transformed values; "
                   "KroQuant with random near-identity (uncalibrated) factors")
    return out


def check_parity(w, run_kq, run_k2, run_kx, Cs, Ss):
    """Outputs of the timed launches against the oracle, as they were timed
    (no fp32 output): the hot path and the on-the-fly variant to the method's
    tolerance (oracle.mx_compare: scales identical, codes within adjacent
    flips that sit at rounding ties of the oracle's y, at most 1e-4 of them),
    the fixed-order path bit for bit."""
    import torch

    import oracle
    cr, sr, yr = oracle.quantize(w.X, w.A, w.B, want_y=True)
    torch.cuda.synchronize()
    out = {}
    for key, run in (("hot_path", run_kq), ("onthefly", run_k2)):
        run(0)
        torch.cuda.synchronize()
        rep = oracle.mx_compare(Cs[0].cpu().numpy(), Ss[0].cpu().numpy(), cr, sr, y_ref=yr)
        out[key] = (("ok" if rep["ok"] else "FAIL") + f": scale mismatches {rep['scale_mismatches']}, "
                    f"code flips {rep['flips']}/{rep['codes']} (non-adjacent {rep['non_adjacent']}, "
                    f"off a rounding tie {rep['off_tie']})")
    run_kx(0)
    torch.cuda.synchronize()
    exact_ok = np.array_equal(Cs[0].cpu().numpy(), cr) and np.array_equal(Ss[0].cpu().numpy(), sr)
    out["exact_path"] = "bit-exact" if exact_ok else "MISMATCH"
    return out


def _oracle_seconds(w, passes):
    import oracle
    t = []
    for _ in range(passes):
        t0 = time.perf_counter()
        oracle.quantize(w.X, w.A, w.B)
        t.append(time.perf_counter() - t0)
    return float(np.median(t))


def cpu_baseline(w, nbytes, cache, synth):
    """The oracle, untuned, on this host's cores: whole-workload passes of the
    headline workload until at least 10 s have elapsed (at most 30 s, at least
    one pass), then the same oracle on one thread (median of 3); and the Tiny
    and wide FLUX workloads on all cores and on one thread (median of 3 each)."""
    import oracle
    threads = oracle.num_threads()
    times = []
    t_start = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        oracle.quantize(w.X, w.A, w.B)
        times.append(time.perf_counter() - t0)
        el = time.perf_counter() - t_start
        if el >= 10.0 or el + times[-1] > 30.0:
            break
    t = float(np.median(times))
    others = {}
    oracle.set_num_threads(1)
    try:
        t1m = _oracle_seconds(w, 3)
    finally:
        oracle.set_num_threads(threads)
    for name in ("tiny_256x1152", "flux_4608x12288"):
        wo = cache.get(name) or synth.workload(name)
        cache[name] = wo
        nb_o = algorithmic_bytes(*wo.X.shape)
        t_all = _oracle_seconds(wo, 3)
        oracle.set_num_threads(1)
        try:
            t_one = _oracle_seconds(wo, 3)
        finally:
            oracle.set_num_threads(threads)
        others[name] = {"all_cores": {"gbs": round(nb_o / t_all / 1e9, 3), "s_per_pass": round(t_all, 4),
                                      "threads": threads},
                        "one_thread": {"gbs": round(nb_o / t_one / 1e9, 3), "s_per_pass": round(t_one, 4)},
                        "sample": "3 full passes each (median)"}
    return {"value": round(nbytes / t / 1e9, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(times)} full passes of {w.name} (median {t:.3f} s per pass)",
            "single_thread": {"value": round(nbytes / t1m / 1e9, 3), "unit": "GB/s",
                              "sample": f"3 full passes of {w.name} on 1 thread (median {t1m:.3f} s per pass)"},
            "other_workloads": others,
            "host_cpus": os.cpu_count(), "cpu_model": _cpu_model()}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
