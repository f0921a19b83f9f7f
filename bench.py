#!/usr/bin/env python3
"""Benchmark of fused batched HDC inference on one MI355X.

One step = one pass of Alg. 1 (encode, HardSign, similarity, argmax) over one
batch of synthetic inputs already resident in device memory. Prints one JSON
line: whole-job samples/s, the roofline fraction of the dominant kernel
(algorithmic bytes or flops per launch over the measured launch duration),
and the CPU oracle's throughput on a bounded sample as a baseline.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
    python bench.py --sweep-d     # N = 1, F = 3072, K = 10: one line per D (bandwidth map)
    python bench.py --sweep-n     # F = 561, D = 10240, K = 6: one line per N (samples/s curve)
    python bench.py --workload speech --dtype i8      # the int8 model variant
    python bench.py --workload colour_k10 --train     # single-pass training (Sec. II-C)
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import hd_inputs  # noqa: E402

CSRC = os.path.join(ROOT, "paper_2506_09282_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")

METRIC = "inference samples/sec at D=10240 (N=1..65536); % HBM / MFMA roofline"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3, "i8": 5000.0}  # dense; i8 in TOP/s
PEAK_UNIT = {"bf16": "TFLOP/s", "f32": "TFLOP/s", "i8": "TOP/s"}
ESIZE = {"f32": 4, "bf16": 2, "i8": 1}
TRAIN_METRIC = "single-pass training samples/sec (class hypervectors from N labelled samples)"
MALL_BYTES = 256 << 20

# workload -> (dtype, path description)
BENCH_DTYPE = {"activity_n1": "f32", "activity_n32": "f32", "tiny": "f32", "image": "bf16",
               "speech": "bf16", "colour_k10": "bf16", "colour_k100": "bf16", "colour_n1": "f32"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None)
    p.add_argument("--warmup", type=int, default=None)
    p.add_argument("--workload", default="activity_n32", choices=sorted(hd_inputs.WORKLOADS))
    p.add_argument("--dtype", default=None, choices=["f32", "bf16", "i8"])
    p.add_argument("--raw", action="store_true",
                   help="time hd_infer on B and C as given (no packed model): the large-batch "
                        "route re-tiles B and C into the workspace inside every call")
    p.add_argument("--train", action="store_true",
                   help="single-pass training: one step = clear the class counts, "
                        "hd_bundle_classes_packed over the workload's N labelled samples, "
                        "hd_class_hardsign")
    p.add_argument("--copies", type=int, default=0,
                   help="distinct model copies rotated per step (0 = enough to exceed the MALL)")
    p.add_argument("--no-graph", action="store_true", help="time an eager loop instead of a graph")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target CPU time of the oracle baseline sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-floors", action="store_true",
                   help="skip the streaming-read and empty-launch floor measurements")
    p.add_argument("--d", type=int, default=0, help="override the workload's D")
    p.add_argument("--sweep-n", action="store_true",
                   help="samples/s curve: one JSON line per N in hd_inputs.N_SWEEP for the "
                        "activity shape (F=561, D=10240, K=6), no CPU baseline")
    p.add_argument("--sweep-d", action="store_true",
                   help="single-sample bandwidth map: one JSON line per D in hd_inputs.D_SWEEP "
                        "for the colour_n1 shape (F=3072, K=10), no CPU baseline")
    p.add_argument("--stream", type=int, default=0, metavar="NBATCH",
                   help="streaming mode: NBATCH batches of the workload's N samples, all "
                        "resident in device memory, consumed by one persistent launch "
                        "(hd_infer_stream) per timed step; reports per-batch time")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="after timing, run a plain device-to-device copy of this many MiB "
                        "(the reference kernel for scaling hardware byte counters)")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; multi-GPU sharding is a design "
                                   "note only (split-N replicas or split-D with an all-reduce of "
                                   "partial scores)", "n_gpus": args.gpus}))
        sys.exit(2)
    if args.sweep_n:
        args.workload, args.no_cpu_baseline, args.no_floors = "activity_n32", True, True
        base = hd_inputs.WORKLOADS["activity_n32"]
        for n in hd_inputs.N_SWEEP:
            run(args, dataclasses.replace(base, name=f"activity_n{n}", N=n))
        return
    if args.sweep_d:
        args.workload, args.no_cpu_baseline, args.no_floors = "colour_n1", True, True
        base = hd_inputs.WORKLOADS["colour_n1"]
        for d in hd_inputs.D_SWEEP:
            run(args, dataclasses.replace(base, name=f"colour_n1_d{d}", D=d))
        return
    w = hd_inputs.WORKLOADS[args.workload]
    if args.d:
        w = dataclasses.replace(w, name=f"{w.name}_d{args.d}", D=args.d)
    if args.stream:
        run_stream(args, w)
        return
    if args.train:
        run_train(args, w)
        return
    run(args, w)


def make_data(w, dtype, seed=0):
    """The workload's X, B, C as float32 (f32, bf16-rounded for bf16) or int8."""
    if dtype == "i8":
        return hd_inputs.make_int8_inputs(w.N, w.F, w.D, w.K, seed=seed)
    return hd_inputs.make_inputs(w.N, w.F, w.D, w.K, w.x_dist, seed=seed, dtype=dtype)


def to_device(a, dtype, dev):
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)
    if dtype == "i8":
        return torch.from_numpy(np.ascontiguousarray(a, np.int8)).to(dev)
    return torch.from_numpy(hd_inputs.bf16_bits(a).view(np.int16)).to(dev).view(torch.bfloat16)


def run_train(args, w):
    """One step = one single-pass training over the workload's N samples with
    uniform labels: counts cleared (a fill kernel), class sums of
    HardSign(X B) (hd_bundle_classes_packed, B tiled once before timing),
    codebook = HardSign(counts) (hd_class_hardsign)."""
    import torch
    import paper_2506_09282_amd as hd

    dtype = args.dtype or BENCH_DTYPE[args.workload]
    steps = args.steps or 20
    warmup = args.warmup if args.warmup is not None else 3
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] train workload={w.name} N={w.N} F={w.F} D={w.D} K={w.K} dtype={dtype} "
          f"steps={steps} warmup={warmup}", file=sys.stderr, flush=True)
    X, B, _ = make_data(w, dtype)
    y = np.random.default_rng(1).integers(0, w.K, w.N).astype(np.int32)
    Xd, Bd = to_device(X, dtype, dev), to_device(B, dtype, dev)
    yd = torch.from_numpy(y).to(dev)
    model = hd.pack_model(Bd, K=w.K)
    counts = torch.zeros((w.K, w.D), dtype=torch.int32, device=dev)
    M = torch.empty((w.K, w.D), dtype=torch.float32, device=dev)
    kernel = hd.bundle_kernel(w.N, w.F, w.D, w.K, Xd.dtype, packed=True)
    stream = torch.cuda.Stream(device=dev)

    def step():
        counts.zero_()
        hd.bundle_classes_packed(Xd, model, yd, w.K, counts=counts)
        hd.class_hardsign(counts, out=M)

    with torch.cuda.stream(stream):
        for _ in range(warmup):
            step()
    stream.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        ev0.record(stream)
        for _ in range(steps):
            step()
        ev1.record(stream)
    ev1.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    value = w.N / (ms / 1e3)
    flops = 2.0 * w.N * w.F * w.D
    roof = {"bound": "mfma", "achieved": flops / (ms / 1e3) / 1e12,
            "peak": MFMA_PEAK_TFLOPS[dtype], "unit": PEAK_UNIT[dtype],
            "traffic": recorded_traffic(w.name + "_train", kernel, dtype),
            "kernel_time": "whole step (fill + class sums + HardSign)"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in roof.items()}
    out = {
        "metric": TRAIN_METRIC, "value": round(value, 1), "unit": "samples/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.name} training: N={w.N} labelled samples, F={w.F} "
                               f"D={w.D} K={w.K}, labels uniform, X~{w.x_dist if dtype != 'i8' else 'U{-128..127}'}, seed 0",
                   "global_batch": w.N, "parallelism": "single GPU", "kernel": kernel,
                   "model": "B tiled once before timing"},
        "roofline": roof,
    }
    calib_copies(args, dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_train(w, X, B, y, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def cpu_baseline_train(w, X, B, y, target_s):
    """The oracle's bundle on the host cores over a bounded prefix of the
    training set (about target_s seconds)."""
    import oracle
    orc = oracle.default()
    threads = orc.threads(0)
    n_probe = min(w.N, 8 * threads)
    t0 = time.perf_counter()
    orc.bundle(X[:n_probe], B, y[:n_probe], w.K)
    per = (time.perf_counter() - t0) / n_probe
    n = int(max(1, min(w.N, target_s / max(per, 1e-9))))
    t0 = time.perf_counter()
    orc.bundle(X[:n], B, y[:n], w.K)
    dt = time.perf_counter() - t0
    return {"value": round(n / dt, 3), "unit": "samples/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"the first {n} of the {w.N} labelled samples, float64 loops, "
                      f"{dt:.1f} s on {threads} threads"}


def run_stream(args, w):
    """One step = one persistent launch over args.stream batches of N samples
    (a queue already filled); the model is read from HBM once per launch."""
    import torch
    import paper_2506_09282_amd as hd

    nbatch = args.stream
    steps = args.steps or 20
    warmup = args.warmup if args.warmup is not None else 3
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] stream workload={w.name} nbatch={nbatch} N={w.N} F={w.F} D={w.D} K={w.K} "
          f"steps={steps} warmup={warmup}", file=sys.stderr, flush=True)
    X, B, C = hd_inputs.make_inputs(nbatch * w.N, w.F, w.D, w.K, w.x_dist, seed=0)
    Xd = torch.from_numpy(X.reshape(nbatch, w.N, w.F)).to(dev)
    model = hd.pack_model(torch.from_numpy(B).to(dev), torch.from_numpy(C).to(dev))
    labels = torch.empty((nbatch, w.N), dtype=torch.int32, device=dev)
    ws = torch.zeros(hd.stream_workspace_bytes(nbatch, w.N, w.F, w.D, w.K, torch.float32),
                     dtype=torch.uint8, device=dev)
    stream = torch.cuda.Stream(device=dev)

    def step():
        hd.infer_stream(Xd, model, out=(labels, None), workspace=ws)

    with torch.cuda.stream(stream):
        for _ in range(warmup):
            step()
    stream.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        ev0.record(stream)
        for _ in range(steps):
            step()
        ev1.record(stream)
    ev1.synchronize()
    ms = ev0.elapsed_time(ev1)
    batches = steps * nbatch
    s_per_batch = ms / 1e3 / batches
    value = w.N * batches / (ms / 1e3)
    flops = 2.0 * w.N * w.D * (w.F + w.K)
    hbm_per_launch = 4 * (w.F * w.D + w.K * w.D + nbatch * w.N * w.F) + 4 * nbatch * w.N
    roof = {"bound": "mfma", "achieved": flops / s_per_batch / 1e12,
            "peak": MFMA_PEAK_TFLOPS["f32"], "unit": "TFLOP/s",
            "traffic": recorded_traffic(f"{w.name}_stream{nbatch}", "stream_frag_kernel", "f32")}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["hbm_GBs"] = hbm_per_launch / (ms / 1e3 / steps) / 1e9
    roof = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in roof.items()}
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "samples/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms / steps, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name} stream: {nbatch} batches of N={w.N} per launch, "
                               f"F={w.F} D={w.D} K={w.K} X~{w.x_dist}, B,C~N(0,1), HardSign, "
                               f"seed 0", "global_batch": w.N, "batches_per_step": nbatch,
                   "us_per_batch": round(s_per_batch * 1e6, 4), "parallelism": "single GPU",
                   "kernel": "stream_frag_kernel", "model": "packed once before timing"},
        "roofline": roof,
    }
    calib_copies(args, dev)
    print(json.dumps(out), flush=True)


def run(args, w):
    import torch
    import paper_2506_09282_amd as hd

    dtype = args.dtype or BENCH_DTYPE[args.workload]
    small = w.N <= 64
    steps = args.steps or (2000 if small else 100)
    warmup = args.warmup if args.warmup is not None else (200 if small else 10)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] workload={w.name} N={w.N} F={w.F} D={w.D} K={w.K} dtype={dtype} "
          f"steps={steps} warmup={warmup}", file=sys.stderr, flush=True)

    X, B, C = make_data(w, dtype)

    def up(a):
        return to_device(a, dtype, dev)

    esz = ESIZE[dtype]
    model_bytes = esz * (w.F * w.D + w.K * w.D)
    copies = args.copies or (max(1, -(-2 * MALL_BYTES // model_bytes)) if small else 1)
    Xd = up(X)
    Bs = [up(B)]
    Cs = [up(C)]
    for _ in range(copies - 1):
        Bs.append(Bs[0].clone())
        Cs.append(Cs[0].clone())
    # the model is packed once, outside the timed region, like weights loaded
    # for serving; every step reads the packed image (with --raw, B and C as
    # given, and every call packs what it needs itself)
    models = None if args.raw else [hd.pack_model(b, c) for b, c in zip(Bs, Cs)]
    if not args.raw:
        del Bs, Cs
    labels = torch.empty(w.N, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    stream = torch.cuda.Stream(device=dev)
    hdt = {"f32": hd.HD_F32, "bf16": hd.HD_BF16, "i8": hd.HD_I8}[dtype]
    ws_bytes = int(hd.lib().hd_infer_workspace_bytes(w.N, w.F, w.D, w.K, hdt) if args.raw
                   else hd.lib().hd_infer_packed_workspace_bytes(w.N, w.F, w.D, w.K, hdt))
    ws = torch.zeros(max(ws_bytes, 1), dtype=torch.uint8, device=dev)

    def step(i):
        if args.raw:
            hd.infer(Xd, Bs[i % copies], Cs[i % copies], out=(labels, None), workspace=ws)
        else:
            hd.infer_packed(Xd, models[i % copies], out=(labels, None), workspace=ws)

    with torch.cuda.stream(stream):
        for i in range(3):
            step(i)
    stream.synchronize()

    graph_len = min(steps, 100 if small else 10)
    use_graph = not args.no_graph
    graph = None
    if use_graph:
        try:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                for i in range(graph_len):
                    step(i)
            stream.synchronize()
        except Exception as e:  # graph capture unavailable: time the eager loop
            print(f"[bench] graph capture failed ({e}); timing eager launches", file=sys.stderr)
            graph, use_graph = None, False
    reps = -(-steps // graph_len) if use_graph else steps
    steps_timed = reps * graph_len if use_graph else steps

    def timed(n_rep):
        with torch.cuda.stream(stream):
            if use_graph:
                for _ in range(n_rep):
                    graph.replay()
            else:
                for i in range(n_rep):
                    step(i)

    timed(max(1, warmup // (graph_len if use_graph else 1)))
    stream.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        ev0.record(stream)
    timed(reps)
    with torch.cuda.stream(stream):
        ev1.record(stream)
    ev1.synchronize()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1)
    ms_per_step = ms / steps_timed
    value = w.N * steps_timed / (ms / 1e3)
    print(f"[bench] timed {steps_timed} steps in {ms:.3f} ms", file=sys.stderr, flush=True)

    # Roofline of the dominant (only) kernel of a step: one launch per step.
    launch_s = ms_per_step / 1e3
    kernel = hd.infer_kernel(w.N, w.F, w.D, w.K, Xd.dtype, packed=not args.raw)
    traffic = recorded_traffic(w.name + ("_raw" if args.raw else ""), kernel, dtype)
    if small:
        alg_bytes = alg_bytes_of(w, dtype)
        roof = {"bound": "hbm", "achieved": alg_bytes / launch_s / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "traffic": traffic}
    else:
        flops = 2.0 * w.N * w.D * (w.F + w.K)
        roof = {"bound": "mfma", "achieved": flops / launch_s / 1e12,
                "peak": MFMA_PEAK_TFLOPS[dtype], "unit": PEAK_UNIT[dtype], "traffic": traffic}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in roof.items()}

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "samples/s", "n_gpus": 1,
        "steps": steps_timed, "warmup": warmup, "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.note}; N={w.N} F={w.F} D={w.D} K={w.K} "
                               + (f"X~{w.x_dist}, B,C~N(0,1)" if dtype != "i8"
                                  else "X,B,C~U{-128..127} (int8 model variant)")
                               + ", HardSign, seed 0",
                   "global_batch": w.N, "parallelism": "single GPU",
                   "model_copies_rotated": copies, "timing": "hip graph" if use_graph else "eager",
                   "kernel": kernel,
                   "model": ("B and C as given (hd_infer)" if args.raw
                             else "packed once before timing")},
        "roofline": roof,
    }
    if not args.no_floors:
        fl = measure_floors(dev, stream, alg_bytes_of(w, dtype) if small else 0, copies)
        out["floors"] = fl
        if small and fl.get("stream_read_GBs"):
            roof["measured_peak"] = fl["stream_read_GBs"]
            roof["frac_of_measured"] = round(roof["achieved"] / fl["stream_read_GBs"], 4)
    calib_copies(args, dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, X, B, C, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def calib_copies(args, dev):
    """Three plain device-to-device copies of --calib-copy-mib MiB after the
    timed work: the reference dispatches for scaling hardware byte counters."""
    if args.calib_copy_mib <= 0:
        return
    import torch
    n = args.calib_copy_mib << 18  # fp32 elements
    src = torch.ones(n, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()


def alg_bytes_of(w, dtype) -> int:
    """Algorithmic bytes of one call: X, B and C read once, labels written."""
    esz = ESIZE[dtype]
    return esz * (w.N * w.F + w.F * w.D + w.K * w.D) + 4 * w.N


def measure_floors(dev, stream, same_bytes: int, copies: int):
    """Floors of the machine the benchmark runs on, from bench_floors.hip:
    the streaming read bandwidth of a 2 GiB buffer (well past the 256 MB
    last-level cache), the time of one launch that only reads `same_bytes`
    bytes (cold: rotated over enough buffers to exceed the cache, replayed in
    a graph like the timed steps), and the time of one empty launch."""
    import ctypes
    import torch
    lib_path = os.path.join(ROOT, "bench_floors.so")
    if not os.path.exists(lib_path):
        from paper_2506_09282_amd import build as hbuild
        hbuild.build_floors()
    L = ctypes.CDLL(lib_path)
    L.floors_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                     ctypes.c_int, ctypes.c_void_p]
    L.floors_stream_read.restype = ctypes.c_int
    L.floors_empty.argtypes = [ctypes.c_void_p]
    L.floors_empty.restype = ctypes.c_int
    blocks = 4096
    sink = torch.empty(blocks, dtype=torch.float32, device=dev)

    def ev_time(fn, reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            fn()
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) / reps / 1e3

    def check(rc):
        if rc != 0:
            raise RuntimeError(f"bench_floors launch failed ({rc})")

    out = {}
    big = torch.empty(2 << 30, dtype=torch.uint8, device=dev)
    n16 = big.numel() // 16
    sp = stream.cuda_stream
    t = ev_time(lambda: check(L.floors_stream_read(big.data_ptr(), n16, sink.data_ptr(), blocks,
                                                   sp)), 5)
    out["stream_read_GBs"] = round(big.numel() / t / 1e9, 1)
    del big

    def graph_time(fn, n_per_graph=100, reps=20):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for i in range(n_per_graph):
                fn(i)
        stream.synchronize()
        return ev_time(g.replay, reps) / n_per_graph

    out["empty_launch_us"] = round(graph_time(lambda i: check(L.floors_empty(sp))) * 1e6, 3)
    if same_bytes > 0:
        nb = max(copies, 1)
        bufs = [torch.empty(same_bytes // 16 * 16, dtype=torch.uint8, device=dev)
                for _ in range(nb)]
        n = bufs[0].numel() // 16
        t = graph_time(lambda i: check(L.floors_stream_read(
            bufs[i % nb].data_ptr(), n, sink.data_ptr(), 1024, sp)))
        out["read_same_bytes_us"] = round(t * 1e6, 3)
        out["read_same_bytes"] = int(bufs[0].numel())
        del bufs
    torch.cuda.synchronize()
    return out


def source_digest() -> str:
    """SHA-256 over the HIP sources, in name order (identifies the kernels)."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".hpp")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def recorded_traffic(workload: str, kernel: str, dtype: str):
    """HBM bytes per launch from the committed counter summaries under
    profiles/ (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy's readings),
    or None when none matches this workload, kernel, dtype and source digest."""
    if not os.path.isdir(PROFILES):
        return None
    digest = source_digest()
    for name in sorted(os.listdir(PROFILES)):
        if not name.endswith(".md"):
            continue
        with open(os.path.join(PROFILES, name)) as f:
            for line in f:
                if not line.startswith("traffic-record:"):
                    continue
                kv = dict(t.split("=", 1) for t in line.split()[1:] if "=" in t)
                if (kv.get("workload") == workload and kv.get("kernel") == kernel
                        and kv.get("dtype") == dtype and kv.get("source_sha256") == digest):
                    return int(kv["bytes_per_launch"])
    return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, X, B, C, target_s):
    """The oracle as it stands, on the host cores, over a bounded sample; then
    on one thread over a smaller sample."""
    import oracle
    orc = oracle.default()
    threads = orc.threads(0)
    # probe with a few rows per thread, then size the sample to about target_s
    probe_rows = np.arange(4 * threads) % w.N
    t0 = time.perf_counter()
    orc.infer(X, B, C, rows=probe_rows)
    per_row = (time.perf_counter() - t0) / len(probe_rows)
    n_rows = int(max(1, min(target_s / max(per_row, 1e-9), 1e7)))
    rows = np.arange(n_rows) % w.N
    t0 = time.perf_counter()
    orc.infer(X, B, C, rows=rows)
    dt = time.perf_counter() - t0
    # one thread: about a quarter of the time budget
    n1 = int(max(1, min(target_s / 4 / max(per_row * threads, 1e-9), 1e6)))
    rows1 = np.arange(n1) % w.N
    t0 = time.perf_counter()
    orc.infer(X, B, C, rows=rows1, nthreads=1)
    dt1 = time.perf_counter() - t0
    return {"value": round(n_rows / dt, 3), "unit": "samples/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "single_thread_value": round(n1 / dt1, 3),
            "sample": f"{n_rows} rows of the same workload (rows cycled over the batch), "
                      f"float64 loops, {dt:.1f} s on {threads} threads; {n1} rows in "
                      f"{dt1:.1f} s on one thread"}


if __name__ == "__main__":
    main()
