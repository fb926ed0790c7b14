#!/usr/bin/env python3
"""Benchmark of the microscaled-FP4 linear layer on one MI355X.

One step = one pass of the whole hot path over the 14B-like NVFP4 MLP gate/up
projection (X[4096 x 5120] activations with 1% outlier channels, W[27648 x 5120]
= gate || up weights, both bfloat16, seeded synthetic):
  quantize and fake-quant X in one pass (codes + scales for the product, and
    the QAT forward's quantize-dequantize in bfloat16; dynamic global scale:
    one pass over X plus a small fix-up kernel),
  the same for W,
  W4A4 GEMM Y = X^ W^T (FP32 accumulation, bfloat16 output).
The separate quantize and fake-quant entry points are timed apart as well.
All inputs are resident in HBM before timing starts.  Prints ONE JSON line.

value = 2*M*N*K / step time (TFLOP/s of the layer, whole step).  The roofline
entry is for the dominant kernel (the GEMM), timed with HIP events on the
stream the kernels run on.
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

METRIC = "W4A4 GEMM TFLOPS & % FP4 MFMA peak (prefill); quantize/decode HBM GB/s"
GEMM_SOURCES = ["paper_2606_15682_amd/csrc/gemm_tile256.hip", "paper_2606_15682_amd/csrc/gemm.hip",
                "paper_2606_15682_amd/csrc/fp4_device.h"]
# the sources a committed traffic summary was measured on, per kind of row
TRAFFIC_SOURCES = {
    "gemm": GEMM_SOURCES,
    "w4a16": ["paper_2606_15682_amd/csrc/gemm_w4a16.hip", "paper_2606_15682_amd/csrc/fp4_device.h"],
    "kv4": ["paper_2606_15682_amd/csrc/kv4.hip", "paper_2606_15682_amd/csrc/fp4_device.h"],
    "skinny": ["paper_2606_15682_amd/csrc/gemm_skinny.hip", "paper_2606_15682_amd/csrc/fp4_device.h"],
    "sem": ["paper_2606_15682_amd/csrc/sem.hip"],
}


def code_text(src: str) -> str:
    """C/C++ source with its comments and blank lines removed and trailing
    blanks stripped: what a compiled kernel depends on, so that an edit of a
    comment leaves a measurement taken on the source valid.  (String and
    character literals are copied whole, so a // inside one is kept.)"""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    lines = (ln.rstrip() for ln in "".join(out).split("\n"))
    return "\n".join(ln for ln in lines if ln)


def source_hash(kind: str = "gemm") -> str:
    """SHA-256 of the code (code_text) of the sources a row's traffic summary
    was measured on."""
    import hashlib
    h = hashlib.sha256()
    for rel in TRAFFIC_SOURCES[kind]:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(code_text(f.read()).encode("utf-8"))
    return h.hexdigest()


def gemm_source_hash() -> str:
    return source_hash("gemm")


def profiled_traffic_file(name: str, kind: str):
    """HBM bytes per launch (or per step, as the summary states) from the
    committed rocprofv3 FETCH_SIZE/WRITE_SIZE summary profiles/<name> (each
    counter scaled by its reading for a plain copy of known size); None when
    there is no summary or the row's sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_sha256", kv.get("gemm_source_sha256")) != source_hash(kind):
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def profiled_traffic(fmt_name: str, workload: int):
    """Traffic of the tile GEMM of a prefill workload (see profiled_traffic_file)."""
    return profiled_traffic_file("gemm_%s_workload%d_traffic.txt" % (fmt_name, workload), "gemm")


PEAK = {"fp4": 10100.0, "f16": 2500.0, "hbm": 8000.0}   # TFLOP/s, TFLOP/s, GB/s (MI355X published)
# workloads timed as a decode step (quantize X + product, weights quantized once,
# untimed); the others run the whole step (quantize and fake-quant both operands)
DECODE_WORKLOADS = {2}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=4,
                    help="workload number (4 = 14B gate/up; 10 = the same shape in MXFP4; 5 = 32B down-proj "
                         "MXFP4; 2 = NVFP4 W4A4 decode; 6, 7 = MXFP4 W4A16 decode; 8 = SEM loss head; "
                         "9 = KV4 keys)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="skip timing the step as a HIP graph replay")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device copy of this many bytes --steps times "
                         "(calibrates rocprof FETCH_SIZE/WRITE_SIZE against a known size)")
    return ap.parse_args()


def graph_step_ms(step, args) -> float:
    """Mean time of `step` captured once in a HIP graph and replayed args.steps
    times (events around the replays).  The library allocates, clears and
    synchronises nothing, so a step of its calls captures as is."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                       # warm-up on the capture stream
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for _ in range(max(1, args.warmup)):
        graph.replay()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(args.steps):
        graph.replay()
    ev[1].record()
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / args.steps


MALL_DEFEAT_BYTES = 512 << 20       # twice the 256 MB Infinity Cache


def n_copies(nbytes_one: int, args) -> int:
    """Copies of a per-step operand to rotate through so that every timed step
    reads bytes that are not in the Infinity Cache: more than 512 MB in all, and
    enough that the timed steps never come back to a copy the warm-up touched."""
    return max(-(-MALL_DEFEAT_BYTES // max(1, int(nbytes_one))), args.steps + args.warmup + 1)


def timed_rotation(step, n, args):
    """Eager steps over rotating copies (step(i) uses copy i % n): warm-up on
    copies 0 .. W-1, then args.steps timed steps on copies W, W+1, ...; returns
    (wall-clock ms per step, device ms per step from HIP events on the stream)."""
    import torch
    for i in range(args.warmup):
        step(i % n)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(args.steps):
        step((args.warmup + i) % n)
    ev[1].record()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / args.steps, ev[0].elapsed_time(ev[1]) / args.steps


def graph_rotation_ms(step, n, args, replays: int = 3) -> float:
    """Amortized device time per step: n consecutive steps (one per copy, so the
    graph's working set exceeds the Infinity Cache) captured in one HIP graph,
    replayed `replays` times after one untimed replay."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n):
            step(i)
    graph.replay()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(replays):
        graph.replay()
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / (replays * n)
    del graph
    return ms


def copy_calibration(nbytes: int, steps: int):
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": src.numel() * 4, "steps": steps}), flush=True)


def practical_ceilings(x=None, wt=None, steps=10):
    """Context, not targets: what a plain device copy and the vendor library's
    bfloat16 GEMM of the same shape (no quantization; hipBLASLt through torch)
    reach on this GPU.  Neither is on the product path."""
    import torch
    out = {}
    n = 1 << 28                                         # 1 GiB of float32 per buffer
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(steps):
        dst.copy_(src)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / steps
    out["copy_GBps"] = round(2.0 * n * 4 / (ms * 1e-3) / 1e9, 1)
    read = read_probe_gbps(src)
    if read is not None:
        out["read_GBps"] = read
    del src, dst
    if x is not None and wt is not None and x.shape[0] > 64:
        # W^T made contiguous: a plain (non-batched) NN product
        b = wt.t().contiguous()
        y = torch.mm(x, b)
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(steps):
            torch.mm(x, b, out=y)
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / steps
        M, K = x.shape
        N = b.shape[1]
        out["bf16_library_gemm_TFLOPs"] = round(2.0 * M * N * K / (ms * 1e-3) / 1e12, 1)
        out["bf16_library_gemm_ms"] = round(ms, 4)
        del b, y
    torch.cuda.empty_cache()
    out["note"] = ("device copy of 1 GiB (read + write bytes); read-only stream of 1 GiB (libreqat_probe.so); "
                   "torch.mm of the same bfloat16 operands, unquantized (vendor GEMM)")
    return out


def read_probe_gbps(buf, steps: int = 10):
    """Context: the read-only HBM stream rate of libreqat_probe.so's read probe
    over the 1 GiB device tensor `buf` (2048 workgroups, 16-byte loads); None
    when the probe library is not built."""
    import ctypes

    import torch

    from paper_2606_15682_amd import build as pbuild
    if not os.path.exists(pbuild.PROBE_LIB):
        return None
    lib = ctypes.CDLL(pbuild.PROBE_LIB)
    lib.reqat_probe_read.restype = ctypes.c_int
    lib.reqat_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    blocks = 2048
    out = torch.empty(blocks * 256, dtype=torch.int32, device=buf.device)
    nbytes = buf.numel() * buf.element_size()
    st = torch.cuda.current_stream(buf.device).cuda_stream

    def launch():
        if lib.reqat_probe_read(buf.data_ptr(), nbytes, out.data_ptr(), blocks, st) != 0:
            raise RuntimeError("reqat_probe_read failed")

    launch()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(steps):
        launch()
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / steps
    return round(nbytes / (ms * 1e-3) / 1e9, 1)


def mfma_probe_tflops(kind: int, ops, warmup: int = 10, reps: int = 20, iters: int = 1500) -> float:
    """Context, not a target: the rate of the register-only MFMA loop of
    libreqat_probe.so (one wave per SIMD, 256 workgroups) on 8 KB of operand
    words `ops` (uint8 device tensor: A words, then B words) -- what the
    matrix cores sustain on that data with no memory traffic.  kind 0: scaled
    FP4 32x32x64, kind 1: FP16 32x32x16."""
    import ctypes

    import torch

    from paper_2606_15682_amd import build as pbuild
    lib = ctypes.CDLL(pbuild.PROBE_LIB)
    lib.reqat_probe_mfma.restype = ctypes.c_int
    lib.reqat_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_void_p]
    assert ops.dtype == torch.uint8 and ops.numel() == 8192 and ops.is_contiguous()
    blocks = 256
    out = torch.empty(blocks * 256, dtype=torch.float32, device=ops.device)
    st = torch.cuda.current_stream(ops.device).cuda_stream

    def launch():
        rc = lib.reqat_probe_mfma(kind, ops.data_ptr(), out.data_ptr(), blocks, iters, st)
        if rc != 0:
            raise RuntimeError("reqat_probe_mfma failed (%d)" % rc)

    for _ in range(warmup):
        launch()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(reps):
        launch()
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    flops = blocks * 4 * iters * 16 * (131072 if kind == 0 else 32768)
    return flops / (ms * 1e-3) / 1e12


def operand_words(a, b):
    """8 KB of probe operand words: the first 4 KB of a's and of b's bytes (repeated if shorter)."""
    import torch

    def first(t):
        v = t.contiguous().view(torch.uint8).flatten()
        if v.numel() < 4096:
            v = v.repeat(-(-4096 // v.numel()))
        return v[:4096]
    return torch.cat([first(a), first(b)])


class pinned_to_one_core:
    """Runs the enclosed oracle timing on one host core (the affinity of
    taskset -c <core>), restoring the process's affinity afterwards."""

    def __enter__(self):
        self.saved = os.sched_getaffinity(0)
        self.core = min(self.saved)
        os.sched_setaffinity(0, {self.core})
        return self

    def __exit__(self, *exc):
        os.sched_setaffinity(0, self.saved)
        return False


def cpu_baseline(w, xb, wb):
    """Time the CPU oracle (single thread, as it stands, pinned to one core) on
    a bounded sample of the same step and scale its per-element / per-MAC rates
    to the full step."""
    with pinned_to_one_core() as pin:
        out = _cpu_baseline(w, xb, wb)
    out["pinned_core"] = pin.core
    return out


def _cpu_baseline(w, xb, wb):
    import numpy as np
    import oracle
    fmt = oracle.FMT_NVFP4 if w.fmt == "nvfp4" else oracle.FMT_MXFP4
    rows_x = 256
    t0 = time.perf_counter()
    wc, ws_, wg = oracle.quantize(fmt, wb)
    t_qw = time.perf_counter() - t0
    t0 = time.perf_counter()
    xc, xs, xg = oracle.quantize(fmt, np.ascontiguousarray(xb[:rows_x]))
    t_qx = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.fakequant(fmt, np.ascontiguousarray(xb[:rows_x]))
    t_fq = time.perf_counter() - t0
    gemm_rows = 4
    t0 = time.perf_counter()
    oracle.gemm(fmt, xc[:gemm_rows], xs[:gemm_rows], xg, wc, ws_, wg)
    t_mm = time.perf_counter() - t0
    per_q = (t_qw + t_qx) / ((w.N + rows_x) * w.K)
    per_fq = t_fq / (rows_x * w.K)
    per_mac = t_mm / (gemm_rows * w.N * w.K)
    full = per_q * (w.M + w.N) * w.K + per_fq * (w.M + w.N) * w.K + per_mac * w.M * w.N * w.K
    return {
        "value": round(2.0 * w.M * w.N * w.K / full / 1e12, 9),
        "unit": "TFLOP/s",
        "cores": 1,
        "kind": "oracle",
        "sample": ("oracle quantize of all of W and of 256 rows of X, fake-quant of 256 rows of X, "
                   "FP64 GEMM of 4 rows of X against all of W; per-element and per-MAC rates "
                   "scaled to the full step (%.1f s of CPU work; full step would take %.0f s)"
                   % (t_qw + t_qx + t_fq + t_mm, full)),
        "host_threads_available": len(os.sched_getaffinity(0)),
    }


def bench_w4a16(args, w):
    """W4A16 decode step: the product of bfloat16 activations with MXFP4 weights
    (quantized once, untimed: served weights are stored quantized).  Bound by HBM."""
    import numpy as np
    import torch

    from paper_2606_15682_amd import reqat
    from paper_2606_15682_amd import workloads as wl

    reqat.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    M, N, K = w.M, w.N, w.K
    x_cpu, w_cpu = wl.make_x(w), wl.make_w(w)
    x = x_cpu.to(dev)
    wc0, ws0, _ = reqat.quantize(w_cpu.to(dev), reqat.MXFP4)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    wsp = torch.empty(max(1, reqat.reqat_w4a16_workspace_bytes(M, N, K)), dtype=torch.uint8, device=dev)
    flops = 2.0 * M * N * K
    nbytes = N * K * (0.5 + 1.0 / 32) + M * K * 2.0 + M * N * 2.0       # W codes + scales, x, Y (bf16)
    # rotate through copies of the weights (> 512 MB in all): every step streams them from HBM.
    # Served weights are stored once in the product's packed image (pack_w4a16,
    # untimed, like the quantization); the product from the row-major codes is context.
    ncp = n_copies(N * K * (0.5 + 1.0 / 32), args)
    copies = [(wc0.clone(), ws0.clone()) for _ in range(ncp)]
    packed = [reqat.pack_w4a16(a, b) for a, b in copies]

    def step(i):
        reqat.gemm_w4a16_packed(x, packed[i], N, out_dtype=torch.bfloat16, out=y, ws=wsp)

    def step_rowmajor(i):
        wc, ws = copies[i]
        reqat.gemm_w4a16(x, wc, ws, out_dtype=torch.bfloat16, out=y, ws=wsp)

    # value: the product over the weight copies, ncp launches captured in one HIP
    # graph (back to back, as a serving loop runs them), per launch
    ms_eager, ms_eager_dev = timed_rotation(step, ncp, args)
    ms_step = graph_rotation_ms(step, ncp, args)
    ms_kernel = ms_step
    ms_rowmajor = graph_rotation_ms(step_rowmajor, ncp, args)
    # context: the same weights every step (they then sit in the Infinity Cache)
    _, ms_resident = timed_rotation(lambda i: step(0), ncp, args)
    gbs = nbytes / (ms_kernel * 1e-3) / 1e9
    ksplit = reqat.reqat_w4a16_workspace_bytes(M, N, K) // (4 * M * N)   # FP32 partial sums per split
    out = {
        "metric": METRIC,
        "value": round(nbytes / (ms_step * 1e-3) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; Student-t or Gaussian-with-outlier activations, N(0,0.02) weights)",
        "config": {"workload": w.name, "M": M, "N": N, "K": K, "format": "mxfp4 weights, bf16 activations",
                   "gemm_out": "bf16", "global_batch": M, "parallelism": "single GPU",
                   "step": "W4A16 GEMM (weights pre-quantized and packed, untimed), each step on another of %d "
                           "weight copies (%.0f MB in all, twice the Infinity Cache), the %d steps captured in one "
                           "HIP graph, time per step" % (ncp, ncp * N * K * (0.5 + 1.0 / 32) / 1e6, ncp)},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK["hbm"], "unit": "GB/s",
                     "frac": round(gbs / PEAK["hbm"], 4),
                     "traffic": profiled_traffic_file("w4a16_mxfp4_workload%d_traffic.txt" % args.workload, "w4a16"),
                     "kernel": "gemm_w4a16_kernel on the packed weight image%s (MXFP4 W4A16, algorithmic bytes %d)"
                               % (" + gemm_w4a16_reduce (K split %d ways)" % ksplit if ksplit > 1 else "",
                                  int(nbytes))},
        "kernels": {"gemm_w4a16_packed": {"ms": round(ms_kernel, 4), "GB/s": round(gbs, 1),
                                          "TFLOP/s": round(flops / (ms_kernel * 1e-3) / 1e12, 2),
                                          "note": "per launch in the graph, weights from HBM (rotating copies)"},
                    "gemm_w4a16_rowmajor": {"ms": round(ms_rowmajor, 4),
                                            "GB/s": round(nbytes / (ms_rowmajor * 1e-3) / 1e9, 1),
                                            "note": "context: the same product from the row-major codes and "
                                                    "scales (reqat_gemm_w4a16), per launch in the graph"},
                    "eager": {"ms": round(ms_eager, 4), "device_ms": round(ms_eager_dev, 4),
                              "note": "context: eager launches from Python, wall clock and HIP-event time"},
                    "cache_resident": {"ms": round(ms_resident, 4),
                                       "GB/s": round(nbytes / (ms_resident * 1e-3) / 1e9, 1),
                                       "note": "context only: the same weights every step (Infinity-Cache "
                                               "resident after the first)"}},
    }
    out["ceilings"] = practical_ceilings()
    if not args.no_cpu_baseline:
        with pinned_to_one_core():
            import oracle
            xb, wb = wl.bf16_bits(x_cpu), wl.bf16_bits(w_cpu)
            owc, ows, _ = oracle.quantize(oracle.FMT_MXFP4, wb[:64])
            npts = int(5e8 // K)                        # about 10 s of single-thread CPU work
            ms_, ns_ = np.arange(npts) % M, np.arange(npts) % 64
            t0 = time.perf_counter()
            oracle.gemm_w4a16_points(xb, owc, ows, ms_, ns_)
            dt = time.perf_counter() - t0
            per_mac = dt / (npts * K)
            full = per_mac * M * N * K
            out["cpu_baseline"] = {
                "value": round(nbytes / full / 1e9, 6), "unit": "GB/s", "cores": 1, "kind": "oracle",
                "sample": ("FP64 W4A16 oracle on %d output points (each a %d-term dot product), per-MAC "
                           "rate scaled to the full product and credited with its bytes (%.2f s of CPU work)"
                           % (npts, K, dt))}
    print(json.dumps(out), flush=True)


def bench_decode(args, w):
    """Decode step of the W4A4 layer (M <= 64 activation rows): quantize X and
    multiply by weights that were quantized and packed once, untimed (served
    weights are stored quantized, in the decode product's packed image), in one
    reqat_linear_w4a4_packed call.  Bound by HBM: the weights stream once per
    step.  The same step on the row-major weights is context."""
    import numpy as np
    import torch

    from paper_2606_15682_amd import reqat
    from paper_2606_15682_amd import workloads as wl

    reqat.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    fmt = reqat.NVFP4 if w.fmt == "nvfp4" else reqat.MXFP4
    B = reqat.BLOCK[fmt]
    M, N, K = w.M, w.N, w.K
    x_cpu, w_cpu = wl.make_x(w), wl.make_w(w)
    x = x_cpu.to(dev)
    wc0, wsc0, gw = reqat.quantize(w_cpu.to(dev), fmt)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    gl = torch.empty(1, dtype=torch.float32, device=dev) if fmt == reqat.NVFP4 else None
    lws = torch.empty(reqat.reqat_linear_workspace_bytes(fmt, M, K), dtype=torch.uint8, device=dev)
    w_bytes = N * K * (0.5 + 1.0 / B)
    step_bytes = w_bytes + M * K * 2.0 + M * N * 2.0              # weights once, x read, Y (bf16)
    gemm_bytes = w_bytes + M * K * (0.5 + 1.0 / B) + M * N * 2.0  # weights once, x codes, Y (bf16)
    # rotate through copies of the quantized weights (> 512 MB in all): every
    # step streams its weights from HBM, as a model's layers do
    ncp = n_copies(w_bytes, args)
    copies = [(wc0.clone(), wsc0.clone()) for _ in range(ncp)]
    packed = [reqat.pack_w4a4(a, b, fmt) for a, b in copies]

    def step(i):
        reqat.linear_packed(x, fmt, packed[i], N, gw, out_dtype=torch.bfloat16, out=y, g_out=gl, ws=lws)

    def step_rowmajor(i):
        wc, wsc = copies[i]
        reqat.linear(x, fmt, wc, wsc, gw, out_dtype=torch.bfloat16, out=y, g_out=gl, ws=lws)

    # A decode step is a few microseconds of device work, less than one eager
    # launch from Python costs: steps run back to back only when captured, as a
    # serving loop captures them.  value = the step captured ncp times in one HIP
    # graph (each on its own weight copy), per step; eager launches are context.
    ms_eager, ms_dev = timed_rotation(step, ncp, args)
    ms_step = graph_rotation_ms(step, ncp, args)
    ms_step_rowmajor = graph_rotation_ms(step_rowmajor, ncp, args)
    _, ms_resident = timed_rotation(lambda i: step(0), ncp, args)

    # the product alone (activation codes from one quantize), timed apart, also over the copies
    xc, xs, gx = reqat.quantize(x, fmt)

    def gemm_step(i):
        reqat.gemm_packed(fmt, xc, xs, gx, packed[i], N, gw, out_dtype=torch.bfloat16, out=y)

    def gemm_step_rowmajor(i):
        wc, wsc = copies[i]
        reqat.gemm(fmt, xc, xs, gx, wc, wsc, gw, out_dtype=torch.bfloat16, out=y)

    ms_gemm = graph_rotation_ms(gemm_step, ncp, args)
    ms_gemm_rowmajor = graph_rotation_ms(gemm_step_rowmajor, ncp, args)
    gbs_gemm = gemm_bytes / (ms_gemm * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if fmt == reqat.NVFP4 else "fp4",
        "data": "synthetic (seeded; Gaussian activations with outlier channels, N(0,0.02) weights)",
        "config": {"workload": w.name, "M": M, "N": N, "K": K, "format": w.fmt, "gemm_out": "bf16",
                   "global_batch": M, "parallelism": "single GPU",
                   "step": "quantize X + W4A4 GEMM in one reqat_linear_w4a4_packed call (weights quantized "
                           "and packed once, untimed), each step on another of %d weight copies (%.0f MB in all, "
                           "twice the Infinity Cache); the %d steps captured in one HIP graph, time per step"
                           % (ncp, ncp * w_bytes / 1e6, ncp)},
        "roofline": {"bound": "hbm", "achieved": round(gbs_gemm, 1), "peak": PEAK["hbm"], "unit": "GB/s",
                     "frac": round(gbs_gemm / PEAK["hbm"], 4),
                     "traffic": profiled_traffic_file("gemm_skinny_%s_workload%d_traffic.txt" % (w.fmt, args.workload),
                                                      "skinny"),
                     "kernel": "gemm_skinny_kernel on the packed weight image (%s W4A4 GEMM, M <= 64; "
                               "algorithmic bytes %d)" % (w.fmt, int(gemm_bytes))},
        "kernels": {"linear_step_rowmajor": {"ms": round(ms_step_rowmajor, 4),
                                             "GB/s": round(step_bytes / (ms_step_rowmajor * 1e-3) / 1e9, 1),
                                             "note": "context: the same step from the row-major weights "
                                                     "(reqat_linear_w4a4), per step in the graph"},
                    "gemm_rowmajor": {"ms": round(ms_gemm_rowmajor, 4),
                                      "GB/s": round(gemm_bytes / (ms_gemm_rowmajor * 1e-3) / 1e9, 1),
                                      "note": "context: the product from the row-major weights (reqat_gemm_w4a4), "
                                              "per launch in the graph"},
                    "linear_step_eager": {"ms": round(ms_eager, 4), "device_ms": round(ms_dev, 4),
                                          "GB/s": round(step_bytes / (ms_eager * 1e-3) / 1e9, 1),
                                          "note": "context: eager launches from Python (bound by the launch "
                                                  "rate); wall clock and HIP-event time per step"},
                    "gemm": {"ms": round(ms_gemm, 4), "GB/s": round(gbs_gemm, 1),
                             "TFLOP/s": round(2.0 * M * N * K / (ms_gemm * 1e-3) / 1e12, 2),
                             "note": "product alone on the packed image over the weight copies, %d launches in one HIP graph, "
                                     "per launch (HIP events around the replays)" % ncp},
                    "cache_resident_step": {"ms": round(ms_resident, 4),
                                            "GB/s": round(step_bytes / (ms_resident * 1e-3) / 1e9, 1),
                                            "note": "context only: the same weights every step (Infinity-Cache "
                                                    "resident after the first)"}},
    }
    out["ceilings"] = practical_ceilings()
    if not args.no_cpu_baseline:
        with pinned_to_one_core():
            import oracle
            ofmt = oracle.FMT_NVFP4 if fmt == reqat.NVFP4 else oracle.FMT_MXFP4
            xb, wb = wl.bf16_bits(x_cpu), wl.bf16_bits(w_cpu)
            t0 = time.perf_counter()
            owc, ows, owg = oracle.quantize(ofmt, wb[:256])
            oxc, oxs, oxg = oracle.quantize(ofmt, xb)
            n = 0
            while time.perf_counter() - t0 < 10.0:
                oracle.gemm(ofmt, oxc, oxs, oxg, owc, ows, owg)
                n += 1
            dt = time.perf_counter() - t0
            per_row = dt / (n * 256)                      # seconds per weight row of the product (+ quantize share)
            full = per_row * N
            out["cpu_baseline"] = {
                "value": round(step_bytes / full / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
                "sample": ("oracle quantize of X and of 256 weight rows, then the FP64 product against those "
                           "rows repeated for ~10 s (%d passes); per-row rate scaled to all %d rows" % (n, N))}
    print(json.dumps(out), flush=True)


def bench_kv4(args, w):
    """KV4 cache quantization of post-RoPE keys with the calibrated channel
    shift subtracted first (E1M2 codes, E4M3 block scales of 16, computed FP32
    tensor scale).  Bound by HBM: the keys are read once, codes and scales written."""
    import numpy as np
    import torch

    from paper_2606_15682_amd import reqat
    from paper_2606_15682_amd import workloads as wl

    reqat.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    T, C = w.M, w.K
    k_cpu, mu_cpu = wl.make_keys(w)
    k0, mu = k_cpu.to(dev), mu_cpu.to(dev)
    # rotate through copies of the keys (> 512 MB in all): every step reads them from HBM
    ncp = n_copies(T * C * 2, args)
    keys = [k0.clone() for _ in range(ncp)]
    k = k0
    codes = torch.empty((T, C // 2), dtype=torch.uint8, device=dev)
    scales = torch.empty((T, C // 16), dtype=torch.uint8, device=dev)
    g = torch.empty(1, dtype=torch.float32, device=dev)
    fq = torch.empty_like(k)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e[0].record()
        for _ in range(args.steps):
            fn()
        e[1].record()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / args.steps, e[0].elapsed_time(e[1]) / args.steps

    # A KV4 call is tens of microseconds of device work, close to what an eager
    # call from Python costs, so eager calls leave the GPU idle between them.
    # value = the call captured ncp times in one HIP graph (each on its own key
    # copy), per call, as a serving loop captures it; eager calls are context.
    ms_eager, ms_eager_dev = timed_rotation(
        lambda i: reqat.quantize_kv4(keys[i], mu, out=(codes, scales), g_out=g), ncp, args)
    ms_q = graph_rotation_ms(lambda i: reqat.quantize_kv4(keys[i], mu, out=(codes, scales), g_out=g), ncp, args)
    ms_step = ms_q
    gq = g.clone()
    ms_given = graph_rotation_ms(lambda i: reqat.quantize_kv4(keys[i], mu, tensor_scale=gq, out=(codes, scales)),
                                 ncp, args)
    ms_fq = graph_rotation_ms(lambda i: reqat.fakequant_kv4(keys[i], mu, out=fq, g_out=g), ncp, args)
    _, ms_resident = timed(lambda: reqat.quantize_kv4(k, mu, out=(codes, scales), g_out=g))
    q_bytes = T * C * (2 + 0.5 + 1.0 / 16)                        # read keys, write codes + scales
    fq_bytes = T * C * 4.0
    gbs = lambda b, ms: b / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(gbs(q_bytes, ms_step), 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded; N(0,1) keys plus per-channel offsets N(0,2), the offsets given as the shift)",
        "config": {"workload": w.name, "tokens": T, "channels": C, "global_batch": T,
                   "parallelism": "single GPU",
                   "step": "KV4 quantize of keys - shift (computed tensor scale: one pass over the keys + fix-up), each "
                           "step on another of %d key copies (%.0f MB in all, twice the Infinity Cache); the %d "
                           "steps captured in one HIP graph, time per step" % (ncp, ncp * T * C * 2 / 1e6, ncp)},
        "roofline": {"bound": "hbm", "achieved": round(gbs(q_bytes, ms_q), 1), "peak": PEAK["hbm"],
                     "unit": "GB/s", "frac": round(gbs(q_bytes, ms_q) / PEAK["hbm"], 4),
                     "traffic": profiled_traffic_file("kv4_workload%d_traffic.txt" % args.workload, "kv4"),
                     "kernel": "kv4_quantize_deferred_kernel + kv4_fixup_kernel (algorithmic bytes %d)" % int(q_bytes)},
        "kernels": {"quantize_kv4_computed_g": {"ms": round(ms_q, 4), "GB/s": round(gbs(q_bytes, ms_q), 1)},
                    "quantize_kv4_given_g": {"ms": round(ms_given, 4), "GB/s": round(gbs(q_bytes, ms_given), 1)},
                    "fakequant_kv4_computed_g": {"ms": round(ms_fq, 4), "GB/s": round(gbs(fq_bytes, ms_fq), 1)},
                    "quantize_kv4_computed_g_eager": {"ms": round(ms_eager, 4), "device_ms": round(ms_eager_dev, 4),
                                                      "GB/s": round(gbs(q_bytes, ms_eager), 1),
                                                      "note": "context: eager calls from Python, wall clock and "
                                                              "HIP-event time per call"},
                    "cache_resident_computed_g": {"ms": round(ms_resident, 4),
                                                  "GB/s": round(gbs(q_bytes, ms_resident), 1),
                                                  "note": "context only: the same keys every step"}},
    }
    out["ceilings"] = practical_ceilings()
    if not args.no_cpu_baseline:
        with pinned_to_one_core():
            import oracle
            rows = 2048
            kb = wl.bf16_bits(k_cpu[:rows])
            t0 = time.perf_counter()
            n = 0
            while time.perf_counter() - t0 < 10.0:
                oracle.kv4_quantize(kb, mu_cpu.numpy())
                n += 1
            dt = (time.perf_counter() - t0) / n
            out["cpu_baseline"] = {
                "value": round(rows * C * (2 + 0.5 + 1.0 / 16) / dt / 1e9, 4), "unit": "GB/s", "cores": 1,
                "kind": "oracle",
                "sample": "oracle KV4 quantize (computed g) of %d of the %d token rows, repeated for ~10 s (%d passes), "
                          "credited with the same bytes per row as the GPU step" % (rows, T, n)}
    print(json.dumps(out), flush=True)


def bench_sem(args, w):
    """QAT loss head: SEM loss forward and backward (bfloat16 gradient) over
    T x V bfloat16 logits.  Bound by HBM: the logits are read twice and the
    gradient written once."""
    import numpy as np
    import torch

    from paper_2606_15682_amd import reqat
    from paper_2606_15682_amd import workloads as wl

    reqat.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    T, V = w.M, w.N
    z_cpu, t_cpu = wl.make_logits(w)
    z, t = z_cpu.to(dev), t_cpu.to(dev)
    grad = torch.empty_like(z)
    lam = 0.5

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        loss, stats, weights = reqat.sem_loss(z, t, lam)
        if ev is not None:
            ev[1].record()
        reqat.sem_loss_backward(z, t, stats, weights, lam, 1.0, out_dtype=torch.bfloat16, out=grad)
        if ev is not None:
            ev[2].record()

    for _ in range(args.warmup):
        step()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    fwd = float(np.mean([e[0].elapsed_time(e[1]) for e in events]))
    bwd = float(np.mean([e[1].elapsed_time(e[2]) for e in events]))
    b_fwd, b_bwd = T * V * 2.0, T * V * 4.0
    gbs_bwd = b_bwd / (bwd * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round((b_fwd + b_bwd) / (ms_step * 1e-3) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded; logits N(0, 3) in bfloat16, uniform targets)",
        "config": {"workload": w.name, "tokens": T, "vocab": V, "global_batch": T, "parallelism": "single GPU",
                   "step": "SEM loss forward + backward (bfloat16 gradient)"},
        "roofline": {"bound": "hbm", "achieved": round(gbs_bwd, 1), "peak": PEAK["hbm"], "unit": "GB/s",
                     "frac": round(gbs_bwd / PEAK["hbm"], 4),
                     "traffic": profiled_traffic_file("sem_workload%d_traffic.txt" % args.workload, "sem"),
                     "kernel": "sem_backward_kernel (reads T*V*2 B of logits, writes T*V*2 B of gradient)"},
        "kernels": {"sem_forward": {"ms": round(fwd, 4), "GB/s": round(b_fwd / (fwd * 1e-3) / 1e9, 1)},
                    "sem_backward": {"ms": round(bwd, 4), "GB/s": round(gbs_bwd, 1)}},
    }
    out["ceilings"] = practical_ceilings()
    if not args.no_cpu_baseline:
        with pinned_to_one_core():
            import oracle
            rows = 64
            zb = wl.bf16_bits(z_cpu[:rows])
            t0 = time.perf_counter()
            n = 0
            while time.perf_counter() - t0 < 10.0:
                H, nll, lse = oracle.sem_row_stats(zb, t_cpu[:rows].numpy())
                _, _, _, wts = oracle.sem_loss(H, nll, lam, 1e-6)
                oracle.sem_grad(zb, t_cpu[:rows].numpy(), H, lse, wts, lam)
                n += 1
            dt = (time.perf_counter() - t0) / n
            out["cpu_baseline"] = {
                "value": round(rows * V * 6.0 / dt / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
                "sample": "FP64 numpy oracle: loss and gradient of %d of the %d token rows, repeated for ~10 s "
                          "(%d passes), credited with the same bytes per row as the GPU step" % (rows, T, n)}
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.copy_bytes:
        copy_calibration(args.copy_bytes, args.steps)
        return

    import numpy as np
    import torch

    from paper_2606_15682_amd import reqat
    from paper_2606_15682_amd import workloads as wl

    reqat.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = wl.WORKLOADS[args.workload]
    if w.kind == "w4a16":
        bench_w4a16(args, w)
        return
    if w.kind == "sem":
        bench_sem(args, w)
        return
    if w.kind == "kv4":
        bench_kv4(args, w)
        return
    if args.workload in DECODE_WORKLOADS:
        bench_decode(args, w)
        return
    fmt = reqat.NVFP4 if w.fmt == "nvfp4" else reqat.MXFP4
    B = reqat.BLOCK[fmt]
    x_cpu, w_cpu = wl.make_x(w), wl.make_w(w)
    x = x_cpu.to(dev)
    wt = w_cpu.to(dev)
    M, N, K = w.M, w.N, w.K

    xc = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
    xs = torch.empty((M, K // B), dtype=torch.uint8, device=dev)
    wc = torch.empty((N, K // 2), dtype=torch.uint8, device=dev)
    wsc = torch.empty((N, K // B), dtype=torch.uint8, device=dev)
    gx = torch.empty(1, dtype=torch.float32, device=dev) if fmt == reqat.NVFP4 else None
    gw = torch.empty(1, dtype=torch.float32, device=dev) if fmt == reqat.NVFP4 else None
    gfx = torch.empty(1, dtype=torch.float32, device=dev) if fmt == reqat.NVFP4 else None
    gfw = torch.empty(1, dtype=torch.float32, device=dev) if fmt == reqat.NVFP4 else None
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    fx = torch.empty_like(x)
    fw = torch.empty_like(wt)
    names = ["quantize_fakequant_x", "quantize_fakequant_w", "gemm"]

    def step(ev=None):
        # X and W each quantized (codes for the product) and fake-quantized
        # (the QAT forward's bfloat16 values) in one pass over the input
        def mark(i):
            if ev is not None:
                ev[i].record()
        mark(0)
        reqat.quantize_fakequant(x, fmt, out=(xc, xs, fx), g_out=gx)
        mark(1)
        reqat.quantize_fakequant(wt, fmt, out=(wc, wsc, fw), g_out=gw)
        mark(2)
        reqat.gemm(fmt, xc, xs, gx, wc, wsc, gw, out_dtype=torch.bfloat16, out=y)
        mark(3)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    per = {n: float(np.mean([events[i][j].elapsed_time(events[i][j + 1]) for i in range(args.steps)]))
           for j, n in enumerate(names)}
    # the product's operand data for the matrix-core probe (context, below):
    # MXFP4 feeds its packed codes; NVFP4 feeds FP16 code * scale, which is the
    # fake-quant value over the power-of-two g
    if M > 64:
        if fmt == reqat.MXFP4:
            probe_ops, probe_kind = operand_words(xc, wc), 0
        else:
            probe_ops = operand_words((fx.float() / gx).to(torch.float16), (fw.float() / gw).to(torch.float16))
            probe_kind = 1

    # the separate entry points (quantize alone, fake-quant alone), timed apart
    def timed(fn):
        for _ in range(max(1, args.warmup)):
            fn()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        e[0].record()
        for _ in range(args.steps):
            fn()
        e[1].record()
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / args.steps
    per["quantize_x"] = timed(lambda: reqat.quantize(x, fmt, out=(xc, xs), g_out=gx))
    per["quantize_w"] = timed(lambda: reqat.quantize(wt, fmt, out=(wc, wsc), g_out=gw))
    per["fakequant_x"] = timed(lambda: reqat.fakequant(x, fmt, out=fx, g_out=gfx))
    per["fakequant_w"] = timed(lambda: reqat.fakequant(wt, fmt, out=fw, g_out=gfw))

    # the same activation quantize + product through the one-call linear entry
    # point (a kernel right before the product on the same stream), timed apart
    lws = torch.empty(reqat.reqat_linear_workspace_bytes(fmt, M, K), dtype=torch.uint8, device=dev)
    gl = torch.empty(1, dtype=torch.float32, device=dev) if fmt == reqat.NVFP4 else None
    for _ in range(max(1, args.warmup)):
        reqat.linear(x, fmt, wc, wsc, gw, out_dtype=torch.bfloat16, out=y, g_out=gl, ws=lws)
    lev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    lev[0].record()
    for _ in range(args.steps):
        reqat.linear(x, fmt, wc, wsc, gw, out_dtype=torch.bfloat16, out=y, g_out=gl, ws=lws)
    lev[1].record()
    torch.cuda.synchronize()
    linear_ms = lev[0].elapsed_time(lev[1]) / args.steps

    graph_ms = None if args.no_graph else graph_step_ms(step, args)

    # MXFP4: the block-rotated activation quantizer (randomized Hadamard of 32
    # fused into the quantizer), timed apart from the step
    rht_ms = None
    if fmt == reqat.MXFP4:
        signs = 0x6C8E9CF5
        for _ in range(max(1, args.warmup)):
            reqat.quantize_rht(x, signs, out=(xc, xs))
        rev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        rev[0].record()
        for _ in range(args.steps):
            reqat.quantize_rht(x, signs, out=(xc, xs))
        rev[1].record()
        torch.cuda.synchronize()
        rht_ms = rev[0].elapsed_time(rev[1]) / args.steps

    flops = 2.0 * M * N * K
    q_bytes = lambda rows: rows * K * (2 + 0.5 + 1.0 / B)        # read bf16, write codes + scales
    fq_bytes = lambda rows: rows * K * 4.0                        # read bf16, write bf16
    qfq_bytes = lambda rows: rows * K * (4 + 0.5 + 1.0 / B)      # read bf16, write codes + scales + bf16
    gemm_tflops = flops / (per["gemm"] * 1e-3) / 1e12
    mfma_dtype = "f16" if fmt == reqat.NVFP4 else "fp4"
    kern = {
        "gemm": {"ms": round(per["gemm"], 4), "TFLOP/s": round(gemm_tflops, 1),
                 "frac_fp4_peak": round(gemm_tflops / PEAK["fp4"], 4),
                 "frac_own_mfma_peak": round(gemm_tflops / PEAK[mfma_dtype], 4)},
    }
    for n, rows, fn in (("quantize_fakequant_x", M, qfq_bytes), ("quantize_fakequant_w", N, qfq_bytes),
                        ("quantize_x", M, q_bytes), ("quantize_w", N, q_bytes),
                        ("fakequant_x", M, fq_bytes), ("fakequant_w", N, fq_bytes)):
        gbs = fn(rows) / (per[n] * 1e-3) / 1e9
        kern[n] = {"ms": round(per[n], 4), "GB/s": round(gbs, 1),
                   "frac_hbm_peak": round(gbs / PEAK["hbm"], 4),
                   "note": ("one pass + scale fix-up kernel (computed g); credited bytes = read x + writes"
                            if fmt == reqat.NVFP4 else "credited bytes = read x + writes")
                           + ("" if n.startswith("quantize_fakequant") else "; timed apart, not in the step")}

    if M <= 64:
        # few activation rows (the tiny workload): the product streams the weights once
        gemm_bytes = (N + M) * K * (0.5 + 1.0 / B) + M * N * 2.0
        gbs = gemm_bytes / (per["gemm"] * 1e-3) / 1e9
        kern["gemm"]["GB/s"] = round(gbs, 1)
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK["hbm"], "unit": "GB/s",
                    "frac": round(gbs / PEAK["hbm"], 4),
                    "traffic": profiled_traffic_file("gemm_skinny_%s_workload%d_traffic.txt"
                                                     % (w.fmt, args.workload), "skinny"),
                    "kernel": "gemm_skinny_kernel (%s W4A4 GEMM, M <= 64; algorithmic bytes %d)"
                              % (w.fmt, int(gemm_bytes))}
    else:
        roofline = {"bound": "mfma", "achieved": round(gemm_tflops, 2), "peak": PEAK[mfma_dtype],
                    "unit": "TFLOP/s", "frac": round(gemm_tflops / PEAK[mfma_dtype], 4),
                    "traffic": profiled_traffic(w.fmt, args.workload),
                    "kernel": "gemm_tile256_kernel (%s W4A4 GEMM)" % w.fmt}
    if rht_ms is not None:
        gbs = q_bytes(M) / (rht_ms * 1e-3) / 1e9
        kern["quantize_x_rotated"] = {"ms": round(rht_ms, 4), "GB/s": round(gbs, 1),
                                      "frac_hbm_peak": round(gbs / PEAK["hbm"], 4),
                                      "note": "block-rotated MXFP4 quantize of X (Hadamard 32), timed apart"}
    kern["linear"] = {"ms": round(linear_ms, 4),
                      "vs_quantize_x_plus_gemm": round(linear_ms / (per["quantize_x"] + per["gemm"]), 4),
                      "note": "reqat_linear_w4a4: quantize X + GEMM in one call, timed separately"}
    if graph_ms is not None:
        kern["graph_step"] = {"ms": round(graph_ms, 4), "vs_eager_step": round(graph_ms / ms_step, 4),
                              "note": "the same step captured once in a HIP graph and replayed (no launch gaps "
                                      "between its kernels); value and ms_per_step use the eager launches"}
    out = {
        "metric": METRIC,
        "value": round(flops / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": mfma_dtype,
        "data": "synthetic (seeded; Gaussian activations with 1% x20 outlier channels, N(0,0.02) weights)",
        "config": {"workload": w.name, "M": M, "N": N, "K": K, "format": w.fmt,
                   "gemm_out": "bf16", "global_batch": M, "parallelism": "single GPU",
                   "step": "quantize + fake-quant X, quantize + fake-quant W (one pass each, "
                           "dynamic global scales) + W4A4 GEMM"},
        "roofline": roofline,
        "kernels": kern,
    }
    out["ceilings"] = practical_ceilings(x, wt)
    if M > 64:
        kind = probe_kind
        probe = mfma_probe_tflops(kind, probe_ops)
        out["ceilings"]["mfma_probe"] = {
            "TFLOP/s": round(probe, 1), "frac_of_nominal_peak": round(probe / PEAK[mfma_dtype], 4),
            "gemm_frac_of_probe": round(gemm_tflops / probe, 4),
            "note": "register-only %s MFMA loop at one wave per SIMD on the first 4 KB of each operand "
                    "(libreqat_probe.so): what the matrix cores sustain on this data with no memory traffic"
                    % ("scaled FP4 32x32x64" if kind == 0 else "FP16 32x32x16")}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, wl.bf16_bits(x_cpu), wl.bf16_bits(w_cpu))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
