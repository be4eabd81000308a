#!/usr/bin/env python3
"""Benchmark of the fused W4A16 matmul on one MI355X.

One step = one pass of the hot path over the Llama-3-8B MLP shapes, synthetic
seeded data (weights pre-packed offline, inputs resident in HBM):
  * prefill GEMM  M=2048, K=4096,  N=14336, group 128  (up-projection shape)
  * prefill GEMM  M=2048, K=14336, N=4096,  group 128  (down-projection shape)
  * decode GEMV   M=1,    K=4096,  N=14336, group 128, repeated over
    GEMV_REPS distinct weight copies (one token through GEMV_REPS layers), so
    every GEMV streams its weights from HBM, not from the 256 MB MALL.

Prints ONE JSON line.  `value` is the prefill GEMM throughput in TFLOP/s
(2*M*N*K per GEMM over the GEMM kernels' time); the decode GEMV's effective
HBM bandwidth (packed codes + fp16 scales + zero-points per launch over its
average launch time) is reported beside it, each with its roofline fraction.
Kernel times come from HIP events recorded on the launch stream.

`roofline.traffic` is the HBM bytes per launch measured with rocprofv3
FETCH_SIZE / WRITE_SIZE counters (scaled by the same counters on a plain copy
of known size, see --calibrate-copy), recorded in profiles/traffic.json with
the hash of the kernel source they were taken on; it is null whenever that
source has changed since.
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
GEMM_SHAPES = [(2048, 4096, 14336), (2048, 14336, 4096)]
GEMV_SHAPE = (1, 4096, 14336)
GROUP = 128
GEMV_REPS = 32
# 17 copies of each prefill weight (17 x 30.7 MB = 522 MB, more than twice the
# 256 MB MALL), so the timed GEMMs stream their weights from HBM
GEMM_COPIES = 17
# The warm-up runs the W steps it is given and then replays the timed graphs
# until at least this much wall time has passed: the GPU clock takes tens of
# milliseconds of full load to settle, and a warm-up of a few steps (a few
# milliseconds) leaves the first timed launches slower.
WARM_FLOOR_S = 0.3
# The sweeps replay each workload's graph for at least this long before
# timing it, for the same reason.
SWEEP_WARM_S = 0.15
PEAK_F16_TFLOPS = 2516.6      # 256 CU x 4096 FLOP/clk x 2.4 GHz (dense fp16 or bf16 MFMA)
PEAK_HBM_GBS = 8000.0
COPY_BYTES = 1 << 30


def algo_bytes_w4(K, N, G=GROUP):
    """Bytes the method must move per launch: packed 4-bit codes, fp16 scales
    and 4-bit zero-points (the AWQ storage), activations and output excluded."""
    return K * N // 2 + (K // G) * N * 2 + (K // G) * N // 2


def source_hash(name):
    """SHA-256 (first 16 hex digits) of a kernel source and the shared header."""
    h = hashlib.sha256()
    for f in (name, "tf_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2606_11357_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel_file):
    """Per-launch HBM bytes from profiles/traffic.json if taken on this source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        rec = json.load(open(path))[kernel_file]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source_sha256_16") != source_hash(kernel_file):
        return None
    return rec.get("bytes_per_launch")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--context", action="store_true",
                    help="reference points only: dense fp16 torch.matmul on the prefill shapes and a "
                         "device copy of the decode GEMV's byte count")
    ap.add_argument("--mlp", action="store_true",
                    help="Llama-3-8B MLP composite (gate/up GEMM, silu*up, down GEMM) per stage and whole")
    ap.add_argument("--msweep", action="store_true",
                    help="the M sweep (256..8192 step 256) at both Llama MLP shapes, one JSON line each")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the step, time every synthetic workload configuration "
                         "(one JSON line each)")
    ap.add_argument("--rows", default=None,
                    help="with --msweep: only these row counts (comma-separated, 1..8192)")
    ap.add_argument("--workload", default=None,
                    help="with --sweep: only this workload (a name of synth.WORKLOADS)")
    ap.add_argument("--dtype", default=None, choices=("f16", "bf16"),
                    help="with --sweep or --mlp: only this activation dtype")
    return ap.parse_args()


CPU_CONFIGS = [
    # (name, bits, M, K, N, x_std, repeats): the five synthetic workloads;
    # median of 3 for the small ones, one run for the prefill shapes
    ("C0 W4 GEMM M=16 K=2048 N=2048", 4, 16, 2048, 2048, 1.0, 3),
    ("C1 W4 GEMV M=1 K=4096 N=14336", 4, 1, 4096, 14336, 1.0, 3),
    ("C1 W4 GEMV M=4 K=4096 N=14336", 4, 4, 4096, 14336, 1.0, 3),
    ("C1 W4 GEMV M=8 K=4096 N=14336", 4, 8, 4096, 14336, 1.0, 3),
    ("C2 W8 GEMV M=1 K=4096 N=4096", 8, 1, 4096, 4096, 1.0, 3),
    ("C2 W8 GEMM M=512 K=4096 N=4096", 8, 512, 4096, 4096, 1.0, 3),
    ("C3a W4 GEMM M=2048 K=4096 N=14336", 4, 2048, 4096, 14336, 1.0, 1),
    ("C3b W4 GEMM M=2048 K=14336 N=4096", 4, 2048, 14336, 4096, 1.0, 1),
    ("C4a W4 GEMM M=1024 K=4096 N=32768", 4, 1024, 4096, 32768, 0.5, 1),
    ("C4b W4 GEMM M=1024 K=32768 N=8192", 4, 1024, 32768, 8192, 0.5, 1),
]
ONE_THREAD = ("C0 W4 GEMM M=16 K=2048 N=2048", "C1 W4 GEMV M=1 K=4096 N=14336")


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_times(oracle, d, reps):
    """Median seconds of the oracle's two stages on one workload: unpack +
    dequant (Eq. 2 in float64) and the float64 matmul."""
    td, tm = [], []
    for _ in range(reps):
        t0 = time.perf_counter()
        if d["bits"] == 4:
            q, z = oracle.unpack_w4(d["qweight"]), oracle.unpack_w4(d["qzeros"])
        else:
            q, z = d["qweight"], d["zeros"]
        w = oracle.dequant(q, z, d["s"], GROUP)
        t1 = time.perf_counter()
        y = oracle.matmul(d["x"], w)
        t2 = time.perf_counter()
        assert np.isfinite(y).all()
        del w, y, q, z
        td.append(t1 - t0)
        tm.append(t2 - t1)
    return float(np.median(td)), float(np.median(tm))


def cpu_baseline():
    """The oracle (numpy: unpack, Eq. 2 in float64, float64 BLAS matmul) timed
    on this host on every synthetic workload: dequant and matmul separately,
    median of 3 runs for the small workloads and one run for the prefill
    shapes, with all BLAS threads; a one-thread figure for the M=16 GEMM and
    the M=1 GEMV.  `value` is the prefill GEMM pair's rate (the headline
    metric's workload): 2*M*N*K of both shapes over their oracle time."""
    import oracle
    from paper_2606_11357_amd.synth import make_inputs
    from threadpoolctl import threadpool_info, threadpool_limits
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    per = {}
    t_total = 0.0
    for name, bits, M, K, N, xstd, reps in CPU_CONFIGS:
        d = make_inputs(bits, M, K, N, group=GROUP, seed=0, x_std=xstd)
        tdq, tmm = _oracle_times(oracle, d, reps)
        flops = 2.0 * M * N * K
        rec = {"dequant_s": round(tdq, 4), "matmul_s": round(tmm, 4), "runs": reps,
               "GFLOP/s": round(flops / (tdq + tmm) / 1e9, 3),
               "GB/s": round(algo_bytes(bits, K, N) / (tdq + tmm) / 1e9, 3)}
        t_total += reps * (tdq + tmm)
        if name in ONE_THREAD:
            with threadpool_limits(limits=1):
                t1d, t1m = _oracle_times(oracle, d, reps)
            rec["one_thread"] = {"dequant_s": round(t1d, 4), "matmul_s": round(t1m, 4),
                                 "GFLOP/s": round(flops / (t1d + t1m) / 1e9, 3)}
            t_total += reps * (t1d + t1m)
        per[name] = rec
        del d
    pair = [per[n] for n in ("C3a W4 GEMM M=2048 K=4096 N=14336", "C3b W4 GEMM M=2048 K=14336 N=4096")]
    t_pair = sum(r["dequant_s"] + r["matmul_s"] for r in pair)
    flops_pair = sum(2.0 * M * N * K for (M, K, N) in GEMM_SHAPES)
    return {"value": round(flops_pair / t_pair / 1e12, 4), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "cpu_model": _cpu_model(), "os_cpu_count": os.cpu_count(),
            "blas_threads": int(threads), "seconds": round(t_total, 2),
            "sample": "every synthetic workload once through the oracle (unpack + float64 dequant, "
                      "then float64 BLAS matmul; median of 3 runs below M=2048, one run at M>=1024); value "
                      "= the M=2048 prefill pair, both stages",
            "per_config": per}


def calibrate_copy(torch):
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read": COPY_BYTES,
                      "bytes_written": COPY_BYTES, "launches": 3}), flush=True)


def algo_bytes(bits, K, N, G=GROUP):
    """Packed codes + fp16 scales + zero-points (4-bit packed, 8-bit as bytes)."""
    if bits == 4:
        return algo_bytes_w4(K, N, G)
    return K * N + (K // G) * N * 2 + (K // G) * N


def sweep(torch, tf, make_inputs, reps=50, dtypes=("f16", "bf16"), only=None):
    """Every workload of synth.WORKLOADS, with fp16 and with BF16 activations
    and scales: HIP-event time per launch over 3 replays of a graph of `reps`
    launches rotating over enough distinct copies of the packed weight that
    the copies exceed 512 MB (so weights stream from HBM, not the MALL), the
    library's default workspace, inputs resident."""
    from paper_2606_11357_amd.synth import WORKLOADS, make_inputs_bf16
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    if only is not None and only not in WORKLOADS:
        raise SystemExit(f"unknown workload {only}; one of {', '.join(WORKLOADS)}")
    for dt in dtypes:
        for name, (bits, Ms, K, N, xstd) in WORKLOADS.items():
            if only is not None and name != only:
                continue
            for M in Ms:
                if dt == "bf16":
                    d = make_inputs_bf16(bits, M, K, N, group=GROUP, seed=0, x_std=xstd)
                    s = up(d["s_bits"].view(np.int16))
                    x = up(d["x_bits"].view(np.int16)).view(torch.bfloat16)
                else:
                    d = make_inputs(bits, M, K, N, group=GROUP, seed=0, x_std=xstd)
                    s, x = up(d["s"]), up(d["x"])
                if bits == 4:
                    p0 = tf.pack_w4(up(d["qweight"]), up(d["qzeros"]), s, K, N, GROUP)
                else:
                    p0 = tf.pack_w8(up(d["qweight"]), up(d["zeros"]), s, K, N, GROUP)
                ncopy = int(min(40, max(2, -(-(512 << 20) // p0.numel()))))
                copies = [p0] + [p0.clone() for _ in range(ncopy - 1)]
                y = torch.empty((M, N), dtype=x.dtype, device=dev)
                # decode shapes go through both entry points (the GEMV is vector-ALU
                # only; the GEMM entry may use the matrix cores from 4 rows up)
                for entry in (("gemv", "gemm") if M <= tf.GEMV_MAX_M else ("gemm",)):
                    sweep_one(torch, tf, stream, name, entry, bits, M, K, N, x, y, copies, reps, dt)
                del copies, p0, x, y, d, s
                torch.cuda.empty_cache()


def warm_graph(torch, g, seconds=SWEEP_WARM_S):
    """Replay a captured graph until `seconds` of wall time have passed."""
    t0 = time.perf_counter()
    while True:
        g.replay()
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= seconds:
            return


def sweep_one(torch, tf, stream, name, entry, bits, M, K, N, x, y, copies, reps, dtype="f16"):
    fn = getattr(tf, f"w{bits}a16_{entry}")
    ncopy = len(copies)
    for i in range(5):
        fn(x, copies[i % ncopy], K, N, GROUP, out=y)
    torch.cuda.synchronize()
    # the launches are replayed from a HIP graph, so the host-side cost
    # of a Python call does not leave the GPU idle between small kernels
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(reps):
            fn(x, copies[i % ncopy], K, N, GROUP, out=y)
    warm_graph(torch, g)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(3):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (3 * reps)
    tflops = 2.0 * M * N * K / us / 1e6
    gbs = algo_bytes(bits, K, N) / us / 1e3
    hbm_bound = M <= 16
    print(json.dumps({
        "workload": name, "dtype": dtype, "entry": entry, "bits": bits, "M": M, "K": K, "N": N,
        "group": GROUP,
        "us_per_launch": round(us, 3), "TFLOP/s": round(tflops, 2), "GB/s": round(gbs, 1),
        "bound": "hbm" if hbm_bound else "mfma",
        "frac": round(gbs / PEAK_HBM_GBS if hbm_bound else tflops / PEAK_F16_TFLOPS, 4),
        "weight_copies": ncopy, "launches": 3 * reps, "timing": "HIP graph replay"}),
        flush=True)
    del g


def graph_time_us(torch, fn, reps):
    """Mean µs per call of fn() over 3 replays of a HIP graph of `reps` calls
    (after replaying it for SWEEP_WARM_S)."""
    stream = torch.cuda.current_stream()
    for _ in range(3):
        fn(0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(reps):
            fn(i)
    warm_graph(torch, g)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(3):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / (3 * reps)


PROBE_SHAPES = ((224, 1024, 8), (224, 1024, 4), (256, 1024, 8), (256, 1024, 4), (256, 512, 16),
                (512, 512, 8), (512, 1024, 4), (1024, 256, 8), (1024, 256, 16), (2048, 256, 4),
                (2048, 256, 8), (4096, 256, 2))
# the launch shapes that came out fastest for the decode GEMV's 30.5 MB
# (profiles/context_references.md), timed beside every benchmark line
PROBE_SHAPES_QUICK = ((224, 1024, 4), (4096, 256, 2), (2048, 256, 4))


def read_ceiling(torch, nbytes, reps=64, shapes=PROBE_SHAPES):
    """Streaming-read ceiling for a launch that reads `nbytes` once: the read
    probe (paper_2606_11357_amd/probe, a kernel that only loads) over a sweep
    of launch shapes, rotating over enough buffers to exceed 512 MB so every
    launch reads HBM; HIP-graph replay timing.  Returns one record per shape,
    fastest first."""
    import ctypes
    from paper_2606_11357_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.tf_probe_read.restype = ctypes.c_int
    lib.tf_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_void_p, ctypes.c_void_p]
    dev = torch.device("cuda:0")
    nbytes = nbytes // 16 * 16
    ncopy = -(-(512 << 20) // nbytes)
    bufs = [torch.ones(nbytes, device=dev, dtype=torch.uint8) for _ in range(ncopy)]
    sink = torch.zeros(4, device=dev, dtype=torch.int32)
    out = []
    for grid, block, unroll in shapes:
        def launch(i, g=grid, b=block, u=unroll):
            rc = lib.tf_probe_read(ctypes.c_void_p(bufs[i % ncopy].data_ptr()), nbytes, g, b, u,
                                   ctypes.c_void_p(sink.data_ptr()),
                                   ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            assert rc == 0, rc
        us = graph_time_us(torch, launch, reps)
        out.append({"grid": grid, "block": block, "unroll": unroll, "us_per_launch": round(us, 3),
                    "read_GB/s": round(nbytes / us / 1e3, 1)})
    del bufs
    return sorted(out, key=lambda r: r["us_per_launch"])


def context(torch):
    """Achievable-ceiling references, not targets: torch.matmul in fp16 (the
    weights already dequantized to a dense fp16 [K, N]) on the two prefill
    shapes; the streaming-read ceiling for the decode GEMV's byte count (a
    kernel that only reads, over a sweep of launch shapes); and a device copy
    of the same byte count, rotating over sources so it streams from HBM."""
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev).manual_seed(0)
    for (M, K, N) in GEMM_SHAPES:
        a = torch.randn((M, K), device=dev, dtype=torch.float16, generator=gen)
        ws = [torch.randn((K, N), device=dev, dtype=torch.float16, generator=gen) * 0.02 for _ in range(4)]
        out = torch.empty((M, N), device=dev, dtype=torch.float16)
        us = graph_time_us(torch, lambda i: torch.matmul(a, ws[i % 4], out=out), 20)
        print(json.dumps({"reference": "torch.matmul fp16 (hipBLASLt), dense fp16 weights", "M": M, "K": K,
                          "N": N, "us_per_launch": round(us, 3),
                          "TFLOP/s": round(2.0 * M * N * K / us / 1e6, 2)}), flush=True)
        del a, ws, out
    nbytes = algo_bytes_w4(GEMV_SHAPE[1], GEMV_SHAPE[2])
    for bytes_, what in ((nbytes, "the decode GEMV's metric bytes (K=4096 N=14336 W4)"),
                         (256 << 20, "256 MiB (asymptotic rate)")):
        shapes = read_ceiling(torch, bytes_)
        print(json.dumps({"reference": "streaming read (read-only probe kernel) of " + what, "bytes_read": bytes_,
                          "best": shapes[0], "gemv_like_grid_224x1024": [r for r in shapes if r["grid"] == 224][0],
                          "all_shapes": shapes}), flush=True)
    ncopy = -(-(512 << 20) // nbytes)
    bufs = [torch.empty(nbytes, device=dev, dtype=torch.uint8) for _ in range(ncopy)]
    dst = torch.empty(nbytes, device=dev, dtype=torch.uint8)
    us = graph_time_us(torch, lambda i: dst.copy_(bufs[i % ncopy]), 64)
    print(json.dumps({"reference": "device copy (torch copy_) of the decode GEMV's byte count",
                      "bytes_read": nbytes, "bytes_written": nbytes, "copies": ncopy,
                      "us_per_launch": round(us, 3), "read_GB/s": round(nbytes / us / 1e3, 1),
                      "read+write_GB/s": round(2 * nbytes / us / 1e3, 1)}), flush=True)


def mlp(torch, tf, make_inputs, Ms=(1, 16, 256, 2048, 8192), dtypes=("f16", "bf16")):
    """A Llama-3-8B MLP layer (hidden 4096, intermediate 14336) around the fused
    matmul: one W4A16 GEMM for gate and up (weights concatenated along N,
    N = 28672), tf_silu_mul, one W4A16 GEMM for down (K = 14336); synthetic
    weights, G = 128.  Each stage and the whole layer timed by HIP-graph
    replay (weights used in place: 4 bytes per parameter less than fp16, and
    the 90 MB of packed weights partly stay in the 256 MB MALL across
    replays).  Runs with fp16 and with BF16 activations and scales."""
    from paper_2606_11357_amd.synth import make_inputs_bf16
    dev = torch.device("cuda:0")
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    H, I = 4096, 14336
    for dt in dtypes:
        if dt == "bf16":
            gu = make_inputs_bf16(4, max(Ms), H, 2 * I, group=GROUP, seed=0)
            dn = make_inputs_bf16(4, 1, I, H, group=GROUP, seed=1)
            s_gu, s_dn = up(gu["s_bits"].view(np.int16)), up(dn["s_bits"].view(np.int16))
            xall = up(gu["x_bits"].view(np.int16)).view(torch.bfloat16)
        else:
            gu = make_inputs(4, max(Ms), H, 2 * I, group=GROUP, seed=0)
            dn = make_inputs(4, 1, I, H, group=GROUP, seed=1)
            s_gu, s_dn = up(gu["s"]), up(dn["s"])
            xall = up(gu["x"])
        p_gu = tf.pack_w4(up(gu["qweight"]), up(gu["qzeros"]), s_gu, H, 2 * I, GROUP)
        p_dn = tf.pack_w4(up(dn["qweight"]), up(dn["qzeros"]), s_dn, I, H, GROUP)
        del gu, dn, s_gu, s_dn
        mlp_layers(torch, tf, Ms, dt, xall, p_gu, p_dn, H, I)
        del xall, p_gu, p_dn
        torch.cuda.empty_cache()


def mlp_layers(torch, tf, Ms, dt, xall, p_gu, p_dn, H, I):
    dev = xall.device
    for M in Ms:
        x = xall[:M]
        g = torch.empty((M, 2 * I), dtype=x.dtype, device=dev)
        h = torch.empty((M, I), dtype=x.dtype, device=dev)
        y = torch.empty((M, H), dtype=x.dtype, device=dev)
        gemm_or_gemv = tf.w4a16_gemv if M <= tf.GEMV_MAX_M else tf.w4a16_gemm
        s1 = lambda i: gemm_or_gemv(x, p_gu, H, 2 * I, GROUP, out=g)
        s2 = lambda i: tf.silu_mul(g, out=h)
        s3 = lambda i: gemm_or_gemv(h, p_dn, I, H, GROUP, out=y)

        def layer(i):
            s1(i)
            s2(i)
            s3(i)
        flops = 2.0 * M * (H * 2 * I + I * H)
        reps = int(max(4, min(50, 5e-3 / max(flops / 1.0e15, 8e-6))))
        t = [graph_time_us(torch, f, reps) for f in (s1, s2, s3, layer)]
        print(json.dumps({"workload": "llama3_8b_mlp_w4a16", "dtype": dt, "M": M, "hidden": H, "intermediate": I,
                          "entry": "gemv" if M <= tf.GEMV_MAX_M else "gemm",
                          "us_gate_up": round(t[0], 3), "us_silu_mul": round(t[1], 3),
                          "us_down": round(t[2], 3), "us_layer": round(t[3], 3),
                          "TFLOP/s_layer": round(flops / t[3] / 1e6, 2),
                          "matmul_share": round((t[0] + t[2]) / (t[0] + t[1] + t[2]), 4),
                          "timing": "HIP graph replay"}), flush=True)
        del g, h, y
    torch.cuda.empty_cache()


def msweep(torch, tf, make_inputs, target_ms=6.0, rows=None):
    """The paper's prompt-length sweep: W4A16 GEMM for M = 256..8192 (step
    256, or the row counts in `rows`, each at most 8192) at (K, N) =
    (4096, 14336) and (14336, 4096).  Per shape one input draw at M = 8192
    (each M takes its first M rows of A) and enough copies of the packed
    weight to stream it from HBM; HIP-graph replay as in --sweep, with about
    `target_ms` of GPU time per graph."""
    from paper_2606_11357_amd.synth import M_SWEEP, M_SWEEP_SHAPES
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    for (K, N) in M_SWEEP_SHAPES:
        d = make_inputs(4, max(M_SWEEP), K, N, group=GROUP, seed=0)
        p0 = tf.pack_w4(up(d["qweight"]), up(d["qzeros"]), up(d["s"]), K, N, GROUP)
        ncopy = int(min(24, max(2, -(-(512 << 20) // p0.numel()))))
        copies = [p0] + [p0.clone() for _ in range(ncopy - 1)]
        xall = up(d["x"])
        del d
        for M in (rows or M_SWEEP):
            x = xall[:M]
            y = torch.empty((M, N), dtype=torch.float16, device=dev)
            flops = 2.0 * M * N * K
            reps = int(max(4, min(50, target_ms * 1e-3 / (flops / 1.0e15))))
            for i in range(3):
                tf.w4a16_gemm(x, copies[i % ncopy], K, N, GROUP, out=y)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(reps):
                    tf.w4a16_gemm(x, copies[i % ncopy], K, N, GROUP, out=y)
            warm_graph(torch, g)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(3):
                g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / (3 * reps)
            tflops = flops / us / 1e6
            print(json.dumps({"workload": "w4a16_gemm_msweep", "M": M, "K": K, "N": N, "group": GROUP,
                              "us_per_launch": round(us, 3), "TFLOP/s": round(tflops, 2),
                              "frac": round(tflops / PEAK_F16_TFLOPS, 4), "launches": 3 * reps,
                              "weight_copies": ncopy, "timing": "HIP graph replay"}), flush=True)
            del g, y
        del copies, p0, xall
        torch.cuda.empty_cache()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(nothing here runs across GPUs)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_11357_amd import tilefuse as tf
    from paper_2606_11357_amd.synth import make_inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_copy:
        calibrate_copy(torch)
        return
    if args.context:
        context(torch)
        return
    tf.load()
    dtypes = (args.dtype,) if args.dtype else ("f16", "bf16")
    if args.sweep:
        sweep(torch, tf, make_inputs, dtypes=dtypes, only=args.workload)
        return
    if args.msweep:
        rows = None
        if args.rows:
            rows = [int(r) for r in args.rows.split(",")]
            if any(r < 1 or r > 8192 for r in rows):
                sys.exit("--rows: row counts from 1 to 8192")
        msweep(torch, tf, make_inputs, rows=rows)
        return
    if args.mlp:
        mlp(torch, tf, make_inputs, dtypes=dtypes)
        return
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)

    def upload(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    def packed_w4(d):
        return tf.pack_w4(upload(d["qweight"]), upload(d["qzeros"]), upload(d["s"]),
                          d["K"], d["N"], GROUP)

    # ---- inputs (offline: generation + pack are outside the timed region);
    # GEMM_COPIES copies of each prefill weight (522 MB per shape, more than
    # twice the 256 MB MALL), so the GEMMs stream their weights from HBM
    gemm = []
    for (M, K, N) in GEMM_SHAPES:
        d = make_inputs(4, M, K, N, group=GROUP, seed=0)
        p = packed_w4(d)
        gemm.append(dict(M=M, K=K, N=N, A=upload(d["x"]), copies=[p] + [p.clone() for _ in range(GEMM_COPIES - 1)],
                         out=torch.empty((M, N), dtype=torch.float16, device=dev)))
        del d
    M1, K1, N1 = GEMV_SHAPE
    d = make_inputs(4, M1, K1, N1, group=GROUP, seed=0)
    p0 = packed_w4(d)
    gemv_copies = [p0] + [p0.clone() for _ in range(GEMV_REPS - 1)]
    x1 = upload(d["x"])
    y1 = torch.empty((M1, N1), dtype=torch.float16, device=dev)
    del d
    torch.cuda.synchronize()

    def gemm_one(g, c):
        tf.w4a16_gemm(g["A"], g["copies"][c], g["K"], g["N"], GROUP, out=g["out"])

    def gemv_batch():
        for p in gemv_copies:
            tf.w4a16_gemv(x1, p, K1, N1, GROUP, out=y1)

    # Each phase of the K timed steps is captured as ONE HIP
    # graph: the K launches of a prefill shape, rotating over its weight
    # copies, and the K decode GEMV batches.  Inside a graph the kernels
    # follow each other on the GPU without gaps; each graph replay costs a
    # launch gap of its own, which one replay per phase keeps out of the
    # per-kernel figures.
    gemm_one(gemm[0], 0)     # allocates the default workspace before capture
    torch.cuda.synchronize()
    graphs = []
    for g in gemm:
        cg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(cg):
            for s in range(args.steps):
                gemm_one(g, s % GEMM_COPIES)
        graphs.append(cg)
    g_gemv = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_gemv):
        for s in range(args.steps):
            gemv_batch()
    torch.cuda.synchronize()
    # Warm-up, right before the timed region (capture above leaves the GPU
    # idle, and its clock drops): the W steps as given, eagerly, then replays
    # of the timed graphs until WARM_FLOOR_S of wall time have passed.
    t_w = time.perf_counter()
    for s in range(args.warmup):
        for g in gemm:
            gemm_one(g, s % GEMM_COPIES)
        gemv_batch()
    torch.cuda.synchronize()
    warm_replays = 0
    while time.perf_counter() - t_w < WARM_FLOOR_S:
        for cg in graphs:
            cg.replay()
        g_gemv.replay()
        torch.cuda.synchronize()
        warm_replays += 1
    warm_s = time.perf_counter() - t_w

    # The timed region holds the K steps' work grouped by kernel: the K
    # launches of each prefill shape back to back (weights stream from HBM,
    # the shape's activations stay cache-resident as the previous layer's
    # output would), then the K decode GEMV batches.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(graphs) + 2)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i, cg in enumerate(graphs):
        cg.replay()
        ev[i + 1].record(stream)
    g_gemv.replay()
    ev[-1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    shape_ms = [ev[i].elapsed_time(ev[i + 1]) / args.steps for i in range(len(graphs))]
    gemm_ms = sum(shape_ms)
    gemv_ms = ev[-2].elapsed_time(ev[-1]) / args.steps
    gemm_flops = sum(2.0 * g["M"] * g["N"] * g["K"] for g in gemm)
    tflops = gemm_flops / (gemm_ms * 1e-3) / 1e12
    gemv_us = gemv_ms * 1e3 / GEMV_REPS
    gemv_bytes = algo_bytes_w4(K1, N1)
    gemv_gbs = gemv_bytes / (gemv_us * 1e-6) / 1e9
    # Context for the GEMV's fraction, measured after the timed region: the
    # streaming-read ceiling for its byte count on this GPU (a kernel that
    # only reads; the fastest of a few launch shapes).
    try:
        best = read_ceiling(torch, gemv_bytes, shapes=PROBE_SHAPES_QUICK)[0]
        ceiling = {"value": best["read_GB/s"], "unit": "GB/s", "us_per_launch": best["us_per_launch"],
                   "probe": "read-only kernel over the same byte count, grid %d x %d, %d loads in flight per "
                            "thread" % (best["grid"], best["block"], best["unroll"]),
                   "gemv_frac_of_ceiling": round(gemv_gbs / best["read_GB/s"], 4)}
    except Exception as e:    # e.g. the probe library is not built: the line is printed regardless
        ceiling = {"value": None, "reason": str(e)[:200]}

    line = {
        "metric": "W4A16 GEMM TFLOP/s (M=2048) + GEMV eff. HBM GB/s (M=1), % of roofline",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": "W4A16 (AWQ-style, G=128) prefill GEMM M=2048 at (K=4096,N=14336) and "
                        "(K=14336,N=4096) x%d weight copies + decode GEMV M=1 K=4096 N=14336 x%d "
                        "weight copies" % (GEMM_COPIES, GEMV_REPS),
            "group": GROUP,
            "weights": "4-bit codes, fp16 scales, 4-bit zero-points (seeded uniform)",
            "activations": "fp16 N(0,1)",
        },
        "roofline": {
            "bound": "mfma",
            "achieved": round(tflops, 2),
            "peak": PEAK_F16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tflops / PEAK_F16_TFLOPS, 4),
            "traffic": recorded_traffic("tf_gemm256.hip"),
            "kernel": "gemm256_kernel (the launch plan of each shape is named by TF_LOG=1 and the profiles)",
        },
        "gemv": {
            "value": round(gemv_gbs, 1),
            "unit": "GB/s",
            "us_per_launch": round(gemv_us, 3),
            "bytes_per_launch": gemv_bytes,
            "roofline": {"bound": "hbm", "achieved": round(gemv_gbs, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(gemv_gbs / PEAK_HBM_GBS, 4),
                         "traffic": recorded_traffic("tf_gemv.hip"), "kernel": "gemv_kernel"},
            "read_ceiling": ceiling,
        },
        "gemm_ms_per_step": round(gemm_ms, 4),
        "gemm_us_per_shape": {f"K={K},N={N}": round(t * 1e3, 2) for (M, K, N), t in zip(GEMM_SHAPES, shape_ms)},
        "warmup_s": round(warm_s, 3),
        "warmup_graph_replays": warm_replays,
        "timing": "HIP events on the launch stream around one graph replay per phase (K launches each); "
                  "value = 2*M*N*K of both prefill shapes over their summed mean launch time",
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
