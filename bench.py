"""Benchmark of the signed-symmetric W4 path on one MI355X.

One step is one pass of the whole path over one batch of synthetic input, on
the Llama3-8B down-projection shape (N=4096 outputs, K=14336, q=4, g=32,
signed symmetric scales):

  1. quantize the bf16 weight matrix (load, per-group absmax + sign, scale,
     round/clip, pack)                                   -> ssq_quantize
  2. decode: one GEMV (M=1) through each of ``--layers`` distinct quantized
     copies of that matrix, like one token through a stack of layers
                                                         -> ssq_matmul, M=1
  3. batched decode: M=16 tokens through each of the copies -> ssq_matmul, M=16
  4. prefill: a GEMM with M=512 tokens through ``--gemm-layers`` of the copies
                                                         -> ssq_matmul, M=512
  5. the decode GEMV on the Llama3-70B down-projection (8192x28672), through
     ``--layers70b`` quantized copies                    -> ssq_matmul, M=1

The layer copies total more than the 256 MB Infinity Cache, so the GEMV
streams its codes from HBM.  The GEMV and GEMM launches of a step are captured
once in a HIP graph and replayed (Python cannot issue microsecond kernels fast
enough to keep the GPU busy).  Each phase is bracketed by HIP events on the
stream its kernels run on; a kernel's average duration is the phase time over
its launches.  ``value`` is the decode GEMV's algorithmic HBM bandwidth (codes
+ scales + x + y bytes per launch over its average duration); the other phases
are reported beside it, each with its roofline.  The CPU oracle is timed first,
on one thread and on every host thread (up to 16), before the GPU is touched.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
       python bench.py --sweep      (format sweep: all Llama3-8B projections at every
                                     q, g and mode; the sign-rule diagnostics of that
                                     block; the prefill GEMM per mode; the Llama3-70B
                                     block at q=2; the Qwen3-8B and -14B blocks; a GEMV
                                     K-sweep -- one JSON line; --sweep-parts picks)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "W4 signed-sym decode GEMV HBM GB/s (% peak) + prefill GEMM TFLOP/s, 4096x14336"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, vendor figure
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_counters.json")
CSRC = os.path.join(ROOT, "paper_2607_08779_amd", "csrc")


def kernel_source_sha(files) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "gemv": ["gemv.hip", "ssq_internal.h"],
    "gemm": ["gemm.hip", "mfma_dequant.h", "ssq_internal.h"],
    "batched": ["skinny.hip", "mfma_dequant.h", "ssq_internal.h"],
    "quantize": ["quantize.hip", "ssq_internal.h"],
}


def measured_traffic(kind: str, mode: str = "signed_sym"):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None if absent,
    taken on a different version of the kernel's source, or on another mode."""
    if mode != "signed_sym":
        return None
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    entry = data.get(kind)
    if not entry or entry.get("source_sha") != kernel_source_sha(KERNEL_SOURCES[kind.split(":")[0]]):
        return None
    return entry.get("hbm_bytes_per_launch")


TRACE_FILE = os.path.join(ROOT, "profiles", "kernel_trace.json")


def traced_launch_us(kind: str, mode: str = "signed_sym"):
    """A kernel's average duration from the committed rocprofv3 kernel trace of this
    benchmark, or None if absent or taken on a different version of its source.  The
    trace times the kernel alone; the HIP events of the phases also hold the gaps
    between the graph's kernel nodes."""
    if mode != "signed_sym":
        return None
    try:
        with open(TRACE_FILE) as f:
            entry = json.load(f).get(kind)
    except (OSError, ValueError):
        return None
    if not entry or entry.get("source_sha") != kernel_source_sha(KERNEL_SOURCES[kind.split(":")[0]]):
        return None
    return entry.get("avg_us")


def add_trace_frac(roof: dict, kind: str, mode: str, work: float) -> None:
    """Put the trace-timed rate and fraction of peak beside the event-timed ones."""
    us = traced_launch_us(kind, mode)
    roof["trace_avg_launch_us"] = us
    if us is None:
        roof["trace_frac"] = None
        return
    rate = work / (us * 1e-6) / (1e9 if roof["unit"] == "GB/s" else 1e12)
    roof["trace_achieved"] = round(rate, 2)
    roof["trace_frac"] = round(rate / roof["peak"], 4)


def parse_args():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--layers", type=int, default=16, help="distinct quantized copies (decode depth)")
    p.add_argument("--gemm-layers", type=int, default=4, help="prefill GEMMs per step")
    p.add_argument("--gemm-m", type=int, default=512)
    p.add_argument("--mode", choices=["signed_sym", "unsigned_sym", "asym", "asym_min"], default="signed_sym")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--batched-m", type=int, default=16, help="tokens of the batched-decode phase")
    p.add_argument("--sweep", action="store_true",
                   help="format sweep over the Llama3 shapes instead of the headline step")
    p.add_argument("--sweep-parts", default="formats,diagnostics,q8,prefill,70b,qwen3,ksweep",
                   help="comma list of sweep parts: formats (8B block, every format), diagnostics "
                        "(sign-rule statistics of the 8B block), q8 (Q8_0 activations, integer "
                        "GEMV against the bf16 GEMV), prefill, 70b, qwen3 (Qwen3-8B and -14B "
                        "blocks), ksweep (W4 GEMV at N=4096 over K next to a streaming read)")
    p.add_argument("--phases", default="quantize,gemv,batched,gemm,gemv70b",
                   help="comma list of phases to run (profiling runs isolate one kernel); "
                        "gemv70b is the decode GEMV on the Llama3-70B down-projection "
                        "(8192x28672); 'copy' adds a plain 256 MiB device copy used to "
                        "calibrate byte counters")
    p.add_argument("--quantize-copies", type=int, default=3,
                   help="distinct weight matrices (and outputs) the quantize phase rotates over")
    p.add_argument("--layers70b", type=int, default=4,
                   help="distinct quantized copies of the 8192x28672 matrix (gemv70b phase)")
    return p.parse_args()


def _oracle_rows(args):
    """Quantize rows [lo, hi) of the bf16 matrix with the oracle and run its binary64 GEMV
    on them, `reps` times; returns (quantize seconds, GEMV seconds).  One thread."""
    w_bits, x_bits, lo, hi, K, g, q, mode, reps = args
    from threadpoolctl import threadpool_limits

    from oracle import ssq_oracle as O

    xf = O.bf16_bits_to_f32(x_bits)
    t_quant = t_gemv = 0.0
    with threadpool_limits(limits=1):
        for _ in range(reps):
            t0 = time.perf_counter()
            r = O.quantize(O.bf16_bits_to_f32(w_bits[lo:hi]), g, q, mode)
            t1 = time.perf_counter()
            O.matmul(xf, r.codes, r.scales, r.zp, hi - lo, K, g, q, mins=r.mins)
            t_quant += t1 - t0
            t_gemv += time.perf_counter() - t1
    return t_quant, t_gemv


def host_worker_count() -> int:
    """Host threads this process may run on, at most 16 (one GPU's share of the host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cpu_baseline(w_bits: np.ndarray, x_bits: np.ndarray, N: int, K: int, g: int, q: int,
                 mode: int, gemv_bytes_per_row: float, budget_s: float = 10.0) -> dict:
    """Time the CPU oracle on a bounded sample of the same workload, quantize + binary64
    GEMV, in two legs of about budget_s each: one thread on rows 0..2047, and every host
    thread (up to 16 processes, one thread each) on all rows, split into equal row slices.
    Must run before the process touches the GPU: the all-cores leg forks."""
    import multiprocessing as mp

    quant_bytes_per_row = K * (2 + q / 8 + 2 / g + ({2: 1, 3: 2}.get(mode, 0) / g))
    rows1 = min(N, 2048)
    t_q1, t_v1 = _oracle_rows((w_bits, x_bits, 0, rows1, K, g, q, mode, 1))
    reps1 = max(1, min(8, int(budget_s / max(t_q1 + t_v1, 1e-3))))
    if reps1 > 1:
        t_q1, t_v1 = _oracle_rows((w_bits, x_bits, 0, rows1, K, g, q, mode, reps1))
    else:
        reps1 = 1
    single = {
        "value": round(gemv_bytes_per_row * rows1 * reps1 / t_v1 / 1e9, 6), "unit": "GB/s", "cores": 1,
        "kind": "oracle",
        "sample": (f"oracle quantize + binary64 GEMV on rows 0..{rows1 - 1} of the {N}x{K} matrix "
                   f"({rows1}/{N} of the workload), {reps1} repetition(s), one thread"),
        "quantize_gbs": round(quant_bytes_per_row * rows1 * reps1 / t_q1 / 1e9, 6),
        "seconds": round(t_q1 + t_v1, 2)}

    P = host_worker_count()
    bounds = np.linspace(0, N, P + 1).astype(int)
    per_pass = (t_q1 + t_v1) / reps1 * N / rows1 / P         # estimated seconds per slice pass
    repsP = max(1, min(8, int(budget_s / max(per_pass, 1e-3))))
    jobs = [(w_bits, x_bits, int(bounds[i]), int(bounds[i + 1]), K, g, q, mode, repsP) for i in range(P)]
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(P) as pool:
        parts = pool.map(_oracle_rows, jobs)
    wall = time.perf_counter() - t0
    # each slice's quantize and GEMV times; the slowest slice bounds the parallel pass
    t_qP = max(p[0] for p in parts)
    t_vP = max(p[1] for p in parts)
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {
        "value": round(gemv_bytes_per_row * N * repsP / t_vP / 1e9, 6),
        "unit": "GB/s",
        "cores": P,
        "kind": "oracle",
        "sample": (f"oracle quantize + binary64 GEMV on all {N} rows of the {N}x{K} matrix, "
                   f"{P} processes of one thread on equal row slices, {repsP} repetition(s); "
                   f"GEMV rate = GEMV bytes over the slowest slice's GEMV time"),
        "quantize_gbs": round(quant_bytes_per_row * N * repsP / t_qP / 1e9, 6),
        "seconds": round(wall, 2),
        "single_thread": single,
        "host_cpu": cpu_model,
        "host_threads_available": os.cpu_count(),
    }


SWEEP_MODES = ("signed_sym", "unsigned_sym", "asym", "asym_min")
HBM_TARGET_BYTES = 600 << 20    # distinct weight bytes per timed pass: over twice the Infinity Cache


WARMUP_S = 0.02   # GPU time spent before a sweep measurement's timed repetitions


def _graph_time(torch, fn, reps: int) -> float:
    """Seconds per replay of a HIP graph holding the launches fn() makes."""
    s = torch.cuda.Stream()
    # the side stream starts after the work queued so far (the inputs' producers): an
    # unordered start could let fn()'s output writes land on memory the caller's stream
    # is still reading, e.g. a temporary it freed
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        g.replay()
        e1.record(s)
        torch.cuda.synchronize()
        # Warm-up: replays for about WARMUP_S of GPU time first, so the timed replays run at
        # the clock the load settles at (a cold start measured up to 15 % slower on the
        # prefill GEMM).
        for _ in range(min(1000, int(WARMUP_S / max(e0.elapsed_time(e1) / 1e3, 1e-6)))):
            g.replay()
        torch.cuda.synchronize()
        e0.record(s)
        for _ in range(reps):
            g.replay()
        e1.record(s)
        torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3 / reps


def _eager_time(torch, fn, reps: int) -> float:
    """Seconds per call of fn() launched eagerly on the null stream (ssq_quantize's stream),
    after about WARMUP_S of warm-up calls."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    fn()
    e1.record()
    torch.cuda.synchronize()
    for _ in range(min(1000, int(WARMUP_S / max(e0.elapsed_time(e1) / 1e3, 1e-6)))):
        fn()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3 / reps


def meta_bytes_per_group(mode_name):
    """Bytes stored per group beside the scale: u8 zero point, fp16 minimum, or none."""
    return {"asym": 1, "asym_min": 2}.get(mode_name, 0)


def matmul_bytes(M, N, K, q, g, meta):
    """Algorithmic bytes of one M x N x K matmul on packed weights: codes, fp16 scales and
    `meta` bytes per group, bf16 activations read and bf16 outputs written."""
    return N * K * q // 8 + (2 + meta) * N * K // g + 2 * M * K + 2 * M * N


def quantize_bytes(N, K, q, g, meta):
    """Algorithmic bytes of quantizing bf16 W[N, K]: weights read, codes, scales and
    `meta` bytes per group written."""
    return 2 * N * K + N * K * q // 8 + (2 + meta) * N * K // g


def diagnostics_bytes(N, K, g):
    """bf16 weights read, int16 margin and fp32 gain written per group (the tally's
    per-block counts are a few KB)."""
    return 2 * N * K + 6 * N * K // g


def stream_ceiling(torch, dev, nbytes: int, copies: int, reps: int):
    """The practical HBM ceiling next to the GEMV: a plain streaming read (the
    measurement-only ssq_bench_stream_read kernel) of `copies` distinct buffers of the
    GEMV's byte count, each launch also storing about as many bytes as the GEMV's
    output, replayed in a HIP graph like the GEMV phase.  None if the measurement
    library is not built."""
    import ctypes
    path = os.path.join(ROOT, "paper_2607_08779_amd", "libssq_bench.so")
    if not os.path.exists(path):
        return None
    lib = ctypes.CDLL(path)
    lib.ssq_bench_stream_read.restype = ctypes.c_int
    lib.ssq_bench_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    lib.ssq_bench_stream_read_sink_words.restype = ctypes.c_int64
    lib.ssq_bench_stream_read_sink_words.argtypes = [ctypes.c_int64]
    bufs = [torch.full((nbytes // 4,), i + 1, dtype=torch.int32, device=dev) for i in range(copies)]
    sink = torch.zeros(max(1, lib.ssq_bench_stream_read_sink_words(nbytes)), dtype=torch.int32, device=dev)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        def run():
            for b in bufs:
                st = lib.ssq_bench_stream_read(b.data_ptr(), nbytes, sink.data_ptr(), s.cuda_stream)
                if st != 0:
                    raise RuntimeError(f"ssq_bench_stream_read failed ({st})")
        run()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            run()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            g.replay()
        e1.record(s)
        torch.cuda.synchronize()
    avg = e0.elapsed_time(e1) / 1e3 / (reps * copies)
    del bufs
    return {"kernel": "stream_read_kernel (measurement only)", "bytes_per_launch": nbytes,
            "avg_launch_us": round(avg * 1e6, 3), "gbs": round(nbytes / avg / 1e9, 2),
            "frac": round(nbytes / avg / 1e9 / HBM_PEAK_GBS, 4)}


def sweep(args) -> int:
    """Throughput of every format on the Llama3 shapes (event-timed; weights past the
    Infinity Cache for the decode passes).  One JSON line with a row per case."""
    import torch

    from paper_2607_08779_amd import ssq, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    t_start = time.perf_counter()

    def dev_bf16(a):
        return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)

    rows = []

    def block_pass(wl, names, q, g, mode_name, ms):
        """Quantize the block (its launches in sequence), then matmuls at each M through
        enough quantized copies of the block to stream from HBM."""
        mode = ssq.MODES[mode_name]
        asym = meta_bytes_per_group(mode_name)
        shapes = {n: (wl.layers[n].rows, wl.layers[n].cols) for n in names}
        first = {n: ssq.ssq_quantize(W[n], g, q, mode) for n in names}
        t_q = _eager_time(torch, lambda: [ssq.ssq_quantize(W[n], g, q, mode, out=first[n]) for n in names], 5)
        qb = sum(quantize_bytes(N, K, q, g, asym) for N, K in shapes.values())
        rows.append({"block": wl.name, "op": "quantize", "q": q, "group": g, "mode": mode_name,
                     "launches": len(names), "us": round(t_q * 1e6, 2), "bytes": qb,
                     "gbs": round(qb / t_q / 1e9, 1), "frac_hbm": round(qb / t_q / 1e9 / HBM_PEAK_GBS, 4)})
        wbytes = sum(matmul_bytes(0, N, K, q, g, asym) for N, K in shapes.values())
        copies = [first] + [{n: ssq.ssq_quantize(W[n], g, q, mode) for n in names}
                            for _ in range(max(0, -(-HBM_TARGET_BYTES // wbytes) - 1))]
        for M in ms:
            xs = {K: dev_bf16(synth.activations(M, K, seed=wl.x_seed + M)) for _, K in shapes.values()}
            ys = {n: torch.empty((M, N), dtype=torch.bfloat16, device=dev) for n, (N, K) in shapes.items()}
            wss = {n: ssq.ssq_matmul_workspace(M, N, K, g, q, device=dev) for n, (N, K) in shapes.items()}

            def run():
                for c in copies:
                    for n in names:
                        N, K = shapes[n]
                        ssq.ssq_matmul(xs[K], *c[n], N, K, g, q, out=ys[n], workspace=wss[n])

            t = _graph_time(torch, run, 10) / len(copies)
            mb = sum(matmul_bytes(M, N, K, q, g, asym) for N, K in shapes.values())
            fl = sum(2 * M * N * K for N, K in shapes.values())
            rows.append({"block": wl.name, "op": f"matmul M={M}", "q": q, "group": g, "mode": mode_name,
                         "launches": len(names), "copies": len(copies), "us": round(t * 1e6, 2),
                         "bytes": mb, "gbs": round(mb / t / 1e9, 1),
                         "frac_hbm": round(mb / t / 1e9 / HBM_PEAK_GBS, 4),
                         "tflops": round(fl / t / 1e12, 2)})
        del copies, first
        torch.cuda.empty_cache()

    # Llama3-8B block: q in {2,3,4}, g in {32,64,128}, three modes; decode GEMV (M=1).
    wl = synth.llama3_8b_block()
    names = list(synth.LLAMA3_8B)
    W = {n: dev_bf16(synth.weights(wl.layers[n])) for n in names}
    parts = set(args.sweep_parts.split(","))
    for q in (2, 3, 4) if "formats" in parts else ():
        for g in (32, 64, 128):
            for mode_name in SWEEP_MODES:
                block_pass(wl, names, q, g, mode_name, (1,))

    # Sign-rule diagnostics (Sec. 4 Remark 1) over the block: per-group margin and gain,
    # then the tally.  Fig. 1's two statistics are reported from the tally: the share of
    # groups with m >= 0 (Corollary 1's condition) and the share with g > 0 among those
    # with m > 0.  Synthetic weights: these are not the paper's model figures.
    for q in (2, 3, 4) if "diagnostics" in parts else ():
        for g in (32, 64, 128):
            outs = {n: (torch.empty((N, K // g), dtype=torch.int16, device=dev),
                        torch.empty((N, K // g), dtype=torch.float32, device=dev),
                        torch.empty(9, dtype=torch.int64, device=dev))
                    for n, (N, K) in ((n, (wl.layers[n].rows, wl.layers[n].cols)) for n in names)}
            t = _eager_time(torch, lambda: [ssq.ssq_sign_diagnostics(W[n], g, q, out=outs[n]) for n in names], 5)
            tally = sum(outs[n][2].cpu().view(3, 3) for n in names).numpy()
            groups = int(tally.sum())
            db = sum(diagnostics_bytes(wl.layers[n].rows, wl.layers[n].cols, g) for n in names)
            rows.append({"block": wl.name, "op": "sign_diagnostics", "q": q, "group": g,
                         "launches": len(names), "us": round(t * 1e6, 2), "bytes": db,
                         "gbs": round(db / t / 1e9, 1), "frac_hbm": round(db / t / 1e9 / HBM_PEAK_GBS, 4),
                         "groups": groups, "tally": tally.tolist(),
                         "frac_margin_ge_0": round(float(tally[1:].sum()) / groups, 4),
                         "frac_gain_gt_0_given_margin_gt_0": round(float(tally[2, 2]) / max(1, tally[2].sum()), 4)})
            del outs

    # Q8_0 activations + integer-dot matmul (App. C, App. B.3) against the bf16 path on
    # the same quantized copies of the block (graph-timed), per q and layout: decode
    # (M = 1, the one-token kernel) and batched decode (M = 16, integer MFMA against the
    # bf16 MFMA kernel with its split workspace); the activation quantization is timed
    # separately (one launch per K).
    for q in (2, 3, 4) if "q8" in parts else ():
        for mode_name in ("signed_sym", "asym", "asym_min"):
            mode = ssq.MODES[mode_name]
            meta = meta_bytes_per_group(mode_name)
            shapes = {n: (wl.layers[n].rows, wl.layers[n].cols) for n in names}
            wbytes = sum(matmul_bytes(0, N, K, q, 32, meta) for N, K in shapes.values())
            copies = [{n: ssq.ssq_quantize(W[n], 32, q, mode) for n in names}
                      for _ in range(max(1, -(-HBM_TARGET_BYTES // wbytes)))]
            for M in (1, 16):
                xs = {K: dev_bf16(synth.activations(M, K, seed=wl.x_seed + M)) for _, K in shapes.values()}
                acts = {K: ssq.ssq_quantize_act_q8(x) for K, x in xs.items()}
                ys = {n: torch.empty((M, N), dtype=torch.bfloat16, device=dev) for n, (N, K) in shapes.items()}
                wss = {n: ssq.ssq_matmul_workspace(M, N, K, 32, q, device=dev) for n, (N, K) in shapes.items()}

                def run_q8():
                    for c in copies:
                        for n in names:
                            N, K = shapes[n]
                            ssq.ssq_matmul_q8(*acts[K], *c[n], N, K, 32, q, out=ys[n])

                def run_bf16():
                    for c in copies:
                        for n in names:
                            N, K = shapes[n]
                            ssq.ssq_matmul(xs[K], *c[n], N, K, 32, q, out=ys[n], workspace=wss[n])

                t_q8 = _graph_time(torch, run_q8, 10) / len(copies)
                t_bf = _graph_time(torch, run_bf16, 10) / len(copies)
                # 25 rounds per graph: a replay of a graph of two microsecond launches is
                # bound by the host's graph launch, not by the kernels
                t_act = _graph_time(torch, lambda: [ssq.ssq_quantize_act_q8(x, out=acts[K])
                                                    for _ in range(25) for K, x in xs.items()], 10) / 25
                mb = sum(N * K * q // 8 + (2 + meta) * N * K // 32 + M * (K + K // 16 + 2 * N)
                         for N, K in shapes.values())
                rows.append({"block": wl.name, "op": f"q8 matmul M={M}", "q": q, "group": 32, "mode": mode_name,
                             "launches": len(names), "copies": len(copies), "us": round(t_q8 * 1e6, 2),
                             "bytes": mb, "gbs": round(mb / t_q8 / 1e9, 1),
                             "frac_hbm": round(mb / t_q8 / 1e9 / HBM_PEAK_GBS, 4),
                             "bf16_us": round(t_bf * 1e6, 2), "speedup_vs_bf16": round(t_bf / t_q8, 3),
                             "act_quantize_us": round(t_act * 1e6, 2), "act_quantize_launches": len(xs)})
            del copies
            torch.cuda.empty_cache()

    # Prefill GEMM (W4 g32) on both MLP orientations, per mode.
    pf = synth.prefill()
    for n, spec in pf.layers.items() if "prefill" in parts else ():
        Wp = dev_bf16(synth.weights(spec))
        N, K = spec.rows, spec.cols
        for mode_name in SWEEP_MODES:
            mode = ssq.MODES[mode_name]
            c, s_, z = ssq.ssq_quantize(Wp, 32, 4, mode)
            for M in (512, 2048):
                x = dev_bf16(synth.activations(M, K, seed=pf.x_seed + M))
                y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
                ws = ssq.ssq_matmul_workspace(M, N, K, 32, 4, device=dev)
                t = _graph_time(torch, lambda: [ssq.ssq_matmul(x, c, s_, z, N, K, 32, 4, out=y, workspace=ws)
                                                for _ in range(4)], 5) / 4
                tf = 2 * M * N * K / t / 1e12
                rows.append({"block": pf.name, "op": f"gemm {n} M={M}", "q": 4, "group": 32,
                             "mode": mode_name, "N": N, "K": K, "us": round(t * 1e6, 2),
                             "tflops": round(tf, 2), "frac_mfma": round(tf / BF16_PEAK_TFLOPS, 4)})
        del Wp
    del W
    torch.cuda.empty_cache()

    # Llama3-70B block at q=2, g=32: quantize, then M=1 and M=16 per mode.
    if "70b" in parts:
        wl = synth.llama3_70b_block()
        names = list(synth.LLAMA3_70B)
        W = {n: dev_bf16(synth.weights(wl.layers[n])) for n in names}
        for mode_name in SWEEP_MODES:
            block_pass(wl, names, 2, 32, mode_name, (1, 16))
        del W
        torch.cuda.empty_cache()

    # Qwen3-8B and Qwen3-14B blocks (the two largest Qwen3 models of Table 1): quantize,
    # decode (M = 1, 16) and prefill (M = 512) through every projection, per layout, at
    # q = 4 and q = 2.
    for wl_fn in (synth.qwen3_8b_block, synth.qwen3_14b_block) if "qwen3" in parts else ():
        wl = wl_fn()
        names = list(wl.layers)
        W = {n: dev_bf16(synth.weights(wl.layers[n])) for n in names}
        for q in (4, 2):
            for mode_name in SWEEP_MODES:
                block_pass(wl, names, q, 32, mode_name, (1, 16, 512))
        del W
        torch.cuda.empty_cache()

    # W4 g32 signed decode GEMV at N = 4096 over K, each K next to the streaming read of
    # the same byte count: the marginal rate between consecutive K (bytes added over time
    # added) shows the kernel's streaming rate with its fixed per-launch cost removed.
    if "ksweep" in parts:
        prev = None
        for K in (4096, 8192, 14336, 20480, 28672):
            spec = synth.WeightSpec(4096, K, nu=5.0, scale=0.02, outlier_frac=0.001, seed=8000 + K // 1024)
            Wk = dev_bf16(synth.weights(spec))
            c0 = ssq.ssq_quantize(Wk, 32, 4, ssq.SIGNED_SYM)
            del Wk
            b = matmul_bytes(1, 4096, K, 4, 32, 0)
            n_copies = max(2, -(-HBM_TARGET_BYTES // b))
            cs = [c0] + [tuple(None if t is None else t.clone() for t in c0) for _ in range(n_copies - 1)]
            x = dev_bf16(synth.activations(1, K, seed=8100 + K // 1024))
            y = torch.empty((1, 4096), dtype=torch.bfloat16, device=dev)
            t = _graph_time(torch, lambda: [ssq.ssq_matmul(x, *c, 4096, K, 32, 4, out=y) for c in cs], 20) / len(cs)
            del cs, c0
            torch.cuda.empty_cache()
            st = stream_ceiling(torch, dev, b // 16 * 16, n_copies, 20)
            row = {"block": "gemv_ksweep", "op": "matmul M=1", "q": 4, "group": 32, "mode": "signed_sym",
                   "N": 4096, "K": K, "copies": n_copies, "us": round(t * 1e6, 3), "bytes": b,
                   "gbs": round(b / t / 1e9, 1), "frac_hbm": round(b / t / 1e9 / HBM_PEAK_GBS, 4)}
            if st is not None:
                row["stream_us"] = st["avg_launch_us"]
                row["stream_gbs"] = st["gbs"]
                row["gemv_over_stream"] = round(st["avg_launch_us"] / (t * 1e6), 4)
            if prev is not None:
                db = b - prev["bytes"]
                row["marginal_gbs"] = round(db / ((row["us"] - prev["us"]) * 1e-6) / 1e9, 1)
                if st is not None and "stream_us" in prev:
                    row["stream_marginal_gbs"] = round(db / ((row["stream_us"] - prev["stream_us"]) * 1e-6) / 1e9, 1)
            rows.append(row)
            prev = row

    print(json.dumps({"sweep": "format sweep on synthetic Llama3 and Qwen3 shapes", "data": "synthetic",
                      "hbm_peak_gbs": HBM_PEAK_GBS, "bf16_peak_tflops": BF16_PEAK_TFLOPS,
                      "wall_s": round(time.perf_counter() - t_start, 1), "rows": rows}), flush=True)
    return 0


def main() -> int:
    args = parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        return 2
    if args.sweep:
        return sweep(args)
    import torch

    from paper_2607_08779_amd import ssq, synth

    mode = ssq.MODES[args.mode]
    phases = set(args.phases.split(","))

    wl = synth.llama3_8b_decode()
    spec = wl.layers["down_proj"]
    N, K, q, g = spec.rows, spec.cols, 4, 32
    w_bits = synth.weights(spec)                                   # bf16 bits, host
    x1_bits = synth.activations(1, K, seed=wl.x_seed)
    meta = meta_bytes_per_group(args.mode)
    gemv_bytes = matmul_bytes(1, N, K, q, g, meta)
    # the oracle's timing forks worker processes, so it runs before anything touches the GPU
    cpu = None if args.no_cpu_baseline else cpu_baseline(w_bits, x1_bits, N, K, g, q, mode, gemv_bytes / N)

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    xm_bits = synth.activations(args.gemm_m, K, seed=wl.x_seed + args.gemm_m)
    xb_bits = synth.activations(args.batched_m, K, seed=wl.x_seed + args.batched_m)

    def dev_bf16(a):
        return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)

    W = dev_bf16(w_bits)
    x1, xm, xb = dev_bf16(x1_bits), dev_bf16(xm_bits), dev_bf16(xb_bits)
    layers = []
    for _ in range(args.layers):
        layers.append(ssq.ssq_quantize(W, g, q, mode))
    # The quantize phase rotates over --quantize-copies copies of W and of its outputs
    # (3 x 150 MB by default, past the 256 MB Infinity Cache), so each step streams its
    # operands from HBM rather than from the cache a single re-quantized matrix would fit.
    Wq = [W] + [W.clone() for _ in range(args.quantize_copies - 1)]
    staging = [ssq.ssq_quantize(w_, g, q, mode) for w_ in Wq]
    y1 = torch.empty((1, N), dtype=torch.bfloat16, device=dev)
    ym = torch.empty((args.gemm_m, N), dtype=torch.bfloat16, device=dev)
    yb = torch.empty((args.batched_m, N), dtype=torch.bfloat16, device=dev)
    # the prefill GEMM and the batched decode get the split-reduction workspaces they ask
    # for (None: no split)
    gemm_ws = ssq.ssq_matmul_workspace(args.gemm_m, N, K, g, q, device=dev)
    batched_ws = ssq.ssq_matmul_workspace(args.batched_m, N, K, g, q, device=dev)
    torch.cuda.synchronize()

    # The decode GEMVs and prefill GEMMs of one step are captured once in a HIP graph
    # (on torch's capture stream, which ssq_matmul receives as its stream); replaying
    # it dispatches the kernels back to back instead of at Python's launch rate.
    # ssq_quantize is defined on the null stream, so it runs outside the graph.
    def decode_and_prefill(i):
        if "gemv" in phases:
            for r in range(args.layers):
                c, s, z = layers[(i + r) % args.layers]
                ssq.ssq_matmul(x1, c, s, z, N, K, g, q, out=y1)
        if "batched" in phases:
            for r in range(args.layers):
                c, s, z = layers[(i + r) % args.layers]
                ssq.ssq_matmul(xb, c, s, z, N, K, g, q, out=yb, workspace=batched_ws)
        if "gemm" in phases:
            for r in range(args.gemm_layers):
                c, s, z = layers[(i * args.gemm_layers + r) % args.layers]
                ssq.ssq_matmul(xm, c, s, z, N, K, g, q, out=ym, workspace=gemm_ws)

    # Llama3-70B down-projection (8192x28672): the same GEMV on a matrix 4x larger, so
    # the per-launch fixed cost weighs a quarter as much; copies of its quantized form
    # stream from HBM like the 8B layers.
    if "gemv70b" in phases:
        wl70 = synth.llama3_70b_block()
        s70 = wl70.layers["down_proj"]
        N70, K70 = s70.rows, s70.cols
        W70 = dev_bf16(synth.weights(s70))
        first70 = ssq.ssq_quantize(W70, g, q, mode)
        del W70
        layers70 = [first70] + [tuple(None if t is None else t.clone() for t in first70)
                                for _ in range(args.layers70b - 1)]
        x70 = dev_bf16(synth.activations(1, K70, seed=wl70.x_seed + 1))
        y70 = torch.empty((1, N70), dtype=torch.bfloat16, device=dev)
        torch.cuda.empty_cache()

    def decode_70b():
        for c in layers70:
            ssq.ssq_matmul(x70, *c, N70, K70, g, q, out=y70)

    graphs = {}
    if "gemv70b" in phases:
        decode_70b()
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            decode_70b()
        graphs["gemv70b"] = gr
    for part in ("gemv", "batched", "gemm"):
        if part not in phases:
            continue
        saved = set(phases)
        phases.intersection_update({part})
        decode_and_prefill(0)                      # warm the allocator outside capture
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            decode_and_prefill(0)
        graphs[part] = gr
        phases.clear()
        phases.update(saved)
    torch.cuda.synchronize()

    copy_src = copy_dst = None
    if "copy" in phases:    # plain copy of known size: the reference for HBM byte counters
        copy_src = torch.ones(64 << 20, dtype=torch.int32, device=dev)
        copy_dst = torch.empty_like(copy_src)

    def step(i, ev=None):
        if copy_src is not None:
            copy_dst.copy_(copy_src)
        if ev:
            ev[0].record()
        if "quantize" in phases:
            ssq.ssq_quantize(Wq[i % len(Wq)], g, q, mode, out=staging[i % len(Wq)])
        if ev:
            ev[1].record()
        if "gemv" in graphs:
            graphs["gemv"].replay()
        if ev:
            ev[2].record()
        if "batched" in graphs:
            graphs["batched"].replay()
        if ev:
            ev[3].record()
        if "gemm" in graphs:
            graphs["gemm"].replay()
        if ev:
            ev[4].record()
        if "gemv70b" in graphs:
            graphs["gemv70b"].replay()
        if ev:
            ev[5].record()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i, events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    if "gemv" in graphs:   # the replayed graph must match an eager launch bit for bit
        last = layers[(args.layers - 1) % args.layers]
        y_eager = ssq.ssq_matmul(x1, *last, N, K, g, q)
        torch.cuda.synchronize()
        if not torch.equal(y_eager.view(torch.int16), y1.view(torch.int16)):
            raise RuntimeError("graph replay of the GEMV differs from an eager launch")

    def spread(i, per_step):
        """Median per-launch time (us) and coefficient of variation over the timed steps."""
        v = np.array([e[i].elapsed_time(e[i + 1]) * 1e3 / per_step for e in events])
        return round(float(np.median(v)), 3), round(float(v.std() / v.mean()) if v.mean() > 0 else 0.0, 4)

    ceiling = stream_ceiling(torch, dev, (N * K * q // 8 + 2 * N * K // g + 2 * K + 2 * N) // 16 * 16,
                             args.layers, args.steps) if "gemv" in phases else None

    t_q = sum(e[0].elapsed_time(e[1]) for e in events) / 1e3   # seconds
    t_v = sum(e[1].elapsed_time(e[2]) for e in events) / 1e3
    t_b = sum(e[2].elapsed_time(e[3]) for e in events) / 1e3
    t_m = sum(e[3].elapsed_time(e[4]) for e in events) / 1e3
    t_70 = sum(e[4].elapsed_time(e[5]) for e in events) / 1e3
    t_step = sum(e[0].elapsed_time(e[5]) for e in events) / 1e3 / args.steps

    quant_bytes = quantize_bytes(N, K, q, g, meta)
    gemm_flops = 2 * args.gemm_m * N * K
    batched_bytes = matmul_bytes(args.batched_m, N, K, q, g, meta)
    n_gemv = args.steps * args.layers
    n_gemm = args.steps * args.gemm_layers

    out = {
        "metric": METRIC,
        "value": None, "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(t_step * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "llama3_8b_down_proj_4096x14336_w4g32", "N": N, "K": K, "q": q,
                   "group": g, "mode": args.mode, "decode_M": 1, "decode_layers": args.layers,
                   "prefill_M": args.gemm_m, "prefill_layers": args.gemm_layers,
                   "prefill_workspace_bytes": 0 if gemm_ws is None else gemm_ws.numel(),
                   "batched_M": args.batched_m, "quantize_copies": args.quantize_copies,
                   "batched_workspace_bytes": 0 if batched_ws is None else batched_ws.numel(),
                   "weights": f"bf16 Student-t(5)*0.02 + 0.1% x20 outliers, seed {spec.seed}"},
        "wall_s": round(wall, 4),
    }
    if "gemv" in phases:
        avg = t_v / n_gemv
        gbs = gemv_bytes / avg / 1e9
        out["value"] = round(gbs, 2)
        out["roofline"] = {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS,
                           "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                           "traffic": measured_traffic("gemv", args.mode),
                           "kernel": "gemv_kernel (ssq_matmul, M=1)",
                           "bytes_per_launch": gemv_bytes, "avg_launch_us": round(avg * 1e6, 3)}
        out["roofline"]["median_launch_us"], out["roofline"]["cv"] = spread(1, args.layers)
        add_trace_frac(out["roofline"], "gemv", args.mode, gemv_bytes)
        if ceiling is not None:
            ceiling["gemv_over_stream"] = round(gbs / ceiling["gbs"], 4)
        out["ceiling_stream_read"] = ceiling
    if "batched" in phases:
        avg = t_b / n_gemv
        gbs = batched_bytes / avg / 1e9
        out["batched_decode_gbs"] = round(gbs, 2)
        out["roofline_batched"] = {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS,
                                   "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                                   "traffic": measured_traffic("batched", args.mode),
                                   "kernel": ("skinny_stat_kernel" if args.batched_m <= 16 and q in (2, 4) and K % 512 == 0
                                              else "skinny_split_kernel") + f" (ssq_matmul, M={args.batched_m})",
                                   "bytes_per_launch": batched_bytes, "avg_launch_us": round(avg * 1e6, 3),
                                   "tflops": round(2 * args.batched_m * N * K / avg / 1e12, 2)}
        out["roofline_batched"]["median_launch_us"], out["roofline_batched"]["cv"] = spread(2, args.layers)
        add_trace_frac(out["roofline_batched"], "batched", args.mode, batched_bytes)
    if "gemm" in phases:
        avg = t_m / n_gemm
        tf = gemm_flops / avg / 1e12
        out["gemm_tflops"] = round(tf, 2)
        out["roofline_gemm"] = {"bound": "mfma", "achieved": round(tf, 2),
                                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                "frac": round(tf / BF16_PEAK_TFLOPS, 4),
                                "traffic": measured_traffic("gemm", args.mode),
                                "kernel": f"gemm_kernel (ssq_matmul, M={args.gemm_m})",
                                "flops_per_launch": gemm_flops, "avg_launch_us": round(avg * 1e6, 3)}
        out["roofline_gemm"]["median_launch_us"], out["roofline_gemm"]["cv"] = spread(3, args.gemm_layers)
        add_trace_frac(out["roofline_gemm"], "gemm", args.mode, gemm_flops)
    if "gemv70b" in phases:
        avg = t_70 / (args.steps * len(layers70))
        b70 = matmul_bytes(1, N70, K70, q, g, meta)
        gbs = b70 / avg / 1e9
        out["config"]["gemv70b"] = {"N": N70, "K": K70, "copies": len(layers70),
                                    "weights": f"bf16 Student-t(5)*0.015 + 0.1% x20 outliers, seed {s70.seed}"}
        out["roofline_gemv_70b"] = {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS,
                                    "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                                    "traffic": measured_traffic("gemv:70b", args.mode),
                                    "kernel": f"gemv_stat_kernel (ssq_matmul, M=1, {N70}x{K70})",
                                    "bytes_per_launch": b70, "avg_launch_us": round(avg * 1e6, 3)}
        out["roofline_gemv_70b"]["median_launch_us"], out["roofline_gemv_70b"]["cv"] = \
            spread(4, len(layers70))
        add_trace_frac(out["roofline_gemv_70b"], "gemv:70b", args.mode, b70)
    if "quantize" in phases:
        avg = t_q / args.steps
        gbs = quant_bytes / avg / 1e9
        out["quantize_gbs"] = round(gbs, 2)
        out["roofline_quantize"] = {"bound": "hbm", "achieved": round(gbs, 2),
                                    "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                    "frac": round(gbs / HBM_PEAK_GBS, 4),
                                    "traffic": measured_traffic("quantize", args.mode),
                                    "kernel": "quantize_kernel (ssq_quantize)",
                                    "bytes_per_launch": quant_bytes,
                                    "avg_launch_us": round(avg * 1e6, 3)}
        out["roofline_quantize"]["median_launch_us"], out["roofline_quantize"]["cv"] = spread(0, 1)
        add_trace_frac(out["roofline_quantize"], "quantize", args.mode, quant_bytes)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    out["host"] = platform.node()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
