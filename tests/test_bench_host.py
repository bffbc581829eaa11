"""Host-side checks of bench.py: the one-GPU contract, the algorithmic byte and flop
counts the rooflines divide by (against the figures derived for the Llama3 shapes),
and the guard that drops counter readings taken on other kernel sources."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

LLAMA3_8B = {"q": (4096, 4096), "k": (1024, 4096), "v": (1024, 4096), "o": (4096, 4096),
             "gate": (14336, 4096), "up": (14336, 4096), "down": (4096, 14336)}
LLAMA3_70B = {"q": (8192, 8192), "k": (1024, 8192), "v": (1024, 8192), "o": (8192, 8192),
              "gate": (28672, 8192), "up": (28672, 8192), "down": (8192, 28672)}


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_decode_and_quantize_bytes():
    assert bench.matmul_bytes(1, 4096, 14336, 4, 32, 0) == 33_067_008          # 0.5625 B per weight
    assert bench.matmul_bytes(1, 14336, 4096, 4, 32, 0) == 33_067_008
    assert bench.matmul_bytes(1, 4096, 14336, 4, 32, 1) == 34_902_016          # + u8 zero point
    assert bench.matmul_bytes(1, 4096, 4096, 4, 32, 0) == 9_453_568
    assert bench.quantize_bytes(4096, 14336, 4, 32, 0) == 150_470_656
    # weight bytes per weight by group size
    for g, per in ((32, 0.5625), (64, 0.53125), (128, 0.515625)):
        assert bench.matmul_bytes(0, 1024, 1024, 4, g, 0) == per * 1024 * 1024
    for g, per in ((32, 0.3125), (64, 0.28125), (128, 0.265625)):
        assert bench.matmul_bytes(0, 1024, 1024, 2, g, 0) == per * 1024 * 1024
    assert bench.meta_bytes_per_group("signed_sym") == 0
    assert bench.meta_bytes_per_group("asym") == 1 and bench.meta_bytes_per_group("asym_min") == 2


def test_block_totals():
    blk = {q: sum(bench.matmul_bytes(1, n, k, q, 32, 0) for n, k in LLAMA3_8B.values()) for q in (2, 3, 4)}
    assert [round(blk[q] / 1e6, 2) for q in (4, 3, 2)] == [122.85, 95.58, 68.32]
    qb = {q: sum(bench.quantize_bytes(n, k, q, 32, 0) for n, k in LLAMA3_8B.values()) for q in (2, 3, 4)}
    assert [round(qb[q] / 1e6, 1) for q in (4, 3, 2)] == [558.9, 531.6, 504.4]
    m1 = sum(bench.matmul_bytes(1, n, k, 2, 32, 0) for n, k in LLAMA3_70B.values())
    m16 = sum(bench.matmul_bytes(16, n, k, 2, 32, 0) for n, k in LLAMA3_70B.values())
    assert (round(m1 / 1e6, 1), round(m16 / 1e6, 1)) == (267.7, 272.6)
    assert 2 * 512 * 4096 * 14336 == 60_129_542_144                            # GEMM flops at M=512


def test_counter_readings_follow_the_kernel_sources(monkeypatch):
    for kind in bench.KERNEL_SOURCES:
        v = bench.measured_traffic(kind)
        assert v is None or v > 0
    assert bench.measured_traffic("gemv", "asym") is None                      # taken on signed weights only
    monkeypatch.setattr(bench, "kernel_source_sha", lambda files: "0" * 16)
    for kind in bench.KERNEL_SOURCES:
        assert bench.measured_traffic(kind) is None
