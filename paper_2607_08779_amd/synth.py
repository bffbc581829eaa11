"""Seeded synthetic inputs: weight matrices and activations shaped like Llama3 and Qwen3
projections.

This module only draws random numbers and casts them to storage formats; it
holds none of the quantization arithmetic, so the CPU oracle and the HIP
library can both be fed from it without sharing any of the method.

Recipe (stands in for the real Llama3/Qwen3 checkpoints the paper measures on,
which are not available here):

* weights: Student-t(nu) * scale drawn in binary64, rounded to binary32; a
  fraction ``outlier_frac`` of the entries of every row chunk (chosen without
  replacement) is multiplied by ``outlier_mult`` times a uniformly random sign;
  bf16 workloads are then rounded to bfloat16 (half to even, by torch).
* activations: standard normal, drawn in binary32, optionally rounded to bf16.
* determinism: rows are generated in chunks of ``ROW_CHUNK`` rows, chunk c of a
  matrix with seed S drawing from ``SeedSequence([S, c])``.  Any row range can
  therefore be regenerated on its own, which lets the oracle check sampled rows
  of a full-size matrix without materialising the rest.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

ROW_CHUNK = 128


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


@dataclass(frozen=True)
class WeightSpec:
    """Distribution of one synthetic weight matrix [rows, cols]."""

    rows: int
    cols: int
    nu: float
    scale: float
    outlier_frac: float = 0.0
    outlier_mult: float = 20.0
    seed: int = 0
    bf16: bool = True


def _chunk(spec: WeightSpec, c: int) -> np.ndarray:
    r0 = c * ROW_CHUNK
    r1 = min(spec.rows, r0 + ROW_CHUNK)
    n = (r1 - r0) * spec.cols
    rng = np.random.default_rng(np.random.SeedSequence([spec.seed, c]))
    w = rng.standard_t(spec.nu, size=n) * spec.scale
    if spec.outlier_frac > 0:
        n_out = int(round(spec.outlier_frac * n))
        idx = rng.choice(n, n_out, replace=False)
        sign = np.where(rng.random(n_out) < 0.5, -1.0, 1.0)
        w[idx] *= spec.outlier_mult * sign
    return w.astype(np.float32).reshape(r1 - r0, spec.cols)


def weights_f32(spec: WeightSpec, row_start: int = 0, row_stop: int | None = None) -> np.ndarray:
    """Binary32 weights for rows [row_start, row_stop) (before any bf16 rounding)."""
    row_stop = spec.rows if row_stop is None else row_stop
    if not 0 <= row_start <= row_stop <= spec.rows:
        raise ValueError("bad row range")
    if row_start == row_stop:
        return np.zeros((0, spec.cols), np.float32)
    c0, c1 = row_start // ROW_CHUNK, (row_stop - 1) // ROW_CHUNK + 1
    with ThreadPoolExecutor(_threads()) as ex:
        parts = list(ex.map(lambda c: _chunk(spec, c), range(c0, c1)))
    full = np.concatenate(parts, axis=0)
    off = row_start - c0 * ROW_CHUNK
    return full[off: off + (row_stop - row_start)]


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round binary32 to bfloat16 (half to even) with torch; return uint16 bit patterns."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def weights(spec: WeightSpec, row_start: int = 0, row_stop: int | None = None) -> np.ndarray:
    """Storage-format weights: uint16 bf16 bits if ``spec.bf16`` else binary32."""
    w = weights_f32(spec, row_start, row_stop)
    return to_bf16_bits(w) if spec.bf16 else w


def activations(M: int, K: int, seed: int, bf16: bool = True) -> np.ndarray:
    """Standard-normal activations [M, K]: uint16 bf16 bits if ``bf16`` else binary32."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0xAC7]))
    x = rng.standard_normal((M, K), dtype=np.float32)
    return to_bf16_bits(x) if bf16 else x


# ---------------------------------------------------------------------------
# Named workloads (shapes are the public Llama3-8B / Llama3-70B / Qwen3-8B / Qwen3-14B
# projections).
# ---------------------------------------------------------------------------

LLAMA3_8B = {  # name: (rows N, cols K)
    "q_proj": (4096, 4096), "k_proj": (1024, 4096), "v_proj": (1024, 4096),
    "o_proj": (4096, 4096), "gate_proj": (14336, 4096), "up_proj": (14336, 4096),
    "down_proj": (4096, 14336),
}
LLAMA3_70B = {
    "q_proj": (8192, 8192), "k_proj": (1024, 8192), "v_proj": (1024, 8192),
    "o_proj": (8192, 8192), "gate_proj": (28672, 8192), "up_proj": (28672, 8192),
    "down_proj": (8192, 28672),
}
# Qwen3 dense models (Table 1 reports Qwen3 0.6B-14B): head_dim 128, 8 key/value heads.
QWEN3_8B = {
    "q_proj": (4096, 4096), "k_proj": (1024, 4096), "v_proj": (1024, 4096),
    "o_proj": (4096, 4096), "gate_proj": (12288, 4096), "up_proj": (12288, 4096),
    "down_proj": (4096, 12288),
}
QWEN3_14B = {
    "q_proj": (5120, 5120), "k_proj": (1024, 5120), "v_proj": (1024, 5120),
    "o_proj": (5120, 5120), "gate_proj": (17408, 5120), "up_proj": (17408, 5120),
    "down_proj": (5120, 17408),
}
PROJ_INDEX = {name: i for i, name in enumerate(LLAMA3_8B)}


@dataclass(frozen=True)
class Workload:
    """A named set of weight matrices plus the quantization settings it is run at."""

    name: str
    layers: dict = field(default_factory=dict)     # layer name -> WeightSpec
    qs: tuple = (4,)
    groups: tuple = (32,)
    ms: tuple = (1,)
    x_seed: int = 0
    bf16: bool = True


def small_fp32() -> Workload:
    """One binary32 256x512 matrix, Student-t(4)*0.02, no outliers; q=4, g=32, M=1."""
    spec = WeightSpec(256, 512, nu=4.0, scale=0.02, seed=1000, bf16=False)
    return Workload("fp32_256x512", {"w": spec}, qs=(4,), groups=(32,), ms=(1,),
                    x_seed=1100, bf16=False)


def _llama_layers(shapes: dict, names, nu: float, scale: float, base_seed: int) -> dict:
    return {n: WeightSpec(*shapes[n], nu=nu, scale=scale, outlier_frac=0.001,
                          outlier_mult=20.0, seed=base_seed + PROJ_INDEX[n]) for n in names}


def llama3_8b_decode() -> Workload:
    """Llama3-8B decode layers, bf16 t(5)*0.02 + 0.1% x20 outliers; q=4, g=32, M=1."""
    names = ("q_proj", "gate_proj", "up_proj", "down_proj")
    return Workload("llama3_8b_decode_w4g32", _llama_layers(LLAMA3_8B, names, 5.0, 0.02, 2000),
                    qs=(4,), groups=(32,), ms=(1,), x_seed=2100)


def llama3_8b_block() -> Workload:
    """All seven Llama3-8B projections at q in {2,3}, g in {32,64,128}, M=1."""
    return Workload("llama3_8b_block_q23", _llama_layers(LLAMA3_8B, LLAMA3_8B, 5.0, 0.02, 3000),
                    qs=(2, 3), groups=(32, 64, 128), ms=(1,), x_seed=3100)


def prefill() -> Workload:
    """Prefill GEMM: W4 g32 signed weights 14336x4096 and 4096x14336, M in {512, 2048}."""
    names = ("gate_proj", "down_proj")
    return Workload("prefill_w4g32", _llama_layers(LLAMA3_8B, names, 5.0, 0.02, 4000),
                    qs=(4,), groups=(32,), ms=(512, 2048), x_seed=4100)


def llama3_70b_block() -> Workload:
    """Llama3-70B block, bf16 t(5)*0.015 + 0.1% x20 outliers; q=2, g=32, M in {1, 16}."""
    return Workload("llama3_70b_block_q2g32",
                    _llama_layers(LLAMA3_70B, LLAMA3_70B, 5.0, 0.015, 5000),
                    qs=(2,), groups=(32,), ms=(1, 16), x_seed=5100)


def qwen3_8b_block() -> Workload:
    """All seven Qwen3-8B projections, bf16 t(5)*0.02 + 0.1% x20 outliers; q in {2,3,4},
    g=32, M in {1, 16, 512}."""
    return Workload("qwen3_8b_block", _llama_layers(QWEN3_8B, QWEN3_8B, 5.0, 0.02, 6000),
                    qs=(2, 3, 4), groups=(32,), ms=(1, 16, 512), x_seed=6100)


def qwen3_14b_block() -> Workload:
    """All seven Qwen3-14B projections, bf16 t(5)*0.02 + 0.1% x20 outliers; q in {2,3,4},
    g=32, M in {1, 16, 512}."""
    return Workload("qwen3_14b_block", _llama_layers(QWEN3_14B, QWEN3_14B, 5.0, 0.02, 7000),
                    qs=(2, 3, 4), groups=(32,), ms=(1, 16, 512), x_seed=7100)


WORKLOADS = {w().name: w for w in (small_fp32, llama3_8b_decode, llama3_8b_block, prefill,
                                   llama3_70b_block, qwen3_8b_block, qwen3_14b_block)}
