"""Shared helpers for the GPU parity tests: cached synthetic inputs, oracle calls,
row sampling and metric logging.  Imports the oracle (test infrastructure)."""
import functools
import json
import os

import numpy as np
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import synth

METRICS_LOG = os.environ.get("SSQ_PARITY_LOG")


def log_metric(**kv):
    if METRICS_LOG:
        with open(METRICS_LOG, "a") as f:
            f.write(json.dumps(kv) + "\n")


@functools.lru_cache(maxsize=8)
def weights_host(spec: synth.WeightSpec) -> np.ndarray:
    """Storage-format weights (uint16 bf16 bits or float32) for the whole matrix."""
    w = synth.weights(spec)
    w.setflags(write=False)
    return w


def to_device(w: np.ndarray, bf16: bool) -> torch.Tensor:
    if bf16:
        return torch.from_numpy(w.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(w).cuda()


def widen(w: np.ndarray, bf16: bool) -> np.ndarray:
    return O.bf16_bits_to_f32(w) if bf16 else np.asarray(w, np.float32)


def sample_rows(rows: int, n: int = 48, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    pick = {0, 1, rows - 1, rows - 2} | set(rng.choice(rows, min(n, rows), replace=False).tolist())
    return np.array(sorted(r for r in pick if 0 <= r < rows))


def assert_quant_equal(gpu, ref: O.Quantized, rows_idx=None, tag=""):
    codes, scales, zp = gpu
    c = codes.cpu().numpy()
    s = scales.cpu().numpy().view(np.uint16)
    if rows_idx is not None:
        c, s = c[rows_idx], s[rows_idx]
    if not np.array_equal(c, ref.codes):
        r, b = np.argwhere(c != ref.codes)[0]
        raise AssertionError(f"{tag}: codes differ first at row {r} byte {b}: "
                             f"gpu {c[r, b]:#04x} oracle {ref.codes[r, b]:#04x}")
    if not np.array_equal(s, ref.scales):
        r, g = np.argwhere(s != ref.scales)[0]
        raise AssertionError(f"{tag}: scales differ first at row {r} group {g}: "
                             f"gpu {s[r, g]:#06x} oracle {ref.scales[r, g]:#06x}")
    if ref.zp is not None or ref.mins is not None:
        z = zp.cpu().numpy()
        if rows_idx is not None:
            z = z[rows_idx]
        if ref.mins is not None:     # binary16 minimums, returned as int16 bit patterns
            zu = z.view(np.uint16)
            if not np.array_equal(zu, ref.mins):
                r, g = np.argwhere(zu != ref.mins)[0]
                raise AssertionError(f"{tag}: minimums differ first at row {r} group {g}: "
                                     f"gpu {zu[r, g]:#06x} oracle {ref.mins[r, g]:#06x}")
        else:
            assert np.array_equal(z, ref.zp), f"{tag}: zero points differ"
    else:
        assert zp is None


def rel_l2(y: np.ndarray, ref: np.ndarray) -> float:
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(y - ref) / (den if den > 0 else 1.0))


def y_to_f64(y: torch.Tensor) -> np.ndarray:
    return y.float().cpu().numpy().astype(np.float64)
