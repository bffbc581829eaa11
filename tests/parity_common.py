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


# ---------------------------------------------------------------------------
# Guarded outputs: every GPU output the parity tests hand to a kernel sits between
# GUARD_BYTES of a known byte pattern on each side, so a store past either end of the
# buffer (a wrong buffer-descriptor size, a ragged tile written whole) is seen.
# ---------------------------------------------------------------------------

GUARD_BYTES = 256
GUARD_BYTE = 0xA5


class Guarded:
    """A contiguous GPU tensor of `shape`/`dtype` with guard bytes around it.

    The interior is pre-filled with `fill` (0xFF: NaN for float outputs, so an output
    element that no kernel wrote fails the comparison) unless `fill` is None."""

    def __init__(self, shape, dtype, fill=0xFF, device="cuda"):
        shape = tuple(int(s) for s in shape)
        self.nbytes = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
        self.buf = torch.full((self.nbytes + 2 * GUARD_BYTES,), GUARD_BYTE, dtype=torch.uint8,
                              device=device)
        inner = self.buf[GUARD_BYTES:GUARD_BYTES + self.nbytes]
        if fill is not None:
            inner.fill_(fill)
        self.t = inner.view(dtype).view(shape)

    def check(self, tag=""):
        """Assert that both guards still hold the pattern."""
        torch.cuda.synchronize()
        head = self.buf[:GUARD_BYTES].cpu().numpy()
        tail = self.buf[GUARD_BYTES + self.nbytes:].cpu().numpy()
        for name, g in (("before", head), ("after", tail)):
            bad = np.flatnonzero(g != GUARD_BYTE)
            if bad.size:
                raise AssertionError(f"{tag}: {bad.size} guard bytes {name} the output overwritten "
                                     f"(first at offset {int(bad[0])})")


def guarded_quant_outputs(rows, cols, group, q, mode):
    """Guarded (codes, scales, meta) buffers in the layout ssq_quantize writes."""
    g = cols // group if group else 0
    codes = Guarded((rows, cols * q // 8), torch.uint8, fill=0x5A)
    scales = Guarded((rows, g), torch.int16, fill=0x5A)
    meta = None
    if mode == O.ASYM:
        meta = Guarded((rows, g), torch.uint8, fill=0x5A)
    elif mode == O.ASYM_MIN:
        meta = Guarded((rows, g), torch.int16, fill=0x5A)
    return codes, scales, meta


# ---------------------------------------------------------------------------
# Element-wise matmul tolerance.
#
# Let W_hat be the oracle's dequantized weights (binary64) and S[m, n] =
# sqrt(sum_k (x[m, k] W_hat[n, k])^2).  The kernels accumulate in binary32 and round
# the result once to the output type:
#   * bf16 output, weights kept exact (the GEMV at M = 1, 2):
#       |y - y_ref| <= 2^-8 |y_ref| + 2^-12 S
#     (one bf16 rounding, half an ulp = 2^-8 relative, plus binary32 accumulation
#     slack far below one bf16 ulp of S);
#   * bf16 output, weights rounded to bf16 before the MFMA (batched decode, prefill):
#       |y - y_ref| <= 2^-8 |y_ref| + (C_W 2^-8 + 2^-12) S,   C_W = 6
#     each weight carries a relative rounding error below 2^-8 that is independent of
#     the sign of its activation, so the dequantization error of an output is a sum of
#     independent symmetric terms with variance proxy 2^-16 S^2 (Hoeffding: exceeding
#     6 2^-8 S has probability below 2 exp(-18) ~ 3e-8 per output, and the rounding
#     errors are uniform, not extreme, so the real margin is about 10 standard deviations);
#   * binary32 output (weights exact in binary32):
#       |y - y_ref| <= 1e-5 (|y_ref| + S).
# Where the bf16 weight is exactly bf16(W_hat) (symmetric and zero-point formats: the
# kernels form s (u - o) exactly in binary32, then round once), the MFMA paths are also
# held to the exact model y_model = x bf16(W_hat)^T: |y - y_model| <= 2^-8 |y_model| + 2^-12 S.
# ---------------------------------------------------------------------------

C_W = 6.0


def matmul_error_bound(x: np.ndarray, w_hat: np.ndarray, y_ref: np.ndarray, rounded_weights: bool,
                       f32: bool):
    """(bound [M, N], S [M, N]) for the comparison described above."""
    x64 = np.asarray(x, np.float64)
    S = np.sqrt((x64 * x64) @ (w_hat * w_hat).T)
    if f32:
        return 1e-5 * (np.abs(y_ref) + S), S
    c = C_W * 2.0 ** -8 if rounded_weights else 0.0
    return 2.0 ** -8 * np.abs(y_ref) + (c + 2.0 ** -12) * S, S


def bf16_round_f64(a: np.ndarray) -> np.ndarray:
    """Round binary64 values that are exact in binary32 to bfloat16 (half to even)."""
    a32 = np.asarray(a, np.float32)
    assert np.array_equal(a32.astype(np.float64), a), "values not exact in binary32"
    return torch.from_numpy(a32).to(torch.bfloat16).to(torch.float64).numpy()


def assert_within(y: np.ndarray, y_ref: np.ndarray, bound: np.ndarray, tag: str) -> float:
    """Element-wise |y - y_ref| <= bound; returns max |y - y_ref| / bound."""
    err = np.abs(y - y_ref)
    bad = ~(err <= bound)                        # NaN (an unwritten output) fails too
    if bad.any():
        m, n = np.argwhere(bad)[0]
        raise AssertionError(f"{tag}: {int(bad.sum())} outputs beyond the element-wise bound; first "
                             f"[{m}, {n}]: gpu {y[m, n]!r} ref {y_ref[m, n]!r} bound {bound[m, n]:.3e}")
    with np.errstate(invalid="ignore", divide="ignore"):
        ratio = np.where(bound > 0, err / np.where(bound > 0, bound, 1.0), 0.0)
    return float(ratio.max()) if ratio.size else 0.0
