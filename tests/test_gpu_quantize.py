"""GPU parity: ssq_quantize / ssq_quantize_f32 against the CPU oracle, bit for bit.

Codes, binary16 scale bits and zero points must be identical.  Small cases are
compared whole; full-size Llama3 shapes are compared on sampled rows (the
oracle is row-independent, so sampled rows are exact expected values).
"""
import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import (assert_quant_equal, guarded_quant_outputs, sample_rows, to_device,
                                 weights_host, widen)

pytestmark = pytest.mark.gpu

MODES = [O.SIGNED_SYM, O.UNSIGNED_SYM, O.ASYM, O.ASYM_MIN]


def run_case(w_host, bf16, group, q, mode, rows_idx=None, tag=""):
    """Quantize into guarded buffers (the guards must survive), compare with the oracle."""
    W = to_device(w_host, bf16)
    rows, cols = w_host.shape
    bufs = guarded_quant_outputs(rows, cols, group, q, mode)
    out = ssq.ssq_quantize(W, group, q, mode, out=tuple(b.t if b is not None else None for b in bufs))
    torch.cuda.synchronize()
    for b in bufs:
        if b is not None:
            b.check(f"{tag} q={q} g={group} mode={mode}")
    wf = widen(w_host if rows_idx is None else w_host[rows_idx], bf16)
    ref = O.quantize(wf, group, q, mode)
    assert_quant_equal(out, ref, rows_idx, tag=f"{tag} q={q} g={group} mode={mode}")


def random_bf16(rows, cols, seed, nu=5.0, scale=0.02, outliers=0.001):
    spec = synth.WeightSpec(rows, cols, nu=nu, scale=scale, outlier_frac=outliers, seed=seed)
    return synth.weights(spec)


@pytest.mark.parametrize("mode", MODES)
def test_small_fp32_matrix_all_modes(mode):
    """256x512 binary32 Student-t(4)*0.02, q=4, g=32 (the small fp32 workload)."""
    spec = synth.small_fp32().layers["w"]
    run_case(weights_host(spec), False, 32, 4, mode, tag="fp32 256x512")


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", MODES)
def test_fp32_ragged_all_formats(q, group, mode):
    w = synth.weights(synth.WeightSpec(37, 768, nu=4.0, scale=0.02, seed=17, bf16=False))
    run_case(w, False, group, q, mode, tag="fp32 37x768")


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", MODES)
def test_bf16_ragged_all_formats(q, group, mode):
    # 37 x 1536 = 56832 weights: 7 workgroup tiles of 8192 and a ragged tail
    w = random_bf16(37, 1536, seed=100 + q)
    run_case(w, True, group, q, mode, tag="bf16 37x1536")


def _edge_matrix():
    """bf16 rows exercising the degenerate and boundary cases of the grids."""
    rng = np.random.default_rng(5)
    rows = []
    z = np.zeros(128, np.float32)
    rows.append(z.copy())                                  # all-zero groups
    rows.append(-z)                                        # negative zeros
    t = rng.standard_normal(128).astype(np.float32) * 0.1
    t[::32] = 1.0; t[1::32] = -1.0                         # +M / -M ties in every group
    rows.append(t)
    m = (rng.integers(-16, 17, 128) * 0.5).astype(np.float32)
    m[::32] = 8.0                                          # exact halves w/s (alpha = 1 at q=4)
    rows.append(m)
    rows.append(np.full(128, 0.375, np.float32))           # constant groups
    rows.append(np.full(128, -0.375, np.float32))
    tiny = (rng.standard_normal(128) * 1e-39).astype(np.float32)
    rows.append(tiny)                                      # bf16 subnormals (division path)
    big = (rng.standard_normal(128) * 1e35).astype(np.float32)
    rows.append(big)                                       # very large magnitudes
    pos = np.abs(rng.standard_normal(128)).astype(np.float32) + 1.0
    rows.append(pos)                                       # one-signed groups (asym widening)
    rows.append(-pos)
    one = np.zeros(128, np.float32); one[::32] = -3.0
    rows.append(one)                                       # single negative outlier
    # min-max grid with s = (0.4375 + 0.5)/15 = 1/16 exactly: every w = (k + 1/2)/16 sits
    # exactly on a half-integer quotient (the asymmetric quantizer's tie path)
    half = ((rng.integers(-8, 7, 128) + 0.5) / 16).astype(np.float32)
    half[::32] = -0.5; half[1::32] = 0.4375
    rows.append(half)
    return synth.to_bf16_bits(np.stack(rows))


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 128])
@pytest.mark.parametrize("mode", MODES)
def test_bf16_edge_cases(q, group, mode):
    with np.errstate(over="ignore"):
        run_case(_edge_matrix(), True, group, q, mode, tag="edge")


def test_single_group_and_empty():
    w = random_bf16(1, 32, seed=3)
    for mode in MODES:
        run_case(w, True, 32, 4, mode, tag="1x32")
    W = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    codes, scales, zp = ssq.ssq_quantize(W, 32, 4, O.SIGNED_SYM)
    assert codes.numel() == 0 and scales.numel() == 0


@pytest.mark.parametrize("mode", MODES)
def test_llama3_8b_decode_layers_full_size(mode):
    """q=4, g=32 on the four decode layer shapes, full matrices on the GPU,
    sampled rows on the oracle."""
    wl = synth.llama3_8b_decode()
    for name, spec in wl.layers.items():
        w = weights_host(spec)
        idx = sample_rows(spec.rows, seed=spec.seed)
        run_case(w, True, 32, 4, mode, rows_idx=idx, tag=name)


@pytest.mark.parametrize("q", [2, 3])
def test_llama3_8b_block_full_size(q):
    """All seven projections at q in {2,3}, g in {32,64,128}, three modes."""
    wl = synth.llama3_8b_block()
    for name, spec in wl.layers.items():
        w = weights_host(spec)
        idx = sample_rows(spec.rows, n=16, seed=spec.seed)
        for group in wl.groups:
            for mode in MODES:
                run_case(w, True, group, q, mode, rows_idx=idx, tag=name)


def test_llama3_70b_shapes_full_size():
    """q=2, g=32 on every distinct 70B shape: q/o 8192x8192, k/v 1024x8192, gate/up
    28672x8192 (235 M weights) and down 8192x28672."""
    wl = synth.llama3_70b_block()
    for name in ("q_proj", "k_proj", "gate_proj", "down_proj"):
        spec = wl.layers[name]
        w = synth.weights(spec)
        idx = sample_rows(spec.rows, n=16, seed=spec.seed)
        for mode in MODES:
            run_case(w, True, 32, 2, mode, rows_idx=idx, tag=name)


def test_quantize_inside_a_side_stream():
    """A quantize call inside torch.cuda.stream(s), between a producer and a consumer
    queued on s, sees the producer's W and its outputs are seen by the consumer."""
    w = random_bf16(4096, 4096, seed=21)
    src = to_device(w, True)
    ref_codes, ref_scales, _ = ssq.ssq_quantize(src, 32, 4, O.SIGNED_SYM)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        W = torch.empty_like(src)
        W.copy_(src)                                    # producer on s
        codes, scales, _ = ssq.ssq_quantize(W, 32, 4, O.SIGNED_SYM)
        codes_seen, scales_seen = codes.clone(), scales.clone()   # consumers on s
    s.synchronize()
    assert torch.equal(codes_seen, ref_codes) and torch.equal(scales_seen, ref_scales)
