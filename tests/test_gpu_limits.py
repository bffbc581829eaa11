"""GPU parity at the boundary's largest reduction length (K = 2^22, the ABI limit set by
32-bit buffer offsets), through every kernel family: quantize, GEMV, batched decode with
its split reduction, the prefill GEMM with its split reduction, Q8_0 and the sign-rule
diagnostics.  Few rows, so the oracle stays cheap."""
import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import log_metric, rel_l2, to_device, y_to_f64

pytestmark = pytest.mark.gpu

KMAX = 1 << 22


def weights(N, K, seed):
    rng = np.random.default_rng(seed)
    w = rng.standard_t(5, size=(N, K)).astype(np.float32) * 0.02
    return synth.to_bf16_bits(w)


def quantized(wb, group, q, mode=O.SIGNED_SYM):
    codes, scales, zp = ssq.ssq_quantize(to_device(wb, True), group, q, mode)
    torch.cuda.synchronize()
    r = O.quantize(O.bf16_bits_to_f32(wb), group, q, mode)
    assert np.array_equal(codes.cpu().numpy(), r.codes), "codes"
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), r.scales), "scales"
    return (codes, scales, zp), r


def check(y, ref, tag, bar=2e-2):
    err = rel_l2(y_to_f64(y), ref)
    log_metric(test="limits", tag=tag, rel_l2=err)
    assert err <= bar, f"{tag}: rel L2 {err:.2e}"


def test_gemv_and_q8_at_max_k():
    N = 5                                                  # ragged: one full and one partial row group
    wb = weights(N, KMAX, seed=1)
    dev, r = quantized(wb, 128, 4, O.ASYM)
    x = synth.activations(1, KMAX, seed=2)
    y = ssq.ssq_matmul(to_device(x, True), *dev, N, KMAX, 128, 4)
    check(y, O.matmul(O.bf16_bits_to_f32(x), r.codes, r.scales, r.zp, N, KMAX, 128, 4), "gemv K=2^22")
    qx, dx = ssq.ssq_quantize_act_q8(to_device(x, True))
    yq = ssq.ssq_matmul_q8(qx, dx, *dev, N, KMAX, 128, 4)
    torch.cuda.synchronize()
    a = O.quantize_act_q8(O.bf16_bits_to_f32(x))
    assert np.array_equal(qx.cpu().numpy(), a.q) and np.array_equal(dx.cpu().numpy().view(np.uint16), a.d)
    check(yq, O.matmul_q8(a.q, a.d, r.codes, r.scales, r.zp, N, KMAX, 128, 4), "q8 gemv K=2^22", bar=5e-3)


@pytest.mark.parametrize("M", [16, 40])
def test_split_kernels_at_max_k(M):
    """M = 16: batched decode; M = 40: the GEMM; both with the split reduction (the
    largest slice counts) and a ragged weight row block."""
    N = 20
    wb = weights(N, KMAX, seed=M)
    dev, r = quantized(wb, 32, 4)
    x = synth.activations(M, KMAX, seed=M + 1)
    ws = ssq.ssq_matmul_workspace(M, N, KMAX, 32, 4)
    assert ws is not None
    y = ssq.ssq_matmul(to_device(x, True), *dev, N, KMAX, 32, 4, workspace=ws)
    check(y, O.matmul(O.bf16_bits_to_f32(x), r.codes, r.scales, r.zp, N, KMAX, 32, 4), f"split M={M} K=2^22")


def test_diagnostics_at_max_k():
    wb = weights(3, KMAX, seed=7)
    W = to_device(wb, True)
    margin, gain, tally = ssq.ssq_sign_diagnostics(W, 32, 2)
    torch.cuda.synchronize()
    d = O.sign_diagnostics(O.bf16_bits_to_f32(wb), 32, 2)
    assert np.array_equal(margin.cpu().numpy(), d.margin)
    assert np.array_equal(gain.cpu().numpy(), d.gain)
    assert np.array_equal(tally.cpu().numpy(), d.tally)
