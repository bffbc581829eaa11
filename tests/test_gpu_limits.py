"""GPU parity at the boundary's largest reduction length (K = 2^22, the ABI limit set by
32-bit buffer offsets), through every kernel family: quantize, GEMV, batched decode with
its split reduction, the prefill GEMM with its split reduction, Q8_0 and the sign-rule
diagnostics.  Few rows, so the oracle stays cheap."""
import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import assert_within, log_metric, matmul_error_bound, rel_l2, to_device, y_to_f64

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


def check(y, x_bits, r, K, group, q, tag, rows=None):
    """Element-wise against the oracle (tests/parity_common.py's bound: M <= 2 keeps the
    weights exact, larger M rounds them to bf16) and the workloads' rel L2 bar."""
    x = O.bf16_bits_to_f32(x_bits)
    ref = O.matmul(x, r.codes, r.scales, r.zp, r.codes.shape[0], K, group, q)
    w_hat = O.dequantize(r.codes, r.scales, r.zp, K, group, q)
    bound, _ = matmul_error_bound(x, w_hat, ref, rounded_weights=x.shape[0] > 2, f32=False)
    y_all = y_to_f64(y)
    got = y_all if rows is None else y_all[:, rows]
    worst = assert_within(got, ref, bound, tag)
    err = rel_l2(got, ref)
    log_metric(test="limits", tag=tag, rel_l2=err, max_err_over_bound=worst)
    assert err <= 2e-2, f"{tag}: rel L2 {err:.2e}"


def test_gemv_and_q8_at_max_k():
    N = 5                                                  # ragged: one full and one partial row group
    wb = weights(N, KMAX, seed=1)
    dev, r = quantized(wb, 128, 4, O.ASYM)
    x = synth.activations(1, KMAX, seed=2)
    y = ssq.ssq_matmul(to_device(x, True), *dev, N, KMAX, 128, 4)
    check(y, x, r, KMAX, 128, 4, "gemv K=2^22")
    qx, dx = ssq.ssq_quantize_act_q8(to_device(x, True))
    yq = ssq.ssq_matmul_q8(qx, dx, *dev, N, KMAX, 128, 4)
    torch.cuda.synchronize()
    a = O.quantize_act_q8(O.bf16_bits_to_f32(x))
    assert np.array_equal(qx.cpu().numpy(), a.q) and np.array_equal(dx.cpu().numpy().view(np.uint16), a.d)
    ref = O.matmul_q8(a.q, a.d, r.codes, r.scales, r.zp, N, KMAX, 128, 4)
    got = y_to_f64(yq)
    tol = 2.0 ** -8 * np.abs(ref) + 1e-5 * np.abs(ref).max(axis=1, keepdims=True) + 1e-30
    assert_within(got, ref, tol, "q8 gemv K=2^22")
    assert rel_l2(got, ref) <= 5e-3


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
    check(y, x, r, KMAX, 32, 4, f"split M={M} K=2^22")


def test_diagnostics_at_max_k():
    wb = weights(3, KMAX, seed=7)
    W = to_device(wb, True)
    margin, gain, tally = ssq.ssq_sign_diagnostics(W, 32, 2)
    torch.cuda.synchronize()
    d = O.sign_diagnostics(O.bf16_bits_to_f32(wb), 32, 2)
    assert np.array_equal(margin.cpu().numpy(), d.margin)
    assert np.array_equal(gain.cpu().numpy(), d.gain)
    assert np.array_equal(tally.cpu().numpy(), d.tally)


def test_large_row_count():
    """Two million and three weight rows (K = 64): grids of 2^19 GEMV workgroups and 2^14
    batched-decode and GEMM row blocks, ragged at the end.  Quantize, the GEMV at M = 1
    and 2, batched decode (M = 16) and the GEMM (M = 40) with their workspaces, and the
    sign-rule diagnostics, each against the oracle on sampled rows (the last ones
    included); the tally against the counts of the full outputs."""
    N, K, group, q = (1 << 21) + 3, 64, 32, 4
    rng = np.random.default_rng(11)
    wb = synth.to_bf16_bits(rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02))
    W = to_device(wb, True)
    rows = np.unique(np.concatenate([rng.choice(N, 61, replace=False), np.arange(N - 3, N)]))
    wf = O.bf16_bits_to_f32(wb[rows])
    codes, scales, zp = ssq.ssq_quantize(W, group, q, O.SIGNED_SYM)
    torch.cuda.synchronize()
    r = O.quantize(wf, group, q, O.SIGNED_SYM)
    assert np.array_equal(codes.cpu().numpy()[rows], r.codes)
    assert np.array_equal(scales.cpu().numpy().view(np.uint16)[rows], r.scales)
    for M in (1, 2, 16, 40):
        x = synth.activations(M, K, seed=M)
        ws = ssq.ssq_matmul_workspace(M, N, K, group, q)
        y = ssq.ssq_matmul(to_device(x, True), codes, scales, zp, N, K, group, q, workspace=ws)
        check(y, x, r, K, group, q, f"N=2^21+3 M={M}", rows=rows)
    margin, gain, tally = ssq.ssq_sign_diagnostics(W, group, q)
    torch.cuda.synchronize()
    d = O.sign_diagnostics(wf, group, q)
    m, g = margin.cpu().numpy(), gain.cpu().numpy()
    assert np.array_equal(m[rows], d.margin) and np.array_equal(g[rows], d.gain)
    counts = np.zeros((3, 3), np.int64)
    np.add.at(counts, (np.sign(m).astype(np.int64) + 1, np.sign(g).astype(np.int64) + 1), 1)
    assert np.array_equal(tally.cpu().numpy(), counts)
