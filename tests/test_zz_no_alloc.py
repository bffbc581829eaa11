"""ssq_matmul_noalloc (the entry point for callers that cannot allocate) through the C
ABI against ssq_matmul_ws with a fresh workspace of ssq_matmul_workspace_size() bytes:
the same kernels and split plan, so the outputs must agree bit for bit, and both must
meet the element-wise oracle bound.  Several calls in a row share the static scratch,
each later one smaller (fewer tiles or row blocks, so stale partials and counters of
the earlier call sit where the later call could trip over them)."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import Guarded, sample_rows, to_device, weights_host, widen
from tests.test_gpu_matmul import compare_matmul

pytestmark = pytest.mark.gpu


def run_noalloc(x, codes, scales, zp, N, K, group, q, y):
    st = ssq.lib().ssq_matmul_noalloc(ctypes.c_void_p(x.data_ptr()), x.shape[0],
                                      ctypes.c_void_p(codes.data_ptr()), ctypes.c_void_p(scales.data_ptr()),
                                      None if zp is None else ctypes.c_void_p(zp.data_ptr()), N, K, group, q,
                                      ctypes.c_void_p(y.data_ptr()),
                                      ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, ssq.ssq_strerror(st)


CASES = [
    # (M, N, K, q, group, mode, weight seed): prefill headline (GEMM split 4 ways), a ragged
    # GEMM split, batched decode split, a plain GEMV (no scratch), batched decode split again
    (512, 4096, 14336, 4, 32, O.SIGNED_SYM, 4006),
    (130, 200, 3104, 3, 32, O.ASYM, 11),
    (16, 300, 8192, 4, 32, O.SIGNED_SYM, 12),
    (1, 96, 1024, 2, 64, O.SIGNED_SYM, 13),
    (7, 200, 3072, 2, 128, O.UNSIGNED_SYM, 14),
]


def test_noalloc_matches_workspace_entry_point_over_consecutive_calls():
    for M, N, K, q, group, mode, seed in CASES:
        tag = f"noalloc M={M} N={N} K={K} q={q} g={group} mode={mode}"
        print(tag, flush=True)
        spec = synth.WeightSpec(N, K, nu=5.0, scale=0.02, outlier_frac=0.001, seed=seed)
        w = weights_host(spec)
        codes, scales, zp = ssq.ssq_quantize(to_device(w, True), group, q, mode)
        x_host = synth.activations(M, K, seed=seed + 1)
        x = to_device(x_host, True)
        y = Guarded((M, N), torch.bfloat16)
        run_noalloc(x, codes, scales, zp, N, K, group, q, y.t)
        y.check(tag)
        ws = ssq.ssq_matmul_workspace(M, N, K, group, q)
        y_ws = ssq.ssq_matmul(x, codes, scales, zp, N, K, group, q, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(y.t.view(torch.int16), y_ws.view(torch.int16)), f"{tag}: differs from ssq_matmul_ws"
        rows = sample_rows(N, n=24, seed=seed) if N > 64 else np.arange(N)
        ref_q = O.quantize(widen(w[rows], True), group, q, mode)
        # the static scratch serves as the split workspace: the same kernel as ssq_matmul_ws
        compare_matmul(y.t, widen(x_host, True), ref_q, rows, K, group, q, True, tag, workspace=True)


def test_noalloc_inside_a_graph():
    """Captured in a HIP graph and replayed, with eager calls of the entry point between
    replays: every replay and every eager call equals the workspace entry point."""
    M, N, K = 64, 256, 8192
    w = synth.weights(synth.WeightSpec(N, K, nu=5.0, scale=0.02, seed=21))
    codes, scales, _ = ssq.ssq_quantize(to_device(w, True), 32, 4, O.SIGNED_SYM)
    x = to_device(synth.activations(M, K, seed=22), True)
    ws = ssq.ssq_matmul_workspace(M, N, K, 32, 4)
    assert ws is not None
    want = ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4, workspace=ws)
    y = torch.empty_like(want)
    other = torch.empty_like(want)
    run_noalloc(x, codes, scales, None, N, K, 32, 4, y)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            run_noalloc(x, codes, scales, None, N, K, 32, 4, y)
    for _ in range(3):
        y.zero_()
        g.replay()
        torch.cuda.synchronize()
        run_noalloc(x, codes, scales, None, N, K, 32, 4, other)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), want.view(torch.int16))
        assert torch.equal(other.view(torch.int16), want.view(torch.int16))
