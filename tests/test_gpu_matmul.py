"""GPU parity: ssq_matmul (GEMV at M = 1, 2, skinny-M MFMA kernel at 3 <= M <= 32, tiled
MFMA GEMM above) and ssq_matmul_f32 against the binary64 CPU oracle.

Every comparison is element-wise (tests/parity_common.py states the bound and its
derivation): one bf16 rounding of the output plus binary32 accumulation slack, plus,
on the MFMA paths that round each dequantized weight to bf16, C_W = 6 times the
standard scale of that rounding; the symmetric and zero-point formats on the MFMA
paths are also held to the exact model x bf16(W_hat)^T.  The binary32 path is held to
1e-5.  The relative L2 bar of the workloads (2e-2 bf16, 1e-3 binary32) is asserted
too.  Every output (and workspace) sits between guard bytes that are checked after
the call, and starts as NaN so an unwritten output fails.
"""
import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import (Guarded, assert_quant_equal, assert_within, bf16_round_f64,
                                 guarded_quant_outputs, log_metric, matmul_error_bound, rel_l2,
                                 sample_rows, to_device, weights_host, widen, y_to_f64)

pytestmark = pytest.mark.gpu

MODES = [O.SIGNED_SYM, O.UNSIGNED_SYM, O.ASYM, O.ASYM_MIN]
TOL_BF16 = 2e-2
TOL_F32 = 1e-3


def quantize_guarded(W, rows, cols, group, q, mode, tag=""):
    """ssq_quantize into guarded buffers; returns the plain tensors after checking the guards."""
    g = guarded_quant_outputs(rows, cols, group, q, mode)
    out = ssq.ssq_quantize(W, group, q, mode, out=tuple(b.t if b is not None else None for b in g))
    for b in g:
        if b is not None:
            b.check(f"{tag} quantize")
    return out


def exact_weight_path(M, K, q, workspace):
    """Whether ssq_matmul runs the activation-stationary batched-decode kernel: q = 2 or
    4, 3 <= M <= 16, K a multiple of a wavefront's range of 512 weights and either a
    workspace or at most four ranges (one slice of K).  It keeps every weight exact,
    where the dequantizing MFMA kernels round s (u - o) to bf16, so it is held to the
    exact-weight bound."""
    if q not in (2, 4) or not 3 <= M <= 16:
        return False
    return K % 512 == 0 and (workspace or K <= 2048)


def compare_matmul(y, x_real, ref_q, sel, K, group, q, bf16_x, tag, workspace=False):
    """Element-wise comparison of y[:, sel] (a GPU tensor) with the oracle; returns rel L2."""
    M = x_real.shape[0]
    y_ref = O.matmul(x_real, ref_q.codes, ref_q.scales, ref_q.zp, len(sel), K, group, q, mins=ref_q.mins)
    w_hat = O.dequantize(ref_q.codes, ref_q.scales, ref_q.zp, K, group, q, ref_q.mins)
    # batched decode and prefill round W_hat to bf16, except the activation-stationary kernel
    rounded = bf16_x and M > 2 and not exact_weight_path(M, K, q, workspace)
    bound, S = matmul_error_bound(x_real, w_hat, y_ref, rounded, f32=not bf16_x)
    y_all = y_to_f64(y)
    assert not np.isnan(y_all).any(), f"{tag}: output elements left unwritten (NaN fill)"
    y_gpu = y_all[:, sel]
    worst = assert_within(y_gpu, y_ref, bound, tag)
    worst_model = None
    if rounded and ref_q.mins is None:
        y_model = np.asarray(x_real, np.float64) @ bf16_round_f64(w_hat).T
        bound_m = 2.0 ** -8 * np.abs(y_model) + 2.0 ** -12 * S
        worst_model = assert_within(y_gpu, y_model, bound_m, f"{tag} (bf16 weight model)")
    err = rel_l2(y_gpu, y_ref)
    log_metric(test=tag, M=M, N=int(ref_q.codes.shape[0]), K=K, q=q, group=group, rel_l2=err,
               max_err_over_bound=worst, max_err_over_model_bound=worst_model,
               dtype="bf16" if bf16_x else "f32")
    tol = TOL_BF16 if bf16_x else TOL_F32
    assert err <= tol, f"{tag}: rel L2 {err:.3e} > {tol}"
    return err


def check_matmul(w_host, x_host, group, q, mode, rows_idx=None, bf16_w=True, bf16_x=True, tag="",
                 workspace=False, repeat=1, need_split=True):
    """Quantize on the GPU, multiply on the GPU, compare with the oracle on rows_idx.
    With workspace=True the split-reduction entry point runs `repeat` times on one
    workspace and every result is checked (need_split=False: shapes whose plan does not
    split run without one)."""
    N, K = w_host.shape
    M = x_host.shape[0]
    W = to_device(w_host, bf16_w)
    codes, scales, zp = quantize_guarded(W, N, K, group, q, mode, tag=tag)
    X = to_device(x_host, bf16_x)
    ws = None
    if workspace:
        nbytes = ssq.ssq_matmul_workspace_size(M, N, K, group, q)
        assert nbytes > 0 or not need_split, "shape chosen to need a split"
        ws = Guarded((nbytes,), torch.uint8, fill=0) if nbytes else None
    sel = np.arange(N) if rows_idx is None else rows_idx
    ref_q = O.quantize(widen(w_host[sel], bf16_w), group, q, mode)
    assert_quant_equal((codes, scales, zp), ref_q, None if rows_idx is None else sel, tag=tag)
    xr = widen(x_host, bf16_x)
    err = None
    for r in range(repeat):          # same workspace, same answer every call
        y = Guarded((M, N), torch.bfloat16 if bf16_x else torch.float32)
        ssq.ssq_matmul(X, codes, scales, zp, N, K, group, q, out=y.t,
                       workspace=None if ws is None else ws.t)
        y.check(f"{tag} y (call {r})")
        if ws is not None:
            ws.check(f"{tag} workspace (call {r})")
        err = compare_matmul(y.t, xr, ref_q, sel, K, group, q, bf16_x, f"{tag} (call {r})",
                             workspace=ws is not None)
    return err


def rand_w(N, K, seed, bf16=True):
    return synth.weights(synth.WeightSpec(N, K, nu=5.0, scale=0.02, outlier_frac=0.001,
                                          seed=seed, bf16=bf16))


# ---------------------------------------------------------------------------
# Small and ragged cases, every format.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", MODES)
def test_gemv_small_all_formats(q, group, mode):
    w = rand_w(37, 1536, seed=10 * q + group)
    x = synth.activations(1, 1536, seed=q)
    check_matmul(w, x, group, q, mode, tag="gemv 37x1536")


@pytest.mark.parametrize("K", [32, 64, 4096 + 32])
def test_gemv_odd_reduction_lengths(K):
    w = rand_w(9, K, seed=K)
    x = synth.activations(1, K, seed=K)
    for mode in MODES:
        check_matmul(w, x, 32, 4, mode, tag=f"gemv K={K}")


@pytest.mark.parametrize("q,group", [(4, 32), (3, 64), (2, 128)])
def test_gemv_multi_pass_ragged(q, group):
    # K=17408 is 544 blocks: two passes of a 320-thread team, the second one partial.
    K = 17408
    w = rand_w(21, K, seed=q + group)
    x = synth.activations(1, K, seed=5)
    for mode in MODES:
        check_matmul(w, x, group, q, mode, tag=f"gemv multi-pass q={q} g={group}")


@pytest.mark.parametrize("mode", MODES)
def test_gemv_unaligned_metadata(mode):
    """Scales (and zero points) that start off a 16-byte boundary take the per-lane
    load path; the result equals the aligned call bit for bit."""
    N, K = 24, 2048
    w = rand_w(N, K, seed=3)
    codes, scales, zp = ssq.ssq_quantize(to_device(w, True), 32, 4, mode)
    X = to_device(synth.activations(1, K, seed=4), True)
    y_ref = ssq.ssq_matmul(X, codes, scales, zp, N, K, 32, 4)
    s_buf = torch.zeros(scales.numel() + 8, dtype=scales.dtype, device="cuda")
    s_off = s_buf[1:1 + scales.numel()].view(scales.shape)
    s_off.copy_(scales)
    z_off = None
    if zp is not None:
        z_buf = torch.zeros(zp.numel() + 16, dtype=zp.dtype, device="cuda")
        z_off = z_buf[3:3 + zp.numel()].view(zp.shape)
        z_off.copy_(zp)
    assert s_off.data_ptr() % 16 != 0
    y = ssq.ssq_matmul(X, codes, s_off, z_off, N, K, 32, 4)
    torch.cuda.synchronize()
    assert torch.equal(y, y_ref)


@pytest.mark.parametrize("M", [16, 96, 300])
@pytest.mark.parametrize("mode", MODES)
def test_matmul_unaligned_metadata(M, mode):
    """Batched decode and the GEMM with scales (and zero points or minimums) that start
    off a 4-byte boundary (offsets of one element): the result equals the aligned call
    bit for bit, with and without the split workspace."""
    N, K = 200, 1056
    w = rand_w(N, K, seed=31)
    codes, scales, zp = ssq.ssq_quantize(to_device(w, True), 32, 4, mode)
    X = to_device(synth.activations(M, K, seed=32), True)
    s_buf = torch.zeros(scales.numel() + 8, dtype=scales.dtype, device="cuda")
    s_off = s_buf[1:1 + scales.numel()].view(scales.shape)
    s_off.copy_(scales)
    z_off = None
    if zp is not None:
        z_buf = torch.zeros(zp.numel() + 16, dtype=zp.dtype, device="cuda")
        z_off = z_buf[3:3 + zp.numel()].view(zp.shape) if zp.dtype == torch.uint8 else \
            z_buf[1:1 + zp.numel()].view(zp.shape)
        z_off.copy_(zp)
    assert s_off.data_ptr() % 4 != 0
    for ws in (None, ssq.ssq_matmul_workspace(M, N, K, 32, 4)):
        y_ref = ssq.ssq_matmul(X, codes, scales, zp, N, K, 32, 4, workspace=ws)
        y = ssq.ssq_matmul(X, codes, s_off, z_off, N, K, 32, 4, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 128])
@pytest.mark.parametrize("mode", MODES)
def test_gemm_ragged_all_formats(q, group, mode):
    # M=200, N=300 leave partial 128x128 tiles in both directions; at g=32, K=1056 is an odd
    # number of 32-blocks (half of the last 64-deep step is empty)
    K = 1056 if group == 32 else 1152
    w = rand_w(300, K, seed=7 * q + group)
    x = synth.activations(200, K, seed=q + group)
    check_matmul(w, x, group, q, mode, tag=f"gemm 200x300x{K}")


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", MODES)
def test_skinny_all_formats(q, group, mode):
    # batched decode (2 <= M <= 32): N=45 leaves a partial 16-row workgroup; K is an odd
    # number of 32-blocks at g=32 and g=64, so the last 128-wide super-block is partial
    K = {32: 1056, 64: 1088, 128: 1152}[group]
    w = rand_w(45, K, seed=3 * q + group + mode)
    x = synth.activations(7, K, seed=q * group)
    check_matmul(w, x, group, q, mode, tag=f"skinny 7x45x{K}")


@pytest.mark.parametrize("M", [2, 15, 16, 17, 31, 32])
def test_skinny_token_counts(M):
    # one and two 16-token MFMA blocks, both partial and full; K=14336 spreads 112
    # super-blocks over 16 wavefronts
    w = rand_w(40, 14336, seed=M)
    x = synth.activations(M, 14336, seed=M)
    for mode in MODES:
        check_matmul(w, x, 32, 4, mode, tag=f"skinny M={M}")


@pytest.mark.parametrize("K", [32, 64, 128, 4096 + 96])
def test_skinny_short_and_odd_reductions(K):
    # fewer super-blocks than wavefronts, a lone partial super-block, a partial last one
    w = rand_w(33, K, seed=K + 1)
    x = synth.activations(16, K, seed=K + 1)
    for mode in MODES:
        check_matmul(w, x, 32, 3, mode, tag=f"skinny K={K}")


@pytest.mark.parametrize("K", [32, 64, 96, 128, 192])
@pytest.mark.parametrize("mode", [O.SIGNED_SYM, O.ASYM])
def test_gemm_short_reductions(K, mode):
    # one or two 64-deep windows per tile: the loads of the window after the last one
    # (issued at the start of the tile, or by the last window) lie past K and read
    # nothing the result uses; signed scales take the two-window start, zero points not
    w = rand_w(300, K, seed=K + mode)
    x = synth.activations(200, K, seed=K)
    check_matmul(w, x, 32, 4, mode, tag=f"gemm 200x300x{K}")


@pytest.mark.parametrize("M", [2, 3, 16, 32, 33, 129])
def test_gemm_small_token_counts(M):
    w = rand_w(64, 512, seed=M)
    x = synth.activations(M, 512, seed=M)
    check_matmul(w, x, 32, 4, O.SIGNED_SYM, tag=f"gemm M={M}")


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("mode", MODES)
def test_gemm_split_reduction_ragged(q, mode):
    # 4 output tiles (130x200) over K=3104 (97 blocks, 49 steps): split 3 ways, the last
    # slice carrying the odd half-step; three calls on one workspace
    w = rand_w(200, 3104, seed=q + 10 * mode)
    x = synth.activations(130, 3104, seed=q)
    check_matmul(w, x, 32, q, mode, tag="split 130x200x3104", workspace=True, repeat=3)


@pytest.mark.parametrize("M,N,K", [(2048, 5120, 4096), (2000, 4700, 4096)])
@pytest.mark.parametrize("mode", [O.SIGNED_SYM, O.ASYM_MIN])
def test_gemm_split_last_round(M, N, K, mode):
    # more output tiles than CUs (320, and a ragged 296) with a last round less than half
    # full: those tiles (the weight panels from row 4096 on) are cut into K slices
    # through the workspace while the others are computed whole
    w = rand_w(N, K, seed=N + mode)
    x = synth.activations(M, K, seed=M)
    rows = np.concatenate([sample_rows(4096, n=8, seed=1), 4096 + sample_rows(N - 4096, n=40, seed=2)])
    check_matmul(w, x, 32, 4, mode, rows_idx=rows, tag=f"split last round {M}x{N}x{K}", workspace=True,
                 repeat=2)


def test_gemm_output_past_one_gigabyte():
    """A 4096 x 131072 bf16 output (1 GiB): the GEMM stores it with 64-bit addresses rather
    than through a buffer descriptor; sampled rows against the oracle, guards checked."""
    N, K, M = 131072, 512, 4096
    w = rand_w(N, K, seed=17)
    x = synth.activations(M, K, seed=17)
    rows = np.concatenate([sample_rows(N, n=24, seed=5), np.array([N - 129, N - 128, N - 127])])
    check_matmul(w, x, 32, 4, O.SIGNED_SYM, rows_idx=np.unique(rows), tag="gemm 4096x131072x512 (1 GiB y)")


def test_gemm_split_reduction_eight_ways():
    w = rand_w(160, 8192, seed=5)
    x = synth.activations(64, 8192, seed=5)
    check_matmul(w, x, 128, 4, O.SIGNED_SYM, tag="split 64x160x8192", workspace=True, repeat=2)


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("mode", MODES)
def test_skinny_split_reduction_ragged(q, mode):
    # batched decode with a workspace: N=200 is two 128-row blocks (the second partial),
    # K=3104 has 25 super-blocks (the last one partial) over 12 slices (the last three
    # empty); three calls on one workspace
    w = rand_w(200, 3104, seed=q + 10 * mode + 1)
    x = synth.activations(7, 3104, seed=q + 1)
    check_matmul(w, x, 32, q, mode, tag="skinny split 7x200x3104", workspace=True, repeat=3)


@pytest.mark.parametrize("M", [3, 16, 17, 32])
@pytest.mark.parametrize("group", [32, 128])
def test_skinny_split_token_counts(M, group):
    w = rand_w(300, 8192, seed=M + group)
    x = synth.activations(M, 8192, seed=M + group)
    for mode in MODES:
        check_matmul(w, x, group, 4, mode, tag=f"skinny split M={M}", workspace=True, repeat=2)


# Activation-stationary batched decode (q = 2, 4; K a multiple of the wavefront range).

@pytest.mark.parametrize("M", [5, 16])
@pytest.mark.parametrize("q", [2, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", MODES)
def test_stationary_all_formats(M, q, group, mode):
    # N=45: three 16-row tiles, the last one partial.  K=2560: five 512-wide ranges, two
    # slices of four wavefronts (the second with one live); two calls on one workspace
    assert exact_weight_path(M, 2560, q, True)
    w = rand_w(45, 2560, seed=100 + 7 * q + group + mode + M)
    x = synth.activations(M, 2560, seed=q * group + M)
    check_matmul(w, x, group, q, mode, tag=f"stationary {M}x45x2560", workspace=True, repeat=2)


@pytest.mark.parametrize("q", [2, 4])
@pytest.mark.parametrize("M,N,K,workspace", [
    (16, 6400, 4096, True),     # two slices, 400 tiles: runs of two tiles
    (9, 9600, 6144, True),      # three slices, 600 tiles: runs of four, the last one short
    (13, 4100, 3072, True),     # a 4-row last tile and a tile past N in the last run
    (16, 2000, 1024, False),    # one slice (two live wavefronts): no workspace, y per tile
])
def test_stationary_runs(q, M, N, K, workspace):
    assert exact_weight_path(M, K, q, workspace)
    w = rand_w(N, K, seed=N + K + q)
    x = synth.activations(M, K, seed=M + q)
    for mode in (O.SIGNED_SYM, O.ASYM_MIN):
        check_matmul(w, x, 32, q, mode, rows_idx=sample_rows(N, n=48, seed=q), tag=f"stationary runs {M}x{N}x{K}",
                     workspace=workspace, repeat=2 if workspace else 1, need_split=False)


@pytest.mark.parametrize("M,N,K", [(96, 256, 8192), (300, 256, 8192), (16, 256, 8192)])
def test_split_reduction_graph_replay(M, N, K):
    """The split kernels in a HIP graph: the arrival counters reset inside the kernel, so
    every replay (with eager work between) reproduces the first result."""
    w = rand_w(N, K, seed=8)
    W = to_device(w, True)
    codes, scales, _ = ssq.ssq_quantize(W, 32, 4, O.SIGNED_SYM)
    x_host = synth.activations(M, K, seed=8)
    x = to_device(x_host, True)
    ws = ssq.ssq_matmul_workspace(M, N, K, 32, 4)
    assert ws is not None
    y_eager = ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4, workspace=ws)
    ref_q = O.quantize(widen(w, True), 32, 4, O.SIGNED_SYM)
    compare_matmul(y_eager, widen(x_host, True), ref_q, np.arange(N), K, 32, 4, True, f"graph split M={M}",
                   workspace=True)
    y = torch.empty_like(y_eager)
    ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4, out=y, workspace=ws)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4, out=y, workspace=ws)
    for _ in range(4):
        y.zero_()
        graph.replay()
        other = ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), y_eager.view(torch.int16))
        assert rel_l2(y_to_f64(other), y_to_f64(y_eager)) < 1e-2


@pytest.mark.parametrize("M", [1, 3, 5])
@pytest.mark.parametrize("mode", MODES)
def test_f32_path(M, mode):
    spec = synth.small_fp32().layers["w"]
    w = weights_host(spec)
    x = synth.activations(M, 512, seed=1100 + M, bf16=False)
    check_matmul(w, x, 32, 4, mode, bf16_w=False, bf16_x=False, tag=f"f32 256x512 M={M}")


def test_f32_path_other_formats():
    w = synth.weights(synth.WeightSpec(50, 768, nu=4.0, scale=0.02, seed=8, bf16=False))
    x = synth.activations(2, 768, seed=8, bf16=False)
    for q in (2, 3):
        for group in (64, 128):
            check_matmul(w, x, group, q, O.ASYM, bf16_w=False, bf16_x=False, tag="f32 other")


def test_zero_weights_give_zero_output():
    w = np.zeros((16, 256), np.uint16)
    for M in (1, 4):
        x = synth.activations(M, 256, seed=M)
        for mode in MODES:
            W = to_device(w, True)
            codes, scales, zp = ssq.ssq_quantize(W, 32, 4, mode)
            y = ssq.ssq_matmul(to_device(x, True), codes, scales, zp, 16, 256, 32, 4)
            torch.cuda.synchronize()
            assert (y.float() == 0).all()


def test_empty_matmul_is_a_noop():
    codes = torch.zeros((8, 32), dtype=torch.uint8, device="cuda")
    scales = torch.zeros((8, 2), dtype=torch.int16, device="cuda")
    y = ssq.ssq_matmul(torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda"),
                       codes, scales, None, 8, 64, 32, 4)
    assert y.shape == (0, 8)
    y = ssq.ssq_matmul(torch.zeros((3, 64), dtype=torch.bfloat16, device="cuda"),
                       codes, scales, None, 0, 64, 32, 4)
    torch.cuda.synchronize()
    assert y.shape == (3, 0)


@pytest.mark.parametrize("M", [1, 16, 64])
def test_graph_replay_matches_eager(M):
    """ssq_matmul captured in a HIP graph: every replay, with eager work in between,
    equals the eager result bit for bit."""
    N, K = 256, 2048
    w = rand_w(N, K, seed=77)
    W = to_device(w, True)
    codes, scales, _ = ssq.ssq_quantize(W, 32, 4, O.SIGNED_SYM)
    x_host = synth.activations(M, K, seed=M)
    x = to_device(x_host, True)
    y_eager = ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4)
    ref_q = O.quantize(widen(w, True), 32, 4, O.SIGNED_SYM)
    compare_matmul(y_eager, widen(x_host, True), ref_q, np.arange(N), K, 32, 4, True, f"graph M={M}")
    y = torch.empty_like(y_eager)
    ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4, out=y)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4, out=y)
    for _ in range(4):
        y.zero_()
        graph.replay()
        scratch = ssq.ssq_matmul(x, codes, scales, None, N, K, 32, 4)   # eager work between
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), y_eager.view(torch.int16))
        assert torch.equal(scratch.view(torch.int16), y_eager.view(torch.int16))


# ---------------------------------------------------------------------------
# Full-size workloads (sampled output columns).
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode", MODES)
def test_llama3_8b_decode_gemv_full_size(mode):
    wl = synth.llama3_8b_decode()
    for name, spec in wl.layers.items():
        w = weights_host(spec)
        x = synth.activations(1, spec.cols, seed=wl.x_seed)
        check_matmul(w, x, 32, 4, mode, rows_idx=sample_rows(spec.rows, seed=spec.seed),
                     tag=f"decode {name}")


@pytest.mark.parametrize("q", [2, 3])
@pytest.mark.parametrize("group", [32, 64, 128])
def test_llama3_8b_block_gemv_full_size(q, group):
    wl = synth.llama3_8b_block()
    for name in ("q_proj", "k_proj", "gate_proj", "down_proj"):
        spec = wl.layers[name]
        w = weights_host(spec)
        x = synth.activations(1, spec.cols, seed=wl.x_seed)
        for mode in MODES:
            check_matmul(w, x, group, q, mode, rows_idx=sample_rows(spec.rows, n=24, seed=1),
                         tag=f"block {name}")


@pytest.mark.parametrize("M", [512, 2048])
@pytest.mark.parametrize("layer", ["gate_proj", "down_proj"])
def test_prefill_gemm_full_size(M, layer):
    wl = synth.prefill()
    spec = wl.layers[layer]
    w = weights_host(spec)
    x = synth.activations(M, spec.cols, seed=wl.x_seed + M)
    check_matmul(w, x, 32, 4, O.SIGNED_SYM, rows_idx=sample_rows(spec.rows, n=32, seed=M),
                 tag=f"prefill {layer} M={M}")


def test_prefill_gate_split_last_round_full_size():
    """M=2048 on the 14336x4096 gate projection with a workspace: 896 tiles, the last 128
    (rows 12288 on) cut in two K slices."""
    wl = synth.prefill()
    spec = wl.layers["gate_proj"]
    w = weights_host(spec)
    x = synth.activations(2048, spec.cols, seed=wl.x_seed + 2048)
    rows = np.concatenate([sample_rows(12288, n=8, seed=3), 12288 + sample_rows(spec.rows - 12288, n=24, seed=4)])
    check_matmul(w, x, 32, 4, O.SIGNED_SYM, rows_idx=rows, tag="prefill gate_proj M=2048 split last round",
                 workspace=True, repeat=2)


def test_prefill_headline_split_full_size():
    """M=512 on the 4096x14336 down projection through the split-reduction entry point."""
    wl = synth.prefill()
    spec = wl.layers["down_proj"]
    w = weights_host(spec)
    x = synth.activations(512, spec.cols, seed=wl.x_seed + 512)
    check_matmul(w, x, 32, 4, O.SIGNED_SYM, rows_idx=sample_rows(spec.rows, n=32, seed=9),
                 tag="prefill down_proj M=512 split", workspace=True, repeat=2)


@pytest.mark.parametrize("M", [16, 32])
def test_llama3_8b_batched_decode_full_size(M):
    """Batched decode through the split-reduction entry point on every Llama-3-8B
    projection shape, q=4 g=32, sampled rows; both the signed and the Q*_1 layout."""
    wl = synth.llama3_8b_decode()
    for name, spec in wl.layers.items():
        w = weights_host(spec)
        x = synth.activations(M, spec.cols, seed=wl.x_seed + M)
        for mode in (O.SIGNED_SYM, O.ASYM_MIN):
            check_matmul(w, x, 32, 4, mode, rows_idx=sample_rows(spec.rows, n=24, seed=M),
                         tag=f"8b {name} M={M}", workspace=True, repeat=2, need_split=False)


@pytest.mark.parametrize("M,workspace", [(1, False), (16, False), (16, True)])
def test_llama3_70b_matmul_full_size(M, workspace):
    """Every distinct 70B projection shape (q/o 8192x8192, k/v 1024x8192, gate/up
    28672x8192, down 8192x28672) at q=2 g=32, sampled rows."""
    wl = synth.llama3_70b_block()
    for name in ("q_proj", "k_proj", "gate_proj", "down_proj"):
        spec = wl.layers[name]
        w = synth.weights(spec)
        x = synth.activations(M, spec.cols, seed=wl.x_seed + M)
        check_matmul(w, x, 32, 2, O.SIGNED_SYM, rows_idx=sample_rows(spec.rows, n=24, seed=M),
                     tag=f"70b {name} M={M}", workspace=workspace, repeat=2 if workspace else 1, need_split=False)


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 128])
@pytest.mark.parametrize("mode", MODES)
def test_gemv_two_tokens_all_formats(q, group, mode):
    # M = 2 takes the two-token GEMV: 37 rows (ragged row groups), K = 19200 (two passes)
    w = rand_w(37, 19200, seed=q * 7 + group + mode)
    x = synth.activations(2, 19200, seed=q + group)
    check_matmul(w, x, group, q, mode, tag=f"gemv M=2 q={q} g={group} m={mode}")


@pytest.mark.parametrize("mode", MODES)
def test_gemv_two_tokens_full_size(mode):
    # 4096x14336 at M = 2: seven wavefronts each staging two tokens' activations plus
    # the scales and metadata (the largest LDS of the GEMV), sampled rows
    spec = synth.llama3_8b_decode().layers["down_proj"]
    w = weights_host(spec)
    x = synth.activations(2, spec.cols, seed=77)
    check_matmul(w, x, 32, 4, mode, rows_idx=sample_rows(spec.rows, 48, seed=mode), tag=f"gemv M=2 full m={mode}")
