"""GPU parity: the activation-stationary decode GEMV (M = 1).

ssq_matmul takes it for long rows with many 4-row groups: more than two groups per
resident workgroup (rows of up to 32768 weights, one wavefront per 2048).  Each
workgroup walks a run of 4 or 8 groups with the next group's codes in flight; the
cases below take both run lengths, a ragged last wavefront (K not a multiple of 2048),
a ragged last run and ragged last group (N not a multiple of 4 or of the run), every
q, group size and layout.  Sampled rows include the first and last rows of several
runs and the last three rows.  Bounds as in tests/test_gpu_matmul.py (element-wise,
guarded outputs)."""
import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import Guarded, sample_rows, to_device, weights_host
from tests.test_gpu_matmul import MODES, check_matmul

pytestmark = pytest.mark.gpu


def spec(N, K, seed):
    return synth.WeightSpec(N, K, nu=5.0, scale=0.02, outlier_frac=0.001, seed=seed)


def run_rows(N, run_rows_, seed):
    """Sampled rows plus both ends of the first, second and last runs and the last rows."""
    pick = set(sample_rows(N, n=24, seed=seed).tolist())
    for start in (0, run_rows_, (N - 1) // run_rows_ * run_rows_):
        pick |= {start, start + 1, start + run_rows_ - 1}
    pick |= {N - 3, N - 2, N - 1}
    return np.array(sorted(r for r in pick if 0 <= r < N))


# K = 32640 = 1020 blocks: 16 wavefronts, the last with 60 live lanes; N = 2051 rows =
# 513 groups, runs of 4 groups (16 rows), the last run one group of 3 rows.
@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", MODES)
def test_gemv_stream_all_formats(q, group, mode):
    N, K = 2051, 32640
    w = weights_host(spec(N, K, seed=9100))
    x = synth.activations(1, K, seed=9101)
    check_matmul(w, x, group, q, mode, rows_idx=run_rows(N, 16, seed=q * 7 + group + mode),
                 tag=f"gemv stream {N}x{K} q={q} g={group} m={mode}")


# K = 32736 = 1023 blocks (16 wavefronts, the last with 63 live lanes); N = 4101 rows =
# 1026 groups, runs of 8 groups (32 rows), the last run two groups, the last of 1 row.
@pytest.mark.parametrize("mode", MODES)
def test_gemv_stream_runs_of_eight(mode):
    N, K = 4101, 32736
    w = weights_host(spec(N, K, seed=9200))
    x = synth.activations(1, K, seed=9201)
    for q in (4, 2):
        check_matmul(w, x, 32, q, mode, rows_idx=run_rows(N, 32, seed=q + mode),
                     tag=f"gemv stream {N}x{K} q={q} m={mode}")


def test_gemv_stream_repeatable():
    """Two launches on the same operands agree bit for bit, and with the result of a
    HIP graph replay, replayed several times with eager work between replays."""
    N, K = 8192, 28672
    w = weights_host(synth.llama3_70b_block().layers["down_proj"])
    codes, scales, zp = ssq.ssq_quantize(to_device(w, True), 32, 4, O.SIGNED_SYM)
    X = to_device(synth.activations(1, K, seed=9301), True)
    y0 = ssq.ssq_matmul(X, codes, scales, zp, N, K, 32, 4)
    y1 = ssq.ssq_matmul(X, codes, scales, zp, N, K, 32, 4)
    torch.cuda.synchronize()
    assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
    yg = Guarded((1, N), torch.bfloat16)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ssq.ssq_matmul(X, codes, scales, zp, N, K, 32, 4, out=yg.t)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            ssq.ssq_matmul(X, codes, scales, zp, N, K, 32, 4, out=yg.t)
    torch.cuda.synchronize()
    for r in range(3):
        yg.t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        yg.check(f"graph replay {r}")
        assert torch.equal(yg.t.view(torch.int16), y0.view(torch.int16)), f"graph replay {r} differs"
