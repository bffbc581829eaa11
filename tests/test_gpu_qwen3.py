"""GPU parity on the Qwen3-8B and Qwen3-14B projection shapes (Table 1 reports Qwen3
dense models): quantize bit for bit, the decode GEMV (M = 1), batched decode (M = 16,
split reduction) and the prefill GEMM (M = 512, split reduction), against the oracle on
sampled rows, element-wise (tests/parity_common.py).  Qwen3-14B's down projection has
K = 17408 = 544 blocks of 32, two passes of the GEMV's 512-thread team (the second one
ragged) at full size."""
import numpy as np
import pytest

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import sample_rows, weights_host
from tests.test_gpu_matmul import MODES, check_matmul
from tests.test_gpu_quantize import run_case

pytestmark = pytest.mark.gpu

WORKLOADS = {"qwen3_8b": synth.qwen3_8b_block, "qwen3_14b": synth.qwen3_14b_block}
SHAPES = ("q_proj", "k_proj", "gate_proj", "down_proj")     # every distinct shape of a block


@pytest.mark.parametrize("model", list(WORKLOADS))
def test_qwen3_quantize_full_size(model):
    wl = WORKLOADS[model]()
    for name in SHAPES:
        spec = wl.layers[name]
        w = weights_host(spec)
        idx = sample_rows(spec.rows, n=16, seed=spec.seed)
        for mode in MODES:
            run_case(w, True, 32, 4, mode, rows_idx=idx, tag=f"{model} {name}")
        for q in (2, 3):
            run_case(w, True, 32, q, O.SIGNED_SYM, rows_idx=idx, tag=f"{model} {name}")


@pytest.mark.parametrize("model", list(WORKLOADS))
@pytest.mark.parametrize("q", [2, 3, 4])
def test_qwen3_decode_gemv_full_size(model, q):
    wl = WORKLOADS[model]()
    for name in SHAPES:
        spec = wl.layers[name]
        w = weights_host(spec)
        x = synth.activations(1, spec.cols, seed=wl.x_seed)
        modes = MODES if q == 4 else [O.SIGNED_SYM]
        for mode in modes:
            check_matmul(w, x, 32, q, mode, rows_idx=sample_rows(spec.rows, n=24, seed=q),
                         tag=f"{model} {name} M=1 q={q} m={mode}")


@pytest.mark.parametrize("model", list(WORKLOADS))
def test_qwen3_batched_decode_full_size(model):
    wl = WORKLOADS[model]()
    for name in SHAPES:
        spec = wl.layers[name]
        w = weights_host(spec)
        x = synth.activations(16, spec.cols, seed=wl.x_seed + 16)
        for ws in (False, True):
            check_matmul(w, x, 32, 4, O.SIGNED_SYM, rows_idx=sample_rows(spec.rows, n=24, seed=16),
                         tag=f"{model} {name} M=16 ws={ws}", workspace=ws, need_split=False)


@pytest.mark.parametrize("model", list(WORKLOADS))
@pytest.mark.parametrize("name", ["gate_proj", "down_proj"])
def test_qwen3_prefill_full_size(model, name):
    wl = WORKLOADS[model]()
    spec = wl.layers[name]
    w = weights_host(spec)
    x = synth.activations(512, spec.cols, seed=wl.x_seed + 512)
    rows = sample_rows(spec.rows, n=32, seed=512)
    check_matmul(w, x, 32, 4, O.SIGNED_SYM, rows_idx=rows, tag=f"{model} {name} M=512")
    if ssq.ssq_matmul_workspace_size(512, spec.rows, spec.cols, 32, 4) > 0:
        check_matmul(w, x, 32, 4, O.SIGNED_SYM, rows_idx=rows, tag=f"{model} {name} M=512 split",
                     workspace=True)
