"""GPU parity: ssq_export_gguf writes the GGUF blocks of App. B.1's formats table byte for
byte as the oracle's to_gguf (on weights quantized on the GPU, which matches the oracle's
codes bit for bit), for Q4_0/Q4_0s, Q4_1, Q2_0/Q2_0s and Q2_1, every group size, ragged row
counts, with guard bytes around the output."""
import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import Guarded, sample_rows, to_device, weights_host

pytestmark = pytest.mark.gpu


def export_and_compare(w_bits, group, q, mode, rows_idx=None, tag=""):
    N, K = w_bits.shape
    codes, scales, meta = ssq.ssq_quantize(to_device(w_bits, True), group, q, mode)
    mins = meta if mode == O.ASYM_MIN else None
    nbytes = O.gguf_block_bytes(q, mins is not None)
    g = Guarded((N, K // 32, nbytes), torch.uint8, fill=0x5A)
    ssq.ssq_export_gguf(codes, scales, mins, N, K, group, q, out=g.t)
    g.check(f"{tag} blocks")
    sel = np.arange(N) if rows_idx is None else rows_idx
    r = O.quantize(O.bf16_bits_to_f32(w_bits[sel]), group, q, mode)
    ref = O.to_gguf(r.u, r.scales, r.mins, group, q)
    got = g.t.cpu().numpy()[sel]
    if not np.array_equal(got, ref):
        n, b, k = np.argwhere(got != ref)[0]
        raise AssertionError(f"{tag}: row {sel[n]} block {b} byte {k}: gpu {got[n, b, k]:#04x} oracle {ref[n, b, k]:#04x}")


@pytest.mark.parametrize("q", [2, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", [O.SIGNED_SYM, O.UNSIGNED_SYM, O.ASYM_MIN])
def test_export_gguf_all_formats(q, group, mode):
    w = synth.weights(synth.WeightSpec(37, 1024, nu=5.0, scale=0.02, outlier_frac=0.001, seed=q + group + mode))
    export_and_compare(w, group, q, mode, tag=f"export q={q} g={group} m={mode}")


def test_export_gguf_llama3_8b_down_proj_full_size():
    """4096x14336 at W4 g32 signed (Q4_0s): 1,835,008 blocks, sampled rows against the oracle."""
    spec = synth.llama3_8b_decode().layers["down_proj"]
    w = weights_host(spec)
    export_and_compare(w, 32, 4, O.SIGNED_SYM, rows_idx=sample_rows(spec.rows, 32, seed=3), tag="export down_proj")


def test_export_gguf_rejects_three_bits_and_zero_points():
    w = synth.weights(synth.WeightSpec(4, 64, nu=5.0, scale=0.02, seed=1))
    codes, scales, _ = ssq.ssq_quantize(to_device(w, True), 32, 3, O.SIGNED_SYM)
    with pytest.raises(ssq.SSQError):
        ssq.ssq_export_gguf(codes, scales, None, 4, 64, 32, 3)
    codes, scales, zp = ssq.ssq_quantize(to_device(w, True), 32, 4, O.ASYM)
    with pytest.raises(TypeError):
        ssq.ssq_export_gguf(codes, scales, zp, 4, 64, 32, 4)
