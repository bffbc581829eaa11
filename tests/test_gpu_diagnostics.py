"""GPU parity: ssq_sign_diagnostics against the CPU oracle (Sec. 4 Def. 1, Lemma 1,
Remark 1).  Margins, gains (binary32 values) and the tally must be identical:
both sides form the gain from exact binary64 sums with one final rounding."""
import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import ssq, synth
from tests.parity_common import Guarded, sample_rows, to_device, widen

pytestmark = pytest.mark.gpu


def tally_of(margin: np.ndarray, gain: np.ndarray) -> np.ndarray:
    """3x3 counts of groups by (sign of the margin, sign of the gain), -1/0/+1 -> 0/1/2."""
    counts = np.zeros((3, 3), np.int64)
    np.add.at(counts, (np.sign(margin).astype(np.int64).ravel() + 1,
                       np.sign(gain).astype(np.int64).ravel() + 1), 1)
    return counts


def check(w_host, bf16, group, q, rows_idx=None, tag=""):
    """Diagnostics into guarded buffers; margins and gains against the oracle (on rows_idx),
    the tally against the oracle's (whole matrix) or against counts of the GPU's own
    margins and gains (sampled rows).  Returns the tally."""
    W = to_device(w_host, bf16)
    rows, cols = w_host.shape
    g_margin = Guarded((rows, cols // group), torch.int16, fill=0x5A)
    g_gain = Guarded((rows, cols // group), torch.float32)
    g_tally = Guarded((9,), torch.int64, fill=0x5A)
    margin, gain, tally = ssq.ssq_sign_diagnostics(W, group, q, out=(g_margin.t, g_gain.t, g_tally.t))
    torch.cuda.synchronize()
    for b, name in ((g_margin, "margin"), (g_gain, "gain"), (g_tally, "tally")):
        b.check(f"{tag} {name}")
    m_all, g_all = margin.cpu().numpy(), gain.cpu().numpy()
    assert not np.isnan(g_all).any(), f"{tag}: gains left unwritten"
    assert np.array_equal(tally.cpu().numpy(), tally_of(m_all, g_all)), f"{tag}: tally vs outputs"
    sel = slice(None) if rows_idx is None else rows_idx
    with np.errstate(over="ignore"):                     # a gain past binary32 rounds to inf
        ref = O.sign_diagnostics(widen(w_host[sel], bf16), group, q)
    m = margin.cpu().numpy()[sel]
    g = gain.cpu().numpy()[sel]
    assert np.array_equal(m, ref.margin), f"{tag}: margins differ"
    # Identical binary32 values; a zero gain is exact and the sign of that zero is an
    # artifact of which maximum the two sides pick for M when +0 meets -0.
    if not np.array_equal(g, ref.gain):
        r, b = np.argwhere(g != ref.gain)[0]
        raise AssertionError(f"{tag}: gains differ at ({r}, {b}): gpu {g[r, b]!r} oracle {ref.gain[r, b]!r}")
    if rows_idx is None:
        assert np.array_equal(tally.cpu().numpy(), ref.tally), f"{tag}: tallies differ"
    return tally.cpu().numpy()


def random_bf16(rows, cols, seed, outliers=0.001):
    return synth.weights(synth.WeightSpec(rows, cols, nu=5.0, scale=0.02, outlier_frac=outliers, seed=seed))


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
def test_diagnostics_bf16_all_formats(q, group):
    check(random_bf16(45, 1536, seed=q * 100 + group, outliers=0.01), True, group, q, tag=f"bf16 q={q} g={group}")


@pytest.mark.parametrize("q", [2, 3, 4])
def test_diagnostics_fp32(q):
    rng = np.random.default_rng(q)
    w = (rng.standard_t(4, size=(33, 1024)) * 0.02).astype(np.float32)
    check(w, False, 32, q, tag=f"f32 q={q}")


def test_diagnostics_edge_groups():
    rng = np.random.default_rng(9)
    rows = [np.zeros(64, np.float32), -np.zeros(64, np.float32)]
    t = rng.standard_normal(64).astype(np.float32) * 0.1
    t[::32] = 1.0; t[1::32] = -1.0                       # +M / -M ties
    rows.append(t)
    c = np.zeros(64, np.float32); c[:8] = [1.0, 0.76, 0.76, -0.99, -0.99, 0, 0, 0]   # Corollary 1 counterexample
    rows.append(c)
    rows.append(np.full(64, 0.375, np.float32))          # constant groups: everything clipped one way
    rows.append((rng.standard_normal(64) * 1e-39).astype(np.float32))   # bf16 subnormals
    rows.append((rng.standard_normal(64) * 1e17).astype(np.float32))
    rows.append((rng.standard_normal(64) * 1e35).astype(np.float32))   # gains overflow to inf
    w = synth.to_bf16_bits(np.stack(rows))
    for q in (2, 3, 4):
        check(w, True, 32, q, tag=f"edge q={q}")


def packed_edge_rows(rng):
    """512-weight rows (one wavefront's span in both kernels) of groups that stress the
    bf16 integer statistics: weights exactly at each T = M (1 - 2^-q) and one ulp above,
    +M/-M ties, constant groups, huge values, maxima at the smallest exponents the
    integer path takes, a wave whose groups mix a tiny maximum (the binary32 path) with
    ordinary ones, signed zeros, one-sided groups."""
    rows = []
    r = rng.standard_normal(512) * 0.05
    for k, q in enumerate((2, 3, 4)):
        T = 1.0 - 2.0 ** -q
        for j, v in enumerate((T, T + 2 ** -8, -T, -(T + 2 ** -8))):
            g0 = 32 * (4 * k + j)
            r[g0] = 1.0 if j % 2 == 0 else -1.0
            r[g0 + 1: g0 + 6] = v
    rows.append(r)
    t = rng.standard_normal(512) * 0.1
    t[::32] = 1.0; t[1::32] = -1.0; t[2::64] = -1.0
    rows.append(t)
    c = np.full(512, 0.375); c[256:] = -0.8125
    rows.append(c)
    rows.append(rng.standard_normal(512) * 1e35)
    e2 = rng.uniform(-1.9, 1.9, 512) * 2.0 ** -125        # maxima with biased exponent 2
    e2[::32] = 1.5 * 2.0 ** -125
    rows.append(e2)
    mixed = rng.standard_normal(512) * 0.02
    mixed[128:256] = rng.choice([-1.0, 1.0], 128) * rng.uniform(1, 1.99, 128) * 2.0 ** -126   # exponent 1
    rows.append(mixed)
    z = rng.standard_normal(512) * 0.02
    z[0:32] = -0.0; z[0] = 0.5                          # -0 beside a positive maximum
    z[32:64] = -np.abs(z[32:64])                       # all negative
    z[64:96] = 0.0; z[70] = -0.25                      # a single nonzero
    z[96:128] = np.abs(z[96:128])                      # all positive
    rows.append(z)
    cx = np.zeros(512); cx[::32] = 1.0; cx[1::32] = 0.76; cx[2::32] = 0.76; cx[3::32] = -0.99; cx[4::32] = -0.99
    cx[5::32] = 0.01
    rows.append(cx)
    return synth.to_bf16_bits(np.stack(rows).astype(np.float32))


@pytest.mark.parametrize("group", [32, 64, 128])
def test_diagnostics_bf16_packed_edges(group):
    w = packed_edge_rows(np.random.default_rng(group))
    for q in (2, 3, 4):
        check(w, True, group, q, tag=f"packed edges g={group} q={q}")
        codes, scales, margin, gain = ssq.ssq_quantize_diag(to_device(w, True), group, q)
        torch.cuda.synchronize()
        with np.errstate(over="ignore"):
            d = O.sign_diagnostics(widen(w, True), group, q)
        assert np.array_equal(margin.cpu().numpy(), d.margin), f"fused g={group} q={q}: margins"
        assert np.array_equal(gain.cpu().numpy(), d.gain), f"fused g={group} q={q}: gains"


def test_diagnostics_llama3_8b_down_proj_full_size():
    """4096x14336 at q in {2,3,4}: sampled rows bit for bit; tally consistent with the
    full per-group outputs (the GPU tally counts what the GPU stored)."""
    spec = synth.llama3_8b_decode().layers["down_proj"]
    w = synth.weights(spec)
    rows = sample_rows(spec.rows, 64, seed=3)
    for q in (2, 3, 4):
        tally = check(w, True, 32, q, rows_idx=rows, tag=f"down_proj q={q}")   # tally == counts of outputs
        assert tally.sum() == spec.rows * spec.cols // 32


def test_diagnostics_tally_across_calls():
    """The blocks' counts and the arrival counter are reused from call to call: a full
    grid, a call without a tally, then a small grid must each give the oracle's tally."""
    big = random_bf16(2048, 4096, seed=11)               # 2^20 chunks: every block of the grid
    small = random_bf16(6, 256, seed=12)                 # a single block
    for w, tag in ((big, "big"), (small, "small"), (big, "big again")):
        W = to_device(w, True)
        ssq.ssq_sign_diagnostics(W, 32, 2, tally=False)
        _, _, tally = ssq.ssq_sign_diagnostics(W, 32, 2)
        torch.cuda.synchronize()
        ref = O.sign_diagnostics(widen(w, True), 32, 2)
        assert np.array_equal(tally.cpu().numpy(), ref.tally), tag


def test_diagnostics_empty():
    W = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    margin, gain, tally = ssq.ssq_sign_diagnostics(W, 32, 4)
    torch.cuda.synchronize()
    assert margin.shape == (0, 2) and gain.shape == (0, 2)
    assert tally.cpu().numpy().sum() == 0


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("bf16", [True, False])
def test_quantize_diag_matches_both_oracles(q, group, bf16):
    """The fused kernel: codes and scales of the signed grid and the sign-rule margin and
    gain, each against its own oracle."""
    rng = np.random.default_rng(q * 10 + group + bf16)
    w = rng.standard_t(4, size=(23, 1024)) * 0.02
    w[rng.random(w.shape) < 0.01] *= 20
    w_host = synth.to_bf16_bits(w.astype(np.float32)) if bf16 else w.astype(np.float32)
    codes, scales, margin, gain = ssq.ssq_quantize_diag(to_device(w_host, bf16), group, q)
    torch.cuda.synchronize()
    wf = widen(w_host, bf16)
    r = O.quantize(wf, group, q, O.SIGNED_SYM)
    d = O.sign_diagnostics(wf, group, q)
    assert np.array_equal(codes.cpu().numpy(), r.codes)
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), r.scales)
    assert np.array_equal(margin.cpu().numpy(), d.margin)
    assert np.array_equal(gain.cpu().numpy(), d.gain)


def test_quantize_diag_full_size_sampled():
    spec = synth.llama3_8b_decode().layers["down_proj"]
    w = synth.weights(spec)
    codes, scales, margin, gain = ssq.ssq_quantize_diag(to_device(w, True), 32, 4)
    m2, g2, _ = ssq.ssq_sign_diagnostics(to_device(w, True), 32, 4, tally=False)
    torch.cuda.synchronize()
    assert torch.equal(margin, m2) and torch.equal(gain.view(torch.int32), g2.view(torch.int32))
    rows = sample_rows(spec.rows, 32, seed=9)
    r = O.quantize(widen(w[rows], True), 32, 4, O.SIGNED_SYM)
    assert np.array_equal(codes.cpu().numpy()[rows], r.codes)
