"""CPU model of the packed 16-bit integer form of the sign-rule statistics that the
bf16 diagnostics kernels use (Sec. 4 Def. 1, Lemma 1, Remark 1), checked against the
oracle bit for bit.  The model follows the kernel's formulation step by step on bf16
bit patterns: the group's largest magnitude per sign from the raw patterns; the unit
u = 2^(em - 135); v = |w|/u from the significand and a saturating exponent
difference; membership and excess from a saturating subtract of floor(T/u); the two
fields (both sets, negative set times 2^15) of the packed accumulators; the exact
excess sum d - |C| frac(T/u); one binary64 product.  It pins the derivation itself
(every field bound and identity it relies on is asserted here), independently of
the GPU, on groups that stress thresholds, ties, constants, signed zeros and the
smallest exponents the integer form accepts."""
import numpy as np
import pytest

from oracle import ssq_oracle as O
from paper_2607_08779_amd import synth


def packed_model(bits, group, q):
    rows, cols = bits.shape
    b = bits.reshape(rows, cols // group, group).astype(np.int64)
    sign = b >> 15
    mag = b & 0x7FFF
    P = np.where(sign == 0, mag, 0).max(-1)                 # signed 16-bit max, clamped at 0
    N = np.where(sign == 1, mag, 0).max(-1)                 # unsigned max minus the sign bit
    gamma_neg = P > N
    mb = np.maximum(P, N)
    em = mb >> 7
    ok = em >= 2                                            # else the binary32 form runs
    mm = 0x80 | (mb & 0x7F)
    tq = (mm << q) - mm                                     # (T/u) 2^(q-1)
    tfl = tq >> (q - 1)
    tfrac = tq - (tfl << (q - 1))
    p = np.clip((mag >> 7) - (em - 2)[..., None], 0, None)   # saturating exponent difference
    assert (p[ok] <= 2).all()
    v = ((b & 0x7F) | 0x80) * p
    assert (v < 1 << 16).all()
    d = np.clip(v - tfl[..., None], 0, None)                # excess over floor(T/u), members only
    assert (d[ok] <= 128).all()
    k = 1 + (sign << 15)                                    # per-half multiplier of v_dot2_u32_u16
    e_acc = (d * k).sum(-1)
    c_acc = (np.minimum(d, 1) * k).sum(-1)
    assert ((e_acc & 0x7FFF) == d.sum(-1)).all() and (e_acc < 1 << 32).all()   # fields do not overlap
    dc = 2 * (c_acc >> 15) - (c_acc & 0x7FFF)
    de = 2 * (e_acc >> 15) - (e_acc & 0x7FFF)
    sgn = np.where(gamma_neg, -1, 1)
    margin = sgn * dc
    excess = sgn * ((de << (q - 1)) - dc * tfrac)
    M = (mb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    with np.errstate(over="ignore"):
        gain = (M * (4.0 / (1 << q)) * np.ldexp(excess.astype(np.float64), em - 135 - (q - 1))).astype(np.float32)
    return margin.astype(np.int16), gain, ok


def groups(seed, group):
    rng = np.random.default_rng(seed)
    rows = [rng.standard_t(5, size=4 * group) * 0.02,
            rng.standard_normal(4 * group) * 10.0 ** rng.integers(-30, 30),
            rng.integers(-8, 9, size=4 * group) * 0.25,                     # ties at +-M and at T
            np.round(rng.standard_normal(4 * group) * 64) / 64,
            rng.uniform(-1.9, 1.9, 4 * group) * 2.0 ** -125,                # maxima with em = 2
            np.full(4 * group, -0.8125)]
    t = rng.standard_normal(4 * group) * 0.05
    for j, q in enumerate((2, 3, 4)):
        T = 1.0 - 2.0 ** -q
        t[group * (j % 4)] = 1.0
        t[group * (j % 4) + 1: group * (j % 4) + 5] = [T, T + 2 ** -8, -T, -(T + 2 ** -8)]
    rows.append(t)
    z = rng.standard_normal(4 * group) * 0.02
    z[:group] = -0.0
    z[0] = 0.5
    rows.append(z)
    return synth.to_bf16_bits(np.stack(rows).astype(np.float32))


@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("q", [2, 3, 4])
def test_packed_model_matches_oracle(q, group):
    for seed in range(4):
        bits = groups(seed * 7 + q, group)
        with np.errstate(over="ignore"):
            ref = O.sign_diagnostics(O.bf16_bits_to_f32(bits), group, q)
        m, g, ok = packed_model(bits, group, q)
        assert ok.mean() > 0.9
        assert np.array_equal(m[ok], ref.margin[ok])
        assert np.array_equal(g[ok].view(np.uint32), ref.gain[ok].view(np.uint32))
