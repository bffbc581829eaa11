"""Pins for the CPU oracle: checks against what the paper and the mathematics fix.

Nothing here trusts the oracle's own arithmetic.  Each test recomputes the
property it checks independently (exact rationals, brute force over the
alphabet, a Python-integer bit stream, torch's library quantizer, the paper's
theorems), chosen so that a plausible slip in the oracle -- a wrong sign rule,
scale, rounding mode, clip range, tie-break, bit order, zero-point handling or
dequantization offset -- fails at least one of them.
"""
import json
import os
import struct
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

from oracle import ssq_oracle as O
from paper_2607_08779_amd import synth

SIGNED, UNSIGNED, ASYM, ASYM_MIN = O.SIGNED_SYM, O.UNSIGNED_SYM, O.ASYM, O.ASYM_MIN


# ---------------------------------------------------------------------------
# Independent helpers (exact rational arithmetic; no oracle code).
# ---------------------------------------------------------------------------

def rne(x: Fr) -> int:
    """Round a rational to the nearest integer, exact halves to even."""
    n = x.numerator // x.denominator
    d = x - n
    if d > Fr(1, 2):
        return n + 1
    if d < Fr(1, 2):
        return n
    return n if n % 2 == 0 else n + 1


def widen_bf16(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_groups(n, g, seed, outlier=True):
    rng = np.random.default_rng(seed)
    w = rng.standard_t(5, size=(n, g)) * 0.02
    if outlier:
        m = rng.random((n, g)) < 0.03
        w[m] *= 20 * np.where(rng.random(m.sum()) < 0.5, -1, 1)
    return widen_bf16(synth.to_bf16_bits(w.astype(np.float32)))


def f32_groups(n, g, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_t(4, size=(n, g)) * 0.02).astype(np.float32)


def near_half(t: Fr, eps=Fr(1, 2**20)) -> bool:
    """True if t is within eps of a half-integer but not exactly on it."""
    fl = t.numerator // t.denominator
    d = abs(t - (fl + Fr(1, 2)))
    return 0 < d < eps


def codes_of(res, q, mode):
    """Signed integer codes c (symmetric) or unsigned indices (asym) from the oracle result."""
    return res.u - (1 << (q - 1)) if mode != ASYM else res.u


# ---------------------------------------------------------------------------
# Closed-form worked examples and the paper's format sizes.
# ---------------------------------------------------------------------------

def test_worked_example_q2(golden_dir):
    gold = json.load(open(os.path.join(golden_dir, "worked_example_q2.json")))
    w = np.array([gold["w"]], np.float32)
    for name, mode in (("signed", SIGNED), ("unsigned", UNSIGNED), ("asym", ASYM)):
        r = O.quantize(w, gold["group"], gold["q"], mode)
        exp = gold[name]
        assert r.u[0].tolist() == exp["u"], name
        assert int(r.codes[0, 0]) == exp["byte"], name
        assert int(r.scales[0, 0]) == exp["scale_bits"], name
        if mode == ASYM:
            assert int(r.zp[0, 0]) == exp["zp"]
            continue
        s = Fr(float(r.scale32[0, 0]))
        c = codes_of(r, gold["q"], mode)[0]
        err2 = sum((Fr(float(wi)) - s * int(ci)) ** 2 for wi, ci in zip(w[0], c))
        assert abs(float(err2) - exp["err2"]) < 1e-6, name
    r = O.quantize(w, gold["group"], gold["q"], ASYM_MIN)
    exp = gold["asym_min"]
    assert r.u[0].tolist() == exp["u"] and int(r.codes[0, 0]) == exp["byte"]
    assert int(r.scales[0, 0]) == exp["scale_bits"] and int(r.mins[0, 0]) == exp["min_bits"]
    assert r.zp is None
    back = O.dequantize(r.codes, r.scales, None, 4, 4, 2, mins=r.mins)
    assert back[0].tolist() == exp["dequant"]


def test_rounding_is_half_to_even():
    # amax = 8 at a positive entry -> gamma = -1, alpha = 1, s = -1 (Eq. (5)); the
    # quotients -w hit exact halves.  Half-to-even gives [-8,-2,-4,2,0,0,-2,-8];
    # half-away-from-zero would give -3, 3, -1, 1 at positions 1, 3, 4, 5.
    w = np.array([[8.0, 2.5, 3.5, -2.5, 0.5, -0.5, 1.5, 7.5]], np.float32)
    r = O.quantize(w, 8, 4, SIGNED)
    assert (r.u[0] - 8).tolist() == [-8, -2, -4, 2, 0, 0, -2, -8]
    assert int(r.scales[0, 0]) == 0xBC00  # binary16(-1.0)


def test_block_sizes_match_paper(golden_dir):
    gold = json.load(open(os.path.join(golden_dir, "paper_block_sizes.json")))
    w = f32_groups(1, 32, 0)
    for q in (2, 4):
        for mode in (SIGNED, UNSIGNED):
            r = O.quantize(w, 32, q, mode)
            assert r.codes.nbytes + r.scales.nbytes == gold[f"Q{q}_0"]
        r = O.quantize(w, 32, q, ASYM)
        # our asymmetric form stores a u8 zero point instead of the fp16 minimum
        assert r.codes.nbytes + r.scales.nbytes + r.zp.nbytes == gold[f"Q{q}_1"] - 1
        r = O.quantize(w, 32, q, ASYM_MIN)   # the paper's Q*_1 layout: fp16 s + fp16 m
        assert r.codes.nbytes + r.scales.nbytes + r.mins.nbytes == gold[f"Q{q}_1"]


# ---------------------------------------------------------------------------
# Packing: compare with a bit stream built from Python integers.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("q", [2, 3, 4, 5, 8])
def test_pack_matches_little_endian_bitstream(q):
    rng = np.random.default_rng(q)
    cols = 64
    u = rng.integers(0, 1 << q, size=(3, cols))
    codes = O.pack(u, q)
    for row in range(3):
        acc = 0
        for k in range(cols):
            acc |= int(u[row, k]) << (k * q)
        assert bytes(codes[row]) == acc.to_bytes(cols * q // 8, "little")
    assert (O.unpack(codes, cols, q) == u).all()


def test_pack_explicit_q4_q2_bytes():
    u4 = np.array([[1, 2, 15, 0]])
    assert O.pack(u4, 4)[0].tolist() == [0x21, 0x0F]
    u2 = np.array([[1, 2, 3, 0, 0, 0, 0, 3]])
    assert O.pack(u2, 2)[0].tolist() == [0b00111001, 0b11000000]


# ---------------------------------------------------------------------------
# Brute force over the alphabet: Eq. (1) returns the nearest grid point.
# ---------------------------------------------------------------------------

def _check_nearest(w, q, mode, group, allow_near_half):
    r = O.quantize(w, group, q, mode)
    rows, cols = w.shape
    c = codes_of(r, q, mode)
    lo, hi = ((0, (1 << q) - 1) if mode == ASYM else (-(1 << (q - 1)), (1 << (q - 1)) - 1))
    checked = 0
    for n in range(rows):
        for b in range(cols // group):
            s = Fr(float(r.scale32[n, b]))
            z = int(r.zp[n, b]) if mode == ASYM else 0
            if s == 0:
                continue
            for k in range(b * group, (b + 1) * group):
                wk = Fr(float(w[n, k]))
                t = wk / s
                if not allow_near_half and near_half(t):
                    continue   # binary32 quotient may round onto/over the half (division reading)
                grid = [(abs(wk - s * (a - z)), a) for a in range(lo, hi + 1)]
                best = min(d for d, _ in grid)
                nearest = [a for d, a in grid if d == best]
                got = int(c[n, k])
                assert got in nearest, (n, k, float(wk), float(s), got, nearest)
                if len(nearest) == 2:   # exact tie between two grid points: even integer wins
                    assert (got - z) % 2 == 0, (n, k, float(wk), float(s), got, nearest)
                checked += 1
    assert checked > 0


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("mode", [SIGNED, UNSIGNED, ASYM])
def test_nearest_grid_point_bf16_inputs(q, mode):
    # bf16 weights: quotient of two 8-bit significands is never within 2^-10 of a
    # half unless exactly on it, so no element needs to be skipped (sym modes).
    w = bf16_groups(40, 32, seed=10 * q + mode).reshape(20, 64)
    _check_nearest(w, q, mode, 32, allow_near_half=(mode != ASYM))


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("mode", [SIGNED, UNSIGNED, ASYM])
def test_nearest_grid_point_f32_inputs(q, mode):
    w = f32_groups(16, 64, seed=100 + 10 * q + mode)
    _check_nearest(w, q, mode, 32, allow_near_half=False)


# ---------------------------------------------------------------------------
# Sign rule (Eq. (5)) and its structural properties (Sec. 4, after Remark 1).
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("q", [2, 3, 4])
def test_sign_rule_outlier_exact_and_clipping_confined(q):
    w = np.concatenate([bf16_groups(300, 32, seed=q), f32_groups(300, 32, seed=50 + q)])
    r = O.quantize(w, 32, q, SIGNED)
    c = codes_of(r, q, SIGNED)
    lo = -(1 << (q - 1))
    for n in range(w.shape[0]):
        g = [Fr(float(v)) for v in w[n]]
        M = max(abs(v) for v in g)
        pos, neg = M in g, -M in g
        s = Fr(float(r.scale32[n, 0]))
        gamma = 1 if s > 0 else -1
        # Eq. (5) with the tie-break reading: gamma = -1 iff the unique extreme is positive
        assert gamma == (-1 if (pos and not neg) else 1)
        assert abs(s) == M / 2 ** (q - 1)
        istar = next(i for i, v in enumerate(g) if abs(v) == M and (gamma == -1) == (v > 0))
        assert int(c[n, istar]) == lo                      # extra code on the outlier
        assert s * int(c[n, istar]) == g[istar]            # represented exactly
        T = M * (1 - Fr(1, 2 ** q))
        clipped = [i for i, v in enumerate(g) if gamma * v > T]    # Def. 1, Eq. (6)
        assert all(gamma * g[i] > 0 for i in clipped)      # clipping confined to the other tail


def test_tie_break_takes_positive_scale():
    w = np.array([[0.5, -0.5, 0.25, 0.125]], np.float32)
    r = O.quantize(w, 4, 2, SIGNED)
    assert r.scale32[0, 0] > 0
    assert (r.u[0] - 2).tolist() == [1, -2, 1, 0]


def test_unsigned_matches_signed_or_negates_it():
    q = 3
    w = bf16_groups(400, 32, seed=7)
    rs, ru = O.quantize(w, 32, q, SIGNED), O.quantize(w, 32, q, UNSIGNED)
    cs, cu = codes_of(rs, q, SIGNED), codes_of(ru, q, UNSIGNED)
    hi = (1 << (q - 1)) - 1
    assert (ru.scale32 > 0).all()
    for n in range(w.shape[0]):
        if rs.scale32[n, 0] > 0:
            assert (cs[n] == cu[n]).all()
        else:
            ok = (np.abs(cs[n]) < hi) & (np.abs(cu[n]) < hi)   # neither side clipped
            assert (cs[n][ok] == -cu[n][ok]).all()


# ---------------------------------------------------------------------------
# Lemma 1 (Eq. (7)) and Theorem 1 (Eq. (8)) in exact arithmetic.
# ---------------------------------------------------------------------------

def _q_gamma(w_row, q, gamma_wanted):
    """Q_gamma(w) for one group from the oracle: the signed/unsigned modes give
    gamma* and +1; Q_{-1}(w) = -Q_{+1}(-w) supplies the remaining sign."""
    w2 = w_row[None, :]
    rs = O.quantize(w2, w2.shape[1], q, SIGNED)
    if float(rs.scale32[0, 0]) == gamma_wanted * abs(float(rs.scale32[0, 0])):
        s, c = Fr(float(rs.scale32[0, 0])), codes_of(rs, q, SIGNED)[0]
        return [s * int(v) for v in c]
    if gamma_wanted == 1:
        ru = O.quantize(w2, w2.shape[1], q, UNSIGNED)
        s, c = Fr(float(ru.scale32[0, 0])), codes_of(ru, q, UNSIGNED)[0]
        return [s * int(v) for v in c]
    ru = O.quantize(-w2, w2.shape[1], q, UNSIGNED)
    s, c = Fr(float(ru.scale32[0, 0])), codes_of(ru, q, UNSIGNED)[0]
    return [-s * int(v) for v in c]


def _theory(g, q, gamma):
    M = max(abs(v) for v in g)
    alpha = M / 2 ** (q - 1)
    T = M * (1 - Fr(1, 2 ** q))
    C = [i for i, v in enumerate(g) if gamma * v > T]
    E = sum((v - alpha * rne(v / alpha)) ** 2 for v in g)
    return M, alpha, T, C, E


@pytest.mark.parametrize("q", [2, 3, 4])
def test_lemma1_and_theorem1_exact(q):
    groups = (list(bf16_groups(150, 32, seed=200 + q)) + list(f32_groups(150, 32, seed=300 + q))
              + list(bf16_groups(100, 16, seed=400 + q)))
    n_checked = 0
    for row in groups:
        g = [Fr(float(v)) for v in row]
        M = max(abs(v) for v in g)
        if M == 0:
            continue
        alpha = M / 2 ** (q - 1)
        if any(near_half(v / alpha) for v in g):
            continue       # binary32 quotient may round onto the half; the theorems assume exactness
        for gamma in (1, -1):
            Q = _q_gamma(row, q, gamma)
            M, alpha, T, C, E = _theory(g, q, gamma)
            err = [(v - qv) ** 2 for v, qv in zip(g, Q)]
            total = sum(err)
            # Lemma 1: ||w - Q_gamma(w)||^2 = E(w) + 2 alpha sum_{C_gamma} (gamma w_i - T)
            assert total == E + 2 * alpha * sum(gamma * g[i] - T for i in C)
            # Theorem 1: per-coordinate ranges and the total bound
            for i, e in enumerate(err):
                if i in C:
                    assert alpha ** 2 / 4 < e <= alpha ** 2
                else:
                    assert e <= alpha ** 2 / 4
            d = len(g)
            assert total <= Fr(1, 2 ** (2 * q)) * M * M * d * (1 + 3 * Fr(len(C), d))
            n_checked += 1
    assert n_checked > 500


def test_theorem1_bound_on_full_size_rows():
    """Theorem 1 never exceeded on 256 rows of the 4096x14336 down-projection workload."""
    spec = synth.llama3_8b_decode().layers["down_proj"]
    w = widen_bf16(synth.weights(spec, 0, 256))
    for q in (2, 3, 4):
        for mode in (SIGNED, UNSIGNED):
            r = O.quantize(w, 32, q, mode)
            c = codes_of(r, q, mode).reshape(256, -1, 32).astype(np.float64)
            s = r.scale32.astype(np.float64)[..., None]
            G = w.reshape(256, -1, 32).astype(np.float64)
            err = (G - s * c) ** 2                       # exact: w - s*c has < 53 bits
            M = np.abs(G).max(-1, keepdims=True)
            gamma = np.sign(s)
            T = M * (1 - 2.0 ** -q)
            inC = gamma * G > T
            a2 = (M / 2 ** (q - 1)) ** 2
            slack = 1 + 1e-12
            assert (err[~inC] <= (a2 / 4 * slack).repeat(32, -1)[~inC]).all()
            assert (err[inC] <= (a2 * slack).repeat(32, -1)[inC]).all()
            bound = 2.0 ** (-2 * q) * M[..., 0] ** 2 * 32 * (1 + 3 * inC.mean(-1))
            assert (err.sum(-1) <= bound * slack).all()


# ---------------------------------------------------------------------------
# Corollary 1 and Remark 1.
# ---------------------------------------------------------------------------

def test_corollary1_counterexample(golden_dir):
    gold = json.load(open(os.path.join(golden_dir, "corollary1_counterexample_q2.json")))
    q = gold["q"]
    row = np.array(gold["w"], np.float32)
    g = [Fr(float(v)) for v in row]
    rs = O.quantize(row[None, :], len(g), q, SIGNED)
    assert (1 if rs.scale32[0, 0] > 0 else -1) == gold["gamma_star"]
    e = {}
    for gamma in (gold["gamma_star"], -gold["gamma_star"]):
        Q = _q_gamma(row, q, gamma)
        e[gamma] = float(sum((v - qv) ** 2 for v, qv in zip(g, Q)))
        _, _, _, C, _ = _theory(g, q, gamma)
        assert C == gold["clipped_star" if gamma == gold["gamma_star"] else "clipped_other"]
    assert abs(e[gold["gamma_star"]] - gold["err2_star"]) < 1e-6
    assert abs(e[-gold["gamma_star"]] - gold["err2_other"]) < 1e-6
    # the cardinality condition holds and gamma* wins the bound, yet loses the realised error
    assert gold["bound_star"] <= gold["bound_other"]
    assert e[gold["gamma_star"]] > e[-gold["gamma_star"]]


@pytest.mark.parametrize("q", [2, 3, 4])
def test_small_clipped_set_implies_lower_error(q):
    """Lemma 1 plus Theorem 1's per-term range give: |C_{gamma*}| <= 1 implies the sign
    rule's realised error is no larger than the other sign's (the outlier sits in
    C_{-gamma*} with the largest possible term alpha/2)."""
    groups = np.concatenate([bf16_groups(400, 8, seed=500 + q), bf16_groups(200, 32, seed=600 + q)
                             .reshape(800, 8)])
    seen = 0
    for row in groups:
        g = [Fr(float(v)) for v in row]
        if max(abs(v) for v in g) == 0:
            continue
        rs = O.quantize(row[None, :], len(g), q, SIGNED)
        gs = 1 if rs.scale32[0, 0] > 0 else -1
        _, _, _, Cs, _ = _theory(g, q, gs)
        if len(Cs) > 1:
            continue
        es = sum((v - qv) ** 2 for v, qv in zip(g, _q_gamma(row, q, gs)))
        eo = sum((v - qv) ** 2 for v, qv in zip(g, _q_gamma(row, q, -gs)))
        assert es <= eo
        seen += 1
    assert seen > 100


# ---------------------------------------------------------------------------
# Theorem 2 against torch's library quantizer.
# ---------------------------------------------------------------------------

def _pow2_groups(n, g, seed):
    """Groups whose largest magnitude is a power of two, so alpha is a power of two and
    torch's multiply-by-reciprocal equals the division of Eq. (1) exactly."""
    w = bf16_groups(n, g, seed)
    rng = np.random.default_rng(seed)
    for row in w:
        i = int(np.argmax(np.abs(row)))
        e = np.floor(np.log2(abs(row[i]))) + 1
        row[i] = np.float32(np.sign(row[i]) * 2.0 ** e) * (1 if rng.random() < 0.9 else -1)
    return w


@pytest.mark.parametrize("q", [2, 3, 4])
def test_theorem2_and_absmax_against_torch_fake_quantize(q):
    w = _pow2_groups(600, 32, seed=700 + q)
    lo, hi = -(1 << (q - 1)), (1 << (q - 1)) - 1
    rs, ru = O.quantize(w, 32, q, SIGNED), O.quantize(w, 32, q, UNSIGNED)
    cs, cu = codes_of(rs, q, SIGNED), codes_of(ru, q, UNSIGNED)
    n_neg = 0
    for n, row in enumerate(w):
        alpha = float(abs(ru.scale32[n, 0]))
        t = torch.from_numpy(row.copy())
        # Eq. (3): the absmax grid is Eq. (1) with s = alpha, z = 0
        ref0 = torch.fake_quantize_per_tensor_affine(t, alpha, 0, lo, hi).numpy()
        assert (ru.scale32[n, 0] * cu[n].astype(np.float32) == ref0).all()
        if rs.scale32[n, 0] < 0:
            # Theorem 2: Q(w; -alpha, 0) = Q(w; alpha, -1).  With the zero point added after
            # rounding the identity holds at exact halves too.
            ref1 = torch.fake_quantize_per_tensor_affine(t, alpha, -1, lo, hi).numpy()
            assert (rs.scale32[n, 0] * cs[n].astype(np.float32) == ref1).all()
            # code level: the sign flip is the q-bit complement of the z=-1 index
            k = np.clip(np.rint(row / np.float32(alpha)) - 1, lo, hi).astype(np.int64)
            assert (rs.u[n] == (1 << q) - 1 - (k - lo)).all()
            n_neg += 1
    assert n_neg > 200


def test_theorem2_grid_identity():
    # -alpha*A_q == alpha*(A_q + 1) as sets (App. A, proof of Theorem 2)
    for q in range(2, 9):
        A = set(range(-(1 << (q - 1)), 1 << (q - 1)))
        assert {-a for a in A} == {a + 1 for a in A}


# ---------------------------------------------------------------------------
# Min-max asymmetric grid (Eq. (2)), degenerate groups, storage conversions.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("q", [2, 3, 4])
def test_asym_grid_properties(q):
    w = np.concatenate([bf16_groups(200, 32, seed=800 + q), f32_groups(200, 32, seed=900 + q),
                        np.abs(f32_groups(50, 32, seed=1)), -np.abs(f32_groups(50, 32, seed=2))])
    r = O.quantize(w, 32, q, ASYM)
    top = 2 ** q - 1
    for n, row in enumerate(w):
        s = Fr(float(r.scale32[n, 0]))
        z = int(r.zp[n, 0])
        # Eq. (2) on the range widened to contain 0 (the u8 zero-point reading)
        mx, mn = max(Fr(float(row.max())), Fr(0)), min(Fr(float(row.min())), Fr(0))
        exact_s = (mx - mn) / top
        assert abs(s - exact_s) <= exact_s * Fr(1, 2 ** 22)  # two binary32 roundings
        zr = -mn / s                                       # real zero point, in [0, 2^q-1]
        assert abs(z - zr) <= Fr(1, 2) + Fr(1, 2 ** 18)
        for k, v in enumerate(row):
            wv = Fr(float(v))
            e = abs(wv - s * (int(r.u[n, k]) - z))
            assert e <= s      # rounding error s/2, plus at most s/2 from the integer z
            if -z * s <= wv <= (top - z) * s:              # inside the grid: rounding only
                assert e <= s / 2 + s * Fr(1, 2 ** 20)


@pytest.mark.parametrize("q", [2, 3, 4])
def test_asym_min_grid_properties(q):
    """The fp16-minimum layout of Eq. (2): exact-rational checks of every code."""
    w = np.concatenate([bf16_groups(150, 32, seed=1800 + q), f32_groups(150, 32, seed=1900 + q),
                        np.abs(f32_groups(40, 32, seed=3)) + 0.5, -np.abs(f32_groups(40, 32, seed=4))])
    r = O.quantize(w, 32, q, ASYM_MIN)
    top = 2 ** q - 1
    n_checked = 0
    for n, row in enumerate(w):
        s = Fr(float(r.scale32[n, 0]))
        mn, mx = Fr(float(row.min())), Fr(float(row.max()))
        exact_s = (mx - mn) / top
        assert abs(s - exact_s) <= exact_s * Fr(1, 2 ** 22)       # two binary32 roundings
        mbits = struct.unpack("<H", struct.pack("<e", float(row.min())))[0]
        assert int(r.mins[n, 0]) == (0 if mbits & 0x7FFF == 0 else mbits)
        u = r.u[n]
        assert u[int(np.argmin(row))] == 0 and u[int(np.argmax(row))] == top
        for k, v in enumerate(row):
            wv = Fr(float(v))
            # Eq. (1) with the real zero point z = -min/s, in exact arithmetic
            t = wv / s + (-mn / s)
            if near_half(t, Fr(1, 2 ** 18)):
                continue      # binary32 rounding of w - min and of the quotient may decide
            assert int(u[k]) == min(max(rne(t), 0), top)
            # nearest point of the grid {s*v + min}: no clipping inside [min, max]
            assert abs(wv - (s * int(u[k]) + mn)) <= s / 2 + s * Fr(1, 2 ** 18)
            n_checked += 1
    assert n_checked > 10000


def test_asym_min_dequantize_reads_s_u_plus_m():
    """W_hat = s16 * u + m16 from the stored bit patterns (exact rationals)."""
    w = bf16_groups(20, 32, seed=77)
    r = O.quantize(w, 32, 4, ASYM_MIN)
    back = O.dequantize(r.codes, r.scales, None, 32, 32, 4, mins=r.mins)
    for n in range(20):
        s16 = Fr(float(struct.unpack("<e", struct.pack("<H", int(r.scales[n, 0])))[0]))
        m16 = Fr(float(struct.unpack("<e", struct.pack("<H", int(r.mins[n, 0])))[0]))
        for k in range(32):
            assert Fr(float(back[n, k])) == s16 * int(r.u[n, k]) + m16
    # and the matmul is that dequantized matrix times x, in binary64
    x = np.random.default_rng(5).standard_normal((3, 32))
    y = O.matmul(x, r.codes, r.scales, None, 20, 32, 32, 4, mins=r.mins)
    assert np.allclose(y, x @ back.T, rtol=1e-12, atol=0)


def test_degenerate_groups():
    q = 4
    w = np.zeros((3, 32), np.float32)
    w[1] = -0.0
    w[2] = 0.375
    for mode in (SIGNED, UNSIGNED):
        r = O.quantize(w, 32, q, mode)
        assert (r.scales[:2] == 0).all() and (r.u[:2] == 8).all()
    r = O.quantize(w, 32, q, SIGNED)       # constant positive group: gamma = -1, code -8
    assert (r.u[2] == 0).all() and r.scale32[2, 0] == np.float32(-0.375 / 8)
    r = O.quantize(w, 32, q, ASYM)
    assert (r.scales[:2] == 0).all() and (r.zp[:2] == 0).all() and (r.u[:2] == 0).all()
    # constant positive group: range [0, 0.375], z = 0, every index 2^q-1, exact up to s rounding
    assert int(r.zp[2, 0]) == 0 and (r.u[2] == 15).all()
    r = O.quantize(w, 32, q, ASYM_MIN)     # constant groups: s = 0, codes 0, m = the constant
    assert (r.scales == 0).all() and (r.u == 0).all()
    assert [int(b) for b in r.mins[:, 0]] == [0x0000, 0x0000, 0x3600]   # +0, -0 stored as +0, 0.375


def test_scale_storage_matches_python_binary16():
    w = f32_groups(64, 32, seed=3)
    for mode in (SIGNED, UNSIGNED, ASYM, ASYM_MIN):
        r = O.quantize(w, 32, 4, mode)
        for s32, bits in zip(r.scale32.ravel(), r.scales.ravel()):
            assert struct.unpack("<H", struct.pack("<e", float(s32)))[0] == int(bits)


def test_bf16_widening_matches_torch():
    bits = np.random.default_rng(0).integers(0, 1 << 16, size=5000, dtype=np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]                      # finite values only
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    assert (O.bf16_bits_to_f32(bits).view(np.uint32) == ref.view(np.uint32)).all()


# ---------------------------------------------------------------------------
# Matmul (App. B.3) by exact brute force with its own bit-stream decoding.
# ---------------------------------------------------------------------------

def _decode_row(codes_row, K, q):
    acc = int.from_bytes(bytes(codes_row), "little")
    return [(acc >> (k * q)) & ((1 << q) - 1) for k in range(K)]


@pytest.mark.parametrize("mode", [SIGNED, UNSIGNED, ASYM])
@pytest.mark.parametrize("q", [2, 3, 4])
def test_matmul_exact_bruteforce(mode, q):
    N, K, g, M = 5, 128, 32, 3
    w = bf16_groups(N * K // 32, 32, seed=31 * q + mode).reshape(N, K)
    x = widen_bf16(synth.activations(M, K, seed=q))
    r = O.quantize(w, g, q, mode)
    y = O.matmul(x, r.codes, r.scales, r.zp, N, K, g, q)
    for n in range(N):
        u = _decode_row(r.codes[n], K, q)
        for m in range(M):
            dot_u = Fr(0)          # integer-GEMM part of App. B.3
            corr = Fr(0)           # row-sum correction part
            for b in range(K // g):
                s = Fr(struct.unpack("<e", struct.pack("<H", int(r.scales[n, b])))[0])
                o = int(r.zp[n, b]) if mode == ASYM else 1 << (q - 1)
                xs = [Fr(float(v)) for v in x[m, b * g:(b + 1) * g]]
                dot_u += s * sum(xv * uv for xv, uv in zip(xs, u[b * g:(b + 1) * g]))
                corr += s * o * sum(xs)
            exact = dot_u - corr
            assert abs(y[m, n] - float(exact)) <= 1e-12 * max(1.0, abs(float(exact)))


def test_matmul_unit_vectors_read_back_dequantized_weights():
    N, K, g, q = 3, 64, 32, 4
    w = bf16_groups(6, 32, seed=9).reshape(N, K)
    r = O.quantize(w, g, q, SIGNED)
    y = O.matmul(np.eye(K, dtype=np.float32), r.codes, r.scales, None, N, K, g, q)
    # bf16 weights: the binary16 scale is exact, so the dequantized outlier equals w
    for n in range(N):
        for b in range(K // g):
            i = b * g + int(np.argmax(np.abs(w[n, b * g:(b + 1) * g])))
            assert y[i, n] == float(w[n, i])


# ---------------------------------------------------------------------------
# Sec. 4 diagnostics: clipped sets (Def. 1), margin and realised gain (Remark 1).
# ---------------------------------------------------------------------------

def test_diagnostics_worked_examples(golden_dir):
    gold = json.load(open(os.path.join(golden_dir, "worked_example_q2.json")))
    d = O.sign_diagnostics(np.array([gold["w"]], np.float32), gold["group"], gold["q"])
    # gamma* = -1: C_{-1} = {}, C_{+1} = {0}; g = E + 2 alpha (w_0 - T) - E = 0.25
    assert int(d.margin[0, 0]) == 1 and float(d.gain[0, 0]) == 0.25
    assert d.tally[2, 2] == 1 and d.tally.sum() == 1
    cx = json.load(open(os.path.join(golden_dir, "corollary1_counterexample_q2.json")))
    w = np.array([cx["w"]], np.float32)
    d = O.sign_diagnostics(w, w.shape[1], cx["q"])
    assert int(d.margin[0, 0]) == len(cx["clipped_other"]) - len(cx["clipped_star"]) == 1
    assert abs(float(d.gain[0, 0]) - (cx["err2_other"] - cx["err2_star"])) < 1e-6   # -0.21 < 0
    assert d.tally[2, 0] == 1


def _rational_grid(v, scale, lo, hi):
    """Def. 1 and Eq. (1) in exact arithmetic: (rounded index, clipped?, Q(v))."""
    r = rne(v / scale)
    return r, not lo <= r <= hi, scale * min(max(r, lo), hi)


@pytest.mark.parametrize("q", [2, 3, 4])
def test_diagnostics_match_brute_force(q):
    """Margin and gain against both signed grids quantized in exact rationals, with the
    clipped set taken from Def. 1's rounding form, not from the threshold T."""
    rows = np.concatenate([bf16_groups(120, 32, seed=2100 + q), f32_groups(120, 32, seed=2200 + q),
                           bf16_groups(60, 16, seed=2300 + q)[:, :16].repeat(2, axis=1)])
    d = O.sign_diagnostics(rows, 32, q)
    lo, hi = -(1 << (q - 1)), (1 << (q - 1)) - 1
    n_checked = 0
    for n, row in enumerate(rows):
        g = [Fr(float(v)) for v in row]
        M = max(abs(v) for v in g)
        if M == 0:
            assert int(d.margin[n, 0]) == 0 and float(d.gain[n, 0]) == 0.0
            continue
        alpha = M / 2 ** (q - 1)
        if any(near_half(v / alpha, Fr(1, 2 ** 20)) or (v / alpha).denominator == 2 for v in g):
            continue     # Def. 1 assumes no quotient on a half-integer
        pos_max = max(g) == M and -min(g) != M      # dominant outlier positive and unmatched
        gamma_star = -1 if pos_max else 1
        size, err = {}, {}
        for gamma in (1, -1):
            res = [_rational_grid(v, gamma * alpha, lo, hi) for v in g]
            size[gamma] = sum(1 for _, clipped, _ in res if clipped)
            err[gamma] = sum((v - qv) ** 2 for v, (_, _, qv) in zip(g, res))
        m = size[-gamma_star] - size[gamma_star]
        gain = err[-gamma_star] - err[gamma_star]
        assert int(d.margin[n, 0]) == m
        got = Fr(float(d.gain[n, 0]))
        assert (got > 0) == (gain > 0) and (got < 0) == (gain < 0)
        assert abs(got - gain) <= abs(gain) * Fr(1, 2 ** 22)
        n_checked += 1
    assert n_checked > 200


def test_diagnostics_tally_counts_groups():
    w = np.concatenate([bf16_groups(400, 32, seed=31), f32_groups(100, 32, seed=32),
                        np.zeros((4, 32), np.float32)])
    for q in (2, 3, 4):
        d = O.sign_diagnostics(w, 32, q)
        assert d.tally.sum() == w.shape[0]
        for sm in (-1, 0, 1):
            for sg in (-1, 0, 1):
                n = int(((np.sign(d.margin) == sm) & (np.sign(d.gain) == sg)).sum())
                assert d.tally[sm + 1, sg + 1] == n
        assert d.tally[1, 1] >= 4     # all-zero groups: no clipping either way


# ---------------------------------------------------------------------------
# Q8_0 activations and the integer-dot matmul (App. C, App. B.3).
# ---------------------------------------------------------------------------

def fl(r: Fr, p: int, emin: int) -> Fr:
    """Round a rational to the binary format with p significant bits and minimum
    normal exponent emin (gradual underflow), half to even; no overflow handling."""
    if r == 0:
        return Fr(0)
    a = abs(r)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if a < Fr(2) ** e:
        e -= 1
    if a >= Fr(2) ** (e + 1):
        e += 1
    ulp = Fr(2) ** (max(e, emin) - p + 1)
    v = rne(a / ulp) * ulp
    return v if r > 0 else -v


def f16_bits_of(r: Fr) -> int:
    """binary16 bits of a value that is already representable (through Python's struct)."""
    return struct.unpack("<H", struct.pack("<e", float(r)))[0]


def test_q8_worked_example(golden_dir):
    gold = json.load(open(os.path.join(golden_dir, "q8_worked_example.json")))
    x = np.array([gold["x"]], np.float32)
    assert np.array_equal(widen_bf16(synth.to_bf16_bits(x)), x)       # bf16 values
    a = O.quantize_act_q8(x)
    assert a.q.tolist() == [gold["q"]]
    assert a.d.tolist() == [gold["d_f16_bits"]]


def test_q8_activations_match_exact_rationals():
    """Every code and scale against exact rational arithmetic: d = fl32(amax/127),
    t = fl32(x/d), q = clip(rne(t)), stored binary16(d)."""
    rng = np.random.default_rng(77)
    x = rng.standard_t(3, size=(6, 256)) * 0.3
    x[rng.random(x.shape) < 0.02] *= 40
    x[0, :32] = np.arange(32) - 16.0                     # quotients near halves
    x[1, 32:64] = 0.0                                    # zero block
    x[2, 64:96] *= 1e-38                                 # tiny: subnormal d, binary16 scale 0
    x = widen_bf16(synth.to_bf16_bits(x.astype(np.float32)))
    a = O.quantize_act_q8(x)
    for m in range(x.shape[0]):
        for b in range(x.shape[1] // 32):
            blk = [Fr(float(v)) for v in x[m, 32 * b:32 * b + 32]]
            amax = max(abs(v) for v in blk)
            d = fl(amax / 127, 24, -126)
            assert a.d[m, b] == (f16_bits_of(fl(d, 11, -14)) if amax else 0)
            for j, v in enumerate(blk):
                want = 0 if amax == 0 else max(-127, min(127, rne(fl(v / d, 24, -126))))
                assert a.q[m, 32 * b + j] == want, (m, b, j)


@pytest.mark.parametrize("q", [2, 3, 4])
@pytest.mark.parametrize("mode", [SIGNED, ASYM, ASYM_MIN])
def test_matmul_q8_matches_exact_rationals(q, mode):
    """y = sum_k (d q_x)[m, k] * W_hat[n, k] with every product and sum exact, against
    the oracle's integer split (App. B.3) evaluated in binary64."""
    rng = np.random.default_rng(100 * q + mode)
    M, N, K, group = 2, 5, 128, 64
    w = f32_groups(N, K, seed=q + 7 * mode)
    r = O.quantize(w, group, q, mode)
    x = widen_bf16(synth.to_bf16_bits((rng.standard_normal((M, K)) * 0.5).astype(np.float32)))
    a = O.quantize_act_q8(x)
    y = O.matmul_q8(a.q, a.d, r.codes, r.scales, r.zp, N, K, group, q, mins=r.mins)
    u = O.unpack(r.codes, K, q)
    s = [[Fr(float(v)) for v in row] for row in O.f16_bits_to_f64(r.scales)]
    mins = O.f16_bits_to_f64(r.mins) if mode == ASYM_MIN else None
    for m in range(M):
        dx = [Fr(float(v)) for v in O.f16_bits_to_f64(a.d[m])]
        for n in range(N):
            exact = Fr(0)
            for k in range(K):
                g = k // group
                if mode == ASYM_MIN:
                    wk = s[n][g] * int(u[n, k]) + Fr(float(mins[n, g]))
                else:
                    o = int(r.zp[n, g]) if mode == ASYM else 1 << (q - 1)
                    wk = s[n][g] * (int(u[n, k]) - o)
                exact += dx[k // 32] * int(a.q[m, k]) * wk
            assert abs(Fr(float(y[m, n])) - exact) <= abs(exact) * Fr(1, 2**50) + Fr(1, 2**80)


def test_matmul_q8_equals_matmul_on_dequantized_activations():
    """The integer split and the weight-only matmul of the dequantized activations
    (d q exact in binary64) are the same sum."""
    rng = np.random.default_rng(5)
    w = bf16_groups(40, 512, seed=6)
    x = widen_bf16(synth.to_bf16_bits((rng.standard_t(4, size=(3, 512)) * 0.2).astype(np.float32)))
    a = O.quantize_act_q8(x)
    xh = (a.q.reshape(3, 16, 32) * O.f16_bits_to_f64(a.d)[..., None]).reshape(3, 512)
    for mode in (SIGNED, UNSIGNED, ASYM, ASYM_MIN):
        r = O.quantize(w, 32, 4, mode)
        y = O.matmul_q8(a.q, a.d, r.codes, r.scales, r.zp, 40, 512, 32, 4, mins=r.mins)
        ref = O.matmul(xh, r.codes, r.scales, r.zp, 40, 512, 32, 4, mins=r.mins)
        assert np.allclose(y, ref, rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------------------
# App. B.1 formats table: GGUF array-of-structures blocks.
# ---------------------------------------------------------------------------

def test_gguf_blocks_match_hand_derived_bytes(golden_dir):
    """Three blocks whose bytes were derived by hand from the formats table (fixture),
    including a negative (signed-symmetric) scale; sizes as the table."""
    gold = json.load(open(os.path.join(golden_dir, "gguf_blocks.json")))
    sizes = json.load(open(os.path.join(golden_dir, "paper_block_sizes.json")))
    for c in gold["cases"]:
        u = np.array([c["u"]])
        s = np.array([[int(c["s_f16"], 16)]], np.uint16)
        m = np.array([[int(c["m_f16"], 16)]], np.uint16) if c["with_min"] else None
        b = O.to_gguf(u, s, m, 32, c["q"])
        assert b.shape == (1, 1, O.gguf_block_bytes(c["q"], c["with_min"]))
        assert b.shape[-1] == sizes[f"Q{c['q']}_{1 if c['with_min'] else 0}"]
        assert b[0, 0].tobytes().hex() == c["hex"], c["format"]
        u2, s2, m2 = O.from_gguf(b, c["q"], c["with_min"])
        assert np.array_equal(u2, u) and np.array_equal(s2, s)
        np.testing.assert_array_equal(O.gguf_dequantize(b, c["q"], c["with_min"])[0, :4], c["weights_first4"])


@pytest.mark.parametrize("q", [2, 4])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("mode", [SIGNED, UNSIGNED, ASYM_MIN])
def test_gguf_round_trip_reads_back_the_same_weights(q, group, mode):
    """Blocks decoded byte by byte give the weights the packed bit stream gives (two
    independent decodings: App. B.1 blocks against App. B.3's dequantization)."""
    w = f32_groups(13, 256, q * 100 + group + mode)
    r = O.quantize(w, group, q, mode)
    b = O.to_gguf(r.u, r.scales, r.mins, group, q)
    assert b.shape == (13, 256 // 32, O.gguf_block_bytes(q, r.mins is not None))
    expect = O.dequantize(r.codes, r.scales, r.zp, 256, group, q, r.mins)
    got = O.gguf_dequantize(b, q, r.mins is not None)
    assert np.array_equal(got, expect)
    u, s, m = O.from_gguf(b, q, r.mins is not None)
    assert np.array_equal(u, O.unpack(r.codes, 256, q))
