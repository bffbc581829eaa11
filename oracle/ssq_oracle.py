"""CPU oracle for group-wise signed symmetric quantization and its dequantizing matmul.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import this
module.  It shares no code with the HIP library (``paper_2607_08779_amd``) and
imports nothing from it: every function here takes plain numpy arrays.

The oracle is written to be read against the paper (Colbert, Dash et al.,
"Signed Symmetric Quantization for Few-Bit Integers"):

* Sec. 1, Eq. (1): the standard integer quantizer
  Q(w) = s * (clip(round(w/s + z); A_q) - z).
* Sec. 3, Eq. (2): the min-max asymmetric grid on the unsigned alphabet.
* Sec. 3, Eq. (3): the absmax ("unsigned symmetric") grid, s = ||w||_inf / 2^(q-1) > 0.
* Sec. 3, Eq. (4)-(5): the signed symmetric family s = gamma*alpha and the sign
  rule gamma* = -sign(w_{i*}), i* = argmax |w_i|.
* App. B.1 (formats table): one fp16 scale per 32-weight block, packed few-bit
  indices, no zero point for the symmetric formats.
* App. B.3 (zero-point cost): Y_ik = sum_b s_kb sum_{j in b} X_ij (Wq_kj - z_kb).
* App. B.1 (Q4_1 / Q2_1 rows of the formats table): the min-max grid stored as an
  fp16 scale s and an fp16 minimum m per block, so that a weight reads back as
  s*u + m (the real zero point z = -min/s of Eq. (2) folded into m = -s*z).
* Sec. 5.2 and App. C (dynamic Q8_0 activations, narrow range A = {-127, ..., 127})
  with App. B.3's integer GEMM term and row-sum correction: ``quantize_act_q8`` and
  ``matmul_q8``.

Arithmetic precision.  The paper fixes no precision for the grid computation;
this oracle computes the scale and the quotient w/s in IEEE binary32 (each
operation correctly rounded, round-half-to-even everywhere), stores the scale
as IEEE binary16 (round-half-to-even) and evaluates the matmul in binary64.
The readings taken where the paper is silent are listed in ``READINGS`` and
each is cited at the line that implements it.

Parity status: every public function here is pinned by tests/test_oracle_pins.py
against closed forms, the paper's theorems (Lemma 1, Theorem 1, Corollary 1,
Theorem 2), brute force over the alphabet and a library quantizer
(``torch.fake_quantize_per_tensor_affine``).  No function is "parity unpinned".
"""
from __future__ import annotations

from typing import NamedTuple, Optional

import numpy as np

SIGNED_SYM = 0      # signed absmax grid, Eq. (5)
UNSIGNED_SYM = 1    # absmax grid with s > 0, Eq. (3)
ASYM = 2            # min-max grid with an integer zero point, Eq. (2)
ASYM_MIN = 3        # min-max grid with an fp16 minimum, Eq. (2) in the App. B.1 Q*_1 layout

MODE_NAMES = {SIGNED_SYM: "signed_sym", UNSIGNED_SYM: "unsigned_sym", ASYM: "asym",
              ASYM_MIN: "asym_min"}

READINGS = {
    "tie_break": "Eq. (5) breaks ties in argmax|w_i| by an unnamed fixed rule; when both +M and -M "
                 "occur the oracle takes gamma=+1 (gamma=-1 only if max(w) > -min(w) strictly).",
    "rounding": "The round-to-nearest operator of Eq. (1) resolves exact halves to even.",
    "division": "t = w/s is one IEEE binary32 division, correctly rounded, then rounded to an integer.",
    "scale_storage": "Codes are computed from the binary32 scale; the stored scale is its binary16 "
                     "rounding (half to even).",
    "amax_zero": "Sec. 4 assumes M > 0; for an all-zero group the oracle stores scale +0 and code 0.",
    "asym_zero_point": "Eq. (2) gives a real z = -min/s; with an unsigned integer zero point the "
                       "range is first widened to contain 0 (min' = min(min w, 0), max' = "
                       "max(max w, 0)), so z = rne(fl32(-min'/s)) lies in [0, 2^q-1] and the grid "
                       "still covers the data.  Codes are clip(rne(fl32(w/s)) + z, 0, 2^q-1), the "
                       "zero point being added after rounding; an all-zero group stores zeros.",
    "asym_min": "For the fp16-minimum layout (App. B.1, Q4_1/Q2_1) the grid is Eq. (2) on the "
                "group's own range (no widening): s = fl32(fl32(max - min)/(2^q-1)), and Eq. (1) "
                "with the real zero point z = -min/s is evaluated as u = clip(rne(fl32(fl32(w - "
                "min)/s)), 0, 2^q-1), which equals round(w/s + z) in exact arithmetic.  The "
                "stored minimum is binary16(min) (half to even; a minimum that is or rounds to "
                "a zero is stored as +0, since -0 and +0 compare equal and either may be the "
                "group's min); a weight reads back "
                "as s*u + m with the stored binary16 s and m.  A constant group (max == min) "
                "stores s = 0, codes 0 and m = binary16(min).",
    "index_encoding": "Symmetric codes c in A_q are stored as the offset-binary index u = c + 2^(q-1).",
    "q8_activations": "Dynamic Q8_0 (per token, blocks of 32, the narrow-range alphabet "
                      "{-127..127}): d = fl32(amax/127), codes clip(rne(fl32(x/d)), -127, 127) from "
                      "the binary32 d, stored scale binary16(d) (half to even; it may underflow to "
                      "0 or overflow to inf, as the format does); an all-zero block stores d = +0 "
                      "and codes 0.  Input activations are bf16.",
    "q8_matmul": "App. B.3 with Q8_0 activations: per 32-activation block b inside weight group "
                 "g, I = sum_j q_j u_j and R = sum_j q_j are exact integers; y = sum_b d_b s_g "
                 "(I - o_g R) (symmetric offset or zero point o) or sum_b d_b (s_g I + m_g R) "
                 "(fp16 minimum), each block term exact in binary64 and the sum over blocks in "
                 "binary64.",
    "bit_order": "Field k of a row occupies bits [k*q, k*q+q) of the row's little-endian bit stream.",
    "gguf_order": "App. B.1's formats table fixes the GGUF block fields and sizes (binary16 s, for "
                  "Q*_1 a binary16 m, then qs; 18/20 bytes at q=4, 10/12 at q=2), not the index "
                  "order inside qs.  Q4 follows the 4-bit unpack the paper names (one shift and "
                  "one mask give indices 0..15 and 16..31): byte j = u[j] | u[j+16] << 4.  Q2 "
                  "follows the described 2-bit unpack (four shift-and extractions, then byte and "
                  "word interleaves restore element order): byte i = u[4i] | u[4i+1] << 2 | "
                  "u[4i+2] << 4 | u[4i+3] << 6.  Binary16 fields are little-endian.  With a "
                  "group of 64 or 128 each 32-weight block repeats its group's s (and m).",
}


class Quantized(NamedTuple):
    """Result of :func:`quantize` (all arrays row-major)."""

    codes: np.ndarray                 # uint8 [rows, cols*q/8], packed indices
    scales: np.ndarray                # uint16 [rows, cols/group], binary16 bit patterns
    zp: Optional[np.ndarray]          # uint8 [rows, cols/group] for ASYM, else None
    scale32: np.ndarray               # float32 [rows, cols/group], the scale the codes used
    u: np.ndarray                     # int64 [rows, cols], unpacked indices
    mins: Optional[np.ndarray] = None  # uint16 [rows, cols/group] binary16 minimums for ASYM_MIN


# ---------------------------------------------------------------------------
# Exact conversions between storage formats and binary32/binary64.
# ---------------------------------------------------------------------------

def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to binary32 exactly (bf16 is the top half of binary32)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def f16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round binary32 values to binary16 (IEEE, half to even) and return the bit patterns."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def f16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of binary16 bit patterns as binary64."""
    return np.ascontiguousarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


# ---------------------------------------------------------------------------
# Eq. (1): the standard integer quantizer, evaluated in binary32.
# ---------------------------------------------------------------------------

def eq1_codes(w: np.ndarray, s: np.ndarray, z: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """Integer part of Eq. (1): clip(round(w/s) + z; [lo, hi]) for an integer zero point z.

    w/s is one correctly rounded binary32 division, rounding is half-to-even
    (numpy.rint) and, because z is an integer, round(w/s + z) = round(w/s) + z.
    Returns the clipped integers as float32 (exact).
    """
    w = np.asarray(w, dtype=np.float32)
    s = np.asarray(s, dtype=np.float32)
    t = w / s                                       # binary32, correctly rounded
    r = np.rint(t) + np.asarray(z, dtype=np.float32)
    return np.clip(r, np.float32(lo), np.float32(hi))


def signed_alphabet(q: int) -> tuple[int, int]:
    """A_q = {-2^(q-1), ..., 2^(q-1)-1} (Sec. 1 notation; Sec. 3, Eq. (3))."""
    return -(1 << (q - 1)), (1 << (q - 1)) - 1


def unsigned_alphabet(q: int) -> tuple[int, int]:
    """A_q = {0, ..., 2^q - 1}, the alphabet of the min-max grid (Sec. 3, Eq. (2))."""
    return 0, (1 << q) - 1


# ---------------------------------------------------------------------------
# Group-wise grids: Eq. (2), Eq. (3), Eq. (4)-(5).
# ---------------------------------------------------------------------------

def _check_shape(W: np.ndarray, group: int, q: int) -> None:
    if W.ndim != 2:
        raise ValueError("W must be 2-D [rows, cols]")
    if group < 1 or W.shape[1] % group:
        raise ValueError("cols must be a multiple of group")
    if not 2 <= q <= 8:
        raise ValueError("q must be in [2, 8]")
    if (W.shape[1] * q) % 8:
        raise ValueError("cols*q must be a multiple of 8 (whole bytes per row)")


def quantize(W: np.ndarray, group: int, q: int, mode: int) -> Quantized:
    """Quantize each group of ``group`` consecutive entries of every row of W.

    W is binary32 [rows, cols] (bf16 inputs are widened exactly first).  Groups run
    along the reduction index, as in App. B.3.
    """
    W = np.ascontiguousarray(W, dtype=np.float32)
    _check_shape(W, group, q)
    rows, cols = W.shape
    G = W.reshape(rows, cols // group, group)
    mx = G.max(axis=-1)                             # max_j w_j
    mn = G.min(axis=-1)                             # min_j w_j

    if mode in (SIGNED_SYM, UNSIGNED_SYM):
        lo, hi = signed_alphabet(q)
        amax = np.maximum(mx, -mn)                  # M = ||w||_inf  (Eq. (3), Eq. (5))
        if mode == SIGNED_SYM:
            # Eq. (5): gamma* = -sign(w_{i*}).  A unique positive extreme gives gamma=-1,
            # a unique negative extreme gives gamma=+1; a tie +M/-M takes gamma=+1.
            gamma = np.where(mx > -mn, np.float32(-1), np.float32(1))
        else:
            gamma = np.ones_like(amax)              # Eq. (3): s > 0 by convention
        alpha = np.ldexp(amax, -(q - 1)).astype(np.float32)     # alpha = M / 2^(q-1), exact
        s32 = (gamma * alpha).astype(np.float32)                # Eq. (4): s = gamma*alpha
        zero = amax == 0
        safe_s = np.where(zero, np.float32(1), s32)
        c = eq1_codes(G, safe_s[..., None], np.float32(0), lo, hi)   # Eq. (1) with z = 0
        c = np.where(zero[..., None], np.float32(0), c)
        s32 = np.where(zero, np.float32(0), s32)    # M = 0: scale +0, every code 0
        u = (c.astype(np.int64) - lo).reshape(rows, cols)   # offset-binary index
        zp = None
    elif mode == ASYM:
        lo, hi = unsigned_alphabet(q)
        mx0 = np.maximum(mx, np.float32(0))                     # range widened to contain 0 so the
        mn0 = np.minimum(mn, np.float32(0))                     # integer zero point fits A_q
        rng32 = (mx0 - mn0).astype(np.float32)                  # fl32(max' - min')
        s32 = (rng32 / np.float32(hi)).astype(np.float32)       # Eq. (2): s = (max-min)/(2^q-1)
        flat = s32 == 0                                         # all-zero group
        safe_s = np.where(flat, np.float32(1), s32)
        z = np.clip(np.rint(-mn0 / safe_s), np.float32(lo), np.float32(hi))  # Eq. (2): z = -min/s
        c = eq1_codes(G, safe_s[..., None], z[..., None], lo, hi)    # clip(round(w/s) + z)
        c = np.where(flat[..., None], np.float32(0), c)
        z = np.where(flat, np.float32(0), z)
        u = c.astype(np.int64).reshape(rows, cols)
        zp = z.astype(np.uint8)
    elif mode == ASYM_MIN:
        lo, hi = unsigned_alphabet(q)
        rng32 = (mx - mn).astype(np.float32)                    # fl32(max - min)
        s32 = (rng32 / np.float32(hi)).astype(np.float32)       # Eq. (2): s = (max-min)/(2^q-1)
        flat = s32 == 0                                         # constant group
        safe_s = np.where(flat, np.float32(1), s32)
        d = (G - mn[..., None]).astype(np.float32)              # fl32(w - min) >= 0
        t = (d / safe_s[..., None]).astype(np.float32)          # fl32((w - min)/s)
        c = np.clip(np.rint(t), np.float32(lo), np.float32(hi))  # Eq. (1): round(w/s + z), z = -min/s
        c = np.where(flat[..., None], np.float32(0), c)
        s32 = np.where(flat, np.float32(0), s32)
        u = c.astype(np.int64).reshape(rows, cols)
        m_bits = f16_bits_from_f32(mn)
        m_bits = np.where((m_bits & 0x7FFF) == 0, np.uint16(0), m_bits)   # a zero minimum: +0
        return Quantized(codes=pack(u, q), scales=f16_bits_from_f32(s32), zp=None,
                         scale32=s32.astype(np.float32), u=u, mins=m_bits.astype(np.uint16))
    else:
        raise ValueError(f"unknown mode {mode}")

    return Quantized(codes=pack(u, q), scales=f16_bits_from_f32(s32), zp=zp,
                     scale32=s32.astype(np.float32), u=u)


# ---------------------------------------------------------------------------
# Sec. 4: clipped sets, cardinality margin and realised gain (Def. 1, Lemma 1,
# Corollary 1, Remark 1).
# ---------------------------------------------------------------------------

class Diagnostics(NamedTuple):
    """Result of :func:`sign_diagnostics` (per group, row-major)."""

    margin: np.ndarray     # int16 [rows, cols/group]: m(w) = |C_{-g*}| - |C_{g*}|
    gain: np.ndarray       # float32 [rows, cols/group]: g(w) = Delta_{-g*} - Delta_{g*}
    tally: np.ndarray      # int64 [3, 3]: groups by (sign m, sign g), index sign + 1


def sign_diagnostics(W: np.ndarray, group: int, q: int) -> Diagnostics:
    """Remark 1's two statistics for every group of the signed absmax grid.

    gamma* is the sign rule of Eq. (5) (with the tie-break reading), alpha = M/2^(q-1)
    and T = M (1 - 2^-q).  Def. 1 (Eq. (6)): C_gamma = {i : gamma w_i > T}.  The margin
    is m(w) = |C_{-gamma*}| - |C_{gamma*}|; by Lemma 1 (Eq. (7)) the realised gain
    g(w) = ||w - Q_{-gamma*}(w)||^2 - ||w - Q_{gamma*}(w)||^2 equals
    2 alpha (sum_{C_{-gamma*}} (-gamma* w_i - T) - sum_{C_{gamma*}} (gamma* w_i - T)).
    Everything is evaluated in binary64, where every term and partial sum is exact for
    binary32 weights; only the final product 2 alpha * (...) rounds (to binary64), and
    the stored gain is its binary32 rounding.  The tally counts groups by the signs of
    the stored margin and gain (index sign + 1 along each axis).
    """
    W = np.ascontiguousarray(W, dtype=np.float32)
    if W.ndim != 2 or group < 1 or W.shape[1] % group:
        raise ValueError("W must be [rows, cols] with cols a multiple of group")
    rows, cols = W.shape
    G = W.reshape(rows, cols // group, group).astype(np.float64)
    mx, mn = G.max(axis=-1), G.min(axis=-1)
    M = np.maximum(mx, -mn)                                      # ||w||_inf
    gamma = np.where(mx > -mn, -1.0, 1.0)                        # Eq. (5), tie -> +1
    T = M * (1.0 - 2.0 ** -q)                                    # exact in binary64
    alpha2 = M * 2.0 ** (2 - q)                                  # 2 alpha = 2 M / 2^(q-1)
    size, excess = {}, {}
    for g in (1.0, -1.0):
        inC = g * G > T[..., None]                               # Def. 1, Eq. (6)
        size[g] = inC.sum(axis=-1)
        excess[g] = np.where(inC, g * G - T[..., None], 0.0).sum(axis=-1)   # exact sums
    star = gamma == 1.0
    c_star = np.where(star, size[1.0], size[-1.0])
    c_other = np.where(star, size[-1.0], size[1.0])
    e_star = np.where(star, excess[1.0], excess[-1.0])
    e_other = np.where(star, excess[-1.0], excess[1.0])
    margin = (c_other - c_star).astype(np.int16)
    gain = (alpha2 * (e_other - e_star)).astype(np.float32)      # Lemma 1
    tally = np.zeros((3, 3), np.int64)
    np.add.at(tally, (np.sign(margin).astype(np.int64) + 1, np.sign(gain).astype(np.int64) + 1), 1)
    return Diagnostics(margin=margin, gain=gain, tally=tally)


# ---------------------------------------------------------------------------
# App. B.1: packing q-bit indices, several per byte.
# ---------------------------------------------------------------------------

def pack(u: np.ndarray, q: int) -> np.ndarray:
    """Pack indices u in [0, 2^q) into a little-endian bit stream per row.

    Field k of a row occupies stream bits [k*q, k*q+q); stream bit b is bit b%8
    of byte b//8.  For q=4 this is byte j = u[2j] | u[2j+1] << 4; for q=2 four
    fields share a byte; for q=3 fields straddle bytes.
    """
    u = np.asarray(u, dtype=np.int64)
    rows, cols = u.shape
    if (cols * q) % 8:
        raise ValueError("cols*q must be a multiple of 8")
    if u.size and (u.min() < 0 or u.max() >= (1 << q)):
        raise ValueError("index out of range")
    bits = ((u[..., None] >> np.arange(q)) & 1).astype(np.uint8)     # [rows, cols, q], LSB first
    return np.packbits(bits.reshape(rows, cols * q), axis=1, bitorder="little")


def unpack(codes: np.ndarray, cols: int, q: int) -> np.ndarray:
    """Inverse of :func:`pack`: int64 indices [rows, cols]."""
    codes = np.asarray(codes, dtype=np.uint8)
    rows = codes.shape[0]
    bits = np.unpackbits(codes, axis=1, bitorder="little")[:, : cols * q]
    bits = bits.reshape(rows, cols, q).astype(np.int64)
    return (bits << np.arange(q)).sum(axis=-1)


# ---------------------------------------------------------------------------
# Dequantization and the weight-only matmul (App. B.3).
# ---------------------------------------------------------------------------

def dequantize(codes: np.ndarray, scales: np.ndarray, zp: Optional[np.ndarray],
               cols: int, group: int, q: int, mins: Optional[np.ndarray] = None) -> np.ndarray:
    """W_hat[n, k] = s[n, b] * (u[n, k] - o[n, b]) in binary64, b = k // group.

    o = 2^(q-1) for the symmetric formats (the index offset) and o = zp for the
    asymmetric one, i.e. Eq. (1) read back with the stored binary16 scale.  With
    ``mins`` (the App. B.1 Q*_1 layout) W_hat = s*u + m instead.
    """
    u = unpack(codes, cols, q).astype(np.float64)
    rows = u.shape[0]
    s = f16_bits_to_f64(scales).reshape(rows, cols // group, 1)
    ug = u.reshape(rows, cols // group, group)
    if mins is not None:
        m = f16_bits_to_f64(mins).reshape(rows, cols // group, 1)
        return (s * ug + m).reshape(rows, cols)
    if zp is None:
        o = np.float64(1 << (q - 1))
    else:
        o = np.asarray(zp, dtype=np.float64).reshape(rows, cols // group, 1)
    return (s * (ug - o)).reshape(rows, cols)


def matmul(x: np.ndarray, codes: np.ndarray, scales: np.ndarray, zp: Optional[np.ndarray],
           N: int, K: int, group: int, q: int, mins: Optional[np.ndarray] = None) -> np.ndarray:
    """y[m, n] = sum_k x[m, k] * W_hat[n, k], evaluated in binary64 (App. B.3)."""
    x64 = np.asarray(x, dtype=np.float64).reshape(-1, K)
    W_hat = dequantize(codes, scales, zp, K, group, q, mins)
    if W_hat.shape[0] != N:
        raise ValueError("codes do not have N rows")
    return x64 @ W_hat.T


# ---------------------------------------------------------------------------
# Q8_0 activations and the integer-dot matmul (Sec. 5.2, App. C; App. B.3).
# ---------------------------------------------------------------------------

Q8_BLOCK = 32       # activations per Q8_0 block (the GGUF block the weight groups align to)
Q8_MAX = 127        # narrow range: K = 2^(8-1) - 1


class QuantizedAct(NamedTuple):
    q: np.ndarray       # int8 [M, K]: codes in {-127, ..., 127}
    d: np.ndarray       # uint16 [M, K/32]: binary16 bits of the block scales


def quantize_act_q8(x: np.ndarray) -> QuantizedAct:
    """Dynamic Q8_0 quantization of activations x [M, K] (bf16 values as binary32).

    Per token and block of 32 the narrow-range symmetric grid of App. C: with
    amax = max |x_j|, d = amax / 127 and q_j = clip(round(x_j / d), -127, 127), i.e.
    Eq. (1) with z = 0 on A = {-127, ..., 127}.  Readings ``q8_activations``: binary32
    d and quotient, half to even, stored scale binary16(d); an all-zero block stores
    d = +0 and codes 0.
    """
    X = np.ascontiguousarray(x, dtype=np.float32)
    if X.ndim != 2 or X.shape[1] % Q8_BLOCK:
        raise ValueError("x must be [M, K] with K a multiple of 32")
    M, K = X.shape
    B = X.reshape(M, K // Q8_BLOCK, Q8_BLOCK)
    amax = np.abs(B).max(axis=-1)                                   # exact
    d32 = (amax / np.float32(Q8_MAX)).astype(np.float32)            # one binary32 division
    zero = amax == 0
    safe = np.where(zero, np.float32(1), d32)
    t = (B / safe[..., None]).astype(np.float32)                    # binary32 quotients
    qv = np.clip(np.rint(t), -Q8_MAX, Q8_MAX)                       # half to even
    qv = np.where(zero[..., None], 0.0, qv)
    d16 = f16_bits_from_f32(np.where(zero, np.float32(0), d32))
    return QuantizedAct(q=qv.astype(np.int8).reshape(M, K), d=d16)


def matmul_q8(qx: np.ndarray, dx: np.ndarray, codes: np.ndarray, scales: np.ndarray,
              zp: Optional[np.ndarray], N: int, K: int, group: int, q: int,
              mins: Optional[np.ndarray] = None) -> np.ndarray:
    """y[m, n] for Q8_0 activations (codes qx [M, K], scales dx [M, K/32]) and packed
    weights, App. B.3 split into the integer GEMM term and the row-sum correction.

    For 32-activation block b of weight group g = b // (group/32):
      I[m, n, b] = sum_{j in b} qx[m, j] u[n, j]   (integer GEMM term)
      R[m, b]    = sum_{j in b} qx[m, j]           (row-sum of the activations)
      y[m, n]    = sum_b d[m, b] s[n, g] (I - o[n, g] R)    symmetric (o = 2^(q-1)) or zero point
      y[m, n]    = sum_b d[m, b] (s[n, g] I + m[n, g] R)    fp16-minimum layout
    The integers are exact, every block term is exact in binary64 (11-bit scales times
    integers below 2^21) and the block sum is evaluated in binary64.
    """
    Q = np.asarray(qx, dtype=np.int64).reshape(-1, K)
    M = Q.shape[0]
    nb = K // Q8_BLOCK
    per = group // Q8_BLOCK                                          # 32-blocks per weight group
    u = unpack(codes, K, q).astype(np.int64)
    if u.shape[0] != N:
        raise ValueError("codes do not have N rows")
    Qb = Q.reshape(M, nb, Q8_BLOCK)
    I = np.einsum("mbj,nbj->mnb", Qb, u.reshape(N, nb, Q8_BLOCK))    # int64, exact
    R = Qb.sum(axis=-1)                                              # [M, nb]
    d = f16_bits_to_f64(dx).reshape(M, nb)
    s = np.repeat(f16_bits_to_f64(scales).reshape(N, K // group), per, axis=1)   # [N, nb]
    if mins is not None:
        m = np.repeat(f16_bits_to_f64(mins).reshape(N, K // group), per, axis=1)
        term = s[None] * I + m[None] * R[:, None, :]
    else:
        o = (np.full((N, nb), 1 << (q - 1), np.int64) if zp is None
             else np.repeat(np.asarray(zp, np.int64).reshape(N, K // group), per, axis=1))
        term = s[None] * (I - o[None] * R[:, None, :]).astype(np.float64)
    return (d[:, None, :] * term).sum(axis=-1)


# ---------------------------------------------------------------------------
# App. B.1 (formats table): llama.cpp GGUF blocks, array of structures.
# ---------------------------------------------------------------------------

def gguf_block_bytes(q: int, with_min: bool) -> int:
    """Bytes of one 32-weight block: binary16 s, [binary16 m,] 32 q-bit indices."""
    return 2 + (2 if with_min else 0) + 32 * q // 8


def to_gguf(u: np.ndarray, scales: np.ndarray, mins: Optional[np.ndarray], group: int, q: int) -> np.ndarray:
    """GGUF blocks of indices u [rows, cols] (cols a multiple of 32) with binary16 scales
    (and minimums) [rows, cols/group]: uint8 [rows, cols/32, gguf_block_bytes(q, ...)].
    Index order inside qs: READINGS["gguf_order"]."""
    u = np.asarray(u, dtype=np.int64)
    rows, cols = u.shape
    nb = cols // 32
    ub = u.reshape(rows, nb, 32)
    if q == 4:
        qs = ub[:, :, :16] | (ub[:, :, 16:] << 4)                                 # [rows, nb, 16]
    elif q == 2:
        quads = ub.reshape(rows, nb, 8, 4)
        qs = quads[..., 0] | (quads[..., 1] << 2) | (quads[..., 2] << 4) | (quads[..., 3] << 6)
    else:
        raise ValueError("GGUF blocks exist for q = 2 and q = 4 only")
    per = group // 32
    fields = [np.repeat(np.asarray(scales, np.uint16).reshape(rows, cols // group), per, axis=1)]
    if mins is not None:
        fields.append(np.repeat(np.asarray(mins, np.uint16).reshape(rows, cols // group), per, axis=1))
    parts = []
    for f in fields:                                         # binary16, little-endian
        parts += [(f & 0xFF)[..., None], (f >> 8)[..., None]]
    parts.append(qs)
    return np.concatenate(parts, axis=-1).astype(np.uint8)


def from_gguf(blocks: np.ndarray, q: int, with_min: bool):
    """Inverse of :func:`to_gguf` at group 32: (u int64 [rows, cols], s uint16 [rows, cols/32],
    m uint16 [rows, cols/32] or None)."""
    b = np.asarray(blocks, dtype=np.uint16)
    rows, nb, _ = b.shape
    s = b[..., 0] | (b[..., 1] << 8)
    m = (b[..., 2] | (b[..., 3] << 8)) if with_min else None
    qs = b[..., 4 if with_min else 2:].astype(np.int64)
    if q == 4:
        u = np.concatenate([qs & 0xF, qs >> 4], axis=-1)                        # [rows, nb, 32]
    else:
        u = np.stack([(qs >> (2 * k)) & 3 for k in range(4)], axis=-1).reshape(rows, nb, 32)
    return u.reshape(rows, nb * 32), s, m


def gguf_dequantize(blocks: np.ndarray, q: int, with_min: bool) -> np.ndarray:
    """Weights in binary64 as the formats read back: s*(u - 2^(q-1)) for Q*_0 (Q*_0s),
    s*u + m for Q*_1."""
    u, s, m = from_gguf(blocks, q, with_min)
    rows, cols = u.shape
    sb = f16_bits_to_f64(s).reshape(rows, cols // 32, 1)
    ub = u.reshape(rows, cols // 32, 32).astype(np.float64)
    if with_min:
        return (sb * ub + f16_bits_to_f64(m).reshape(rows, cols // 32, 1)).reshape(rows, cols)
    return (sb * (ub - (1 << (q - 1)))).reshape(rows, cols)
