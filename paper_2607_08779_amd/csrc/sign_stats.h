// Per-group statistics of the sign rule (Sec. 4 Def. 1, Lemma 1, Remark 1), shared by
// the diagnostics kernel and the fused quantize + diagnostics kernel.
//
// For a group of G weights held 8 per lane by G/8 consecutive lanes, with the group's
// max and -min already reduced: gamma* by Eq. (5) (ties +1), the clipped sets of both
// signs (Def. 1, Eq. (6)), the margin m = |C_{-g*}| - |C_{g*}| and the realised gain
// g = 2 alpha (sum_{C_{-g*}} (-g* w_i - T) - sum_{C_{g*}} (g* w_i - T)) (Lemma 1,
// Eq. (7)), T = M (1 - 2^-q).  The tests and excess sums are exact integer arithmetic:
// with M = f 2^E (frexp) and S = 25 + q - E, every weight of a clipped set, M itself and
// T scale by 2^S to integers below 2^(25+q) (members lie in (M/2, M], so their ulp is at
// least 2^(E-25); T = M - M 2^-q has ulp at least 2^(E-24-q)), and an excess is below
// 2^25, so the sum over a group of up to 128 fits 32 bits.  ldexp by S cannot overflow
// (|w| <= M) and is exact for members; a non-member, whether ldexp rounds it
// (underflow) or the conversion truncates it, stays at or below the integer threshold.
// Only the final product 2 alpha * (sum) 2^-S rounds (binary64); callers store its
// binary32 rounding.
#pragma once

#include "ssq_internal.h"

namespace ssq {

// Integer sum over aligned groups of WIDTH (4, 8 or 16) lanes, in every lane of the
// group, with the DPP pairings of group_max.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_add_u32(uint32_t v) {
  return v + (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int WIDTH>
__device__ __forceinline__ uint32_t group_sum_u32(uint32_t v) {
  v = dpp_add_u32<0xB1>(v);
  v = dpp_add_u32<0x4E>(v);
  if constexpr (WIDTH >= 8) v = dpp_add_u32<0x141>(v);
  if constexpr (WIDTH >= 16) v = dpp_add_u32<0x140>(v);
  return v;
}

// m and g of the lane's group (valid in every lane of it).  mx = max w, nmn = -min w
// over the group.  Every lane of the wavefront must call this (DPP exchanges).
template <int Q, int G>
__device__ __forceinline__ void sign_stats(const float (&w)[8], float mx, float nmn, int& m, double& g) {
  constexpr int kLanes = G / 8;
  const bool gamma_neg = mx > nmn;                        // Eq. (5): gamma* = -1, ties -> +1
  const float M = fmaxf(mx, nmn);                         // ||w||_inf
  const int S = 25 + Q - __builtin_amdgcn_frexp_expf(M);
  const int xm = (int)__builtin_amdgcn_ldexpf(M, S);      // M 2^S
  const uint32_t t = (uint32_t)(xm - (xm >> Q));          // T 2^S
  uint32_t e_all = 0, e_neg = 0;       // excesses (|w_i| - T) 2^S over both clipped sets / C_{-1}
  uint32_t counts = 0;                 // |C_{+1}| + |C_{-1}| + 2^16 |C_{-1}|
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    // Def. 1: w_i is in C_{sign(w_i)} iff |w_i| > T; the saturating difference is the
    // excess of a member and zero otherwise.
    const uint32_t x = (uint32_t)__builtin_amdgcn_ldexpf(fabsf(w[i]), S);   // exact for members
    const uint32_t d = __builtin_elementwise_sub_sat(x, t);
    const uint32_t neg = (uint32_t)(__float_as_int(w[i]) >> 31);            // all ones if w_i < 0
    const uint32_t dn = d & neg;
    e_all += d;
    e_neg += dn;
    counts += min(d, 1u) + (min(dn, 1u) << 16);
  }
  e_all = group_sum_u32<kLanes>(e_all);
  e_neg = group_sum_u32<kLanes>(e_neg);
  counts = group_sum_u32<kLanes>(counts);
  const uint32_t e_pos = e_all - e_neg;
  const int c_neg = (int)(counts >> 16), c_pos = (int)(counts & 0xFFFFu) - c_neg;
  // margin and gain of gamma* against -gamma*: the other sign's set minus gamma*'s
  m = gamma_neg ? c_pos - c_neg : c_neg - c_pos;
  const double excess = gamma_neg ? (double)e_pos - (double)e_neg : (double)e_neg - (double)e_pos;
  const double two_alpha = (double)M * (4.0 / (double)(1 << Q));   // 2 M / 2^(q-1), exact
  g = two_alpha * __builtin_amdgcn_ldexp(excess, -S);      // Lemma 1; the scaling is exact
}

// The same statistics for bf16 weights (their bit patterns, two per dword, w[2j] in the
// low half of pairs[j]) in packed 16-bit integer arithmetic, two weights per
// instruction.  mb is the magnitude bits of M as a bf16 (M's biased exponent
// em = mb >> 7 must be at least 2; callers route smaller groups, including all-zero
// ones, to sign_stats).  With the unit u = 2^(em - 135), a weight whose exponent is
// em - 1 or em is an integer v = |w|/u in [128, 510] (its 8-bit significand times 1 or
// 2), and every member of a clipped set has such an exponent (|w| > T >= 3M/4 > M/2
// for q >= 2).  Smaller exponents map to v = 0: the factor p = sat(e - (em - 2)) is
// 0, 1 or 2 and v = significand * p.  T/u = 2 mm (1 - 2^-q) (mm = M's significand)
// is a multiple of 2^-(q-1): a weight is a member iff v > floor(T/u), so the
// saturating difference d = sat(v - floor(T/u)) is positive exactly for members
// (d <= 2 mm 2^-q + 1 <= 128), and a set's excess is
// sum (v - T/u) = sum d - |C| (T/u - floor(T/u)), an integer after scaling by 2^(q-1).
// Every sum is exact and the one rounding is the product 2 alpha * (sum) u, as in
// sign_stats, so both give the same bits.
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef short i16x2 __attribute__((ext_vector_type(2)));

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_max_u16x2(uint32_t v) {
  const uint32_t moved = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, v),
                                                                __builtin_bit_cast(u16x2, moved)));
}

// min(x, 1) per half-word in one instruction (the compiler otherwise rewrites it as two
// compares and selects per half).
__device__ __forceinline__ u16x2 pk_min1_u16(u16x2 x) {
  uint32_t r;
  asm("v_pk_min_u16 %0, %1, 1 op_sel_hi:[1,0]" : "=v"(r) : "v"(__builtin_bit_cast(uint32_t, x)));
  return __builtin_bit_cast(u16x2, r);
}

// The four pairs of bf16 bit patterns that widened weights w[0..7] came from (pair j
// holds w[2j] in its low half): one byte permute per pair.
__device__ __forceinline__ void bf16_pairs_perm(const float (&w)[8], uint32_t (&d)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j)   // bytes 3:2 of w[2j+1] over bytes 3:2 of w[2j]
    d[j] = __builtin_amdgcn_perm(__float_as_uint(w[2 * j + 1]), __float_as_uint(w[2 * j]), 0x07060302u);
}

// For bf16 weights: the group's largest magnitude among non-negative-signed weights (P)
// and among negative-signed ones (N), as bf16 magnitude bits, in every lane of the
// group; returns mb = max(P, N) (the bits of M) and gamma* = -1 iff P > N (Eq. (5),
// ties +1).  Bit patterns of finite magnitudes order like their values, so this is the
// float rule on integers: as signed 16-bit values the non-negative weights are the
// largest, as unsigned ones the negative weights are.
template <int G>
__device__ __forceinline__ uint32_t group_absmax_bf16(const uint32_t (&d)[4], bool& gamma_neg) {
  constexpr int kLanes = G / 8;
  i16x2 pm = __builtin_bit_cast(i16x2, d[0]);
  u16x2 nm = __builtin_bit_cast(u16x2, d[0]);
#pragma unroll
  for (int j = 1; j < 4; ++j) {
    pm = __builtin_elementwise_max(pm, __builtin_bit_cast(i16x2, d[j]));
    nm = __builtin_elementwise_max(nm, __builtin_bit_cast(u16x2, d[j]));
  }
  const i16x2 zero = {0, 0};
  const u16x2 sign = {0x8000, 0x8000};
  const u16x2 p = __builtin_bit_cast(u16x2, __builtin_elementwise_max(pm, zero));   // none -> 0
  nm = __builtin_elementwise_sub_sat(nm, sign);                                      // none -> 0
  // {P, N} per lane, then over the group (one DPP move and one packed max per step)
  const u16x2 lo = {p.x, nm.x}, hi = {p.y, nm.y};
  uint32_t pn = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(lo, hi));
  pn = dpp_max_u16x2<0xB1>(pn);
  pn = dpp_max_u16x2<0x4E>(pn);
  if constexpr (kLanes >= 8) pn = dpp_max_u16x2<0x141>(pn);
  if constexpr (kLanes >= 16) pn = dpp_max_u16x2<0x140>(pn);
  const uint32_t P = pn & 0xFFFFu, N = pn >> 16;
  gamma_neg = P > N;
  return P > N ? P : N;
}

template <int Q, int G>
__device__ __forceinline__ void sign_stats_bf16(const uint32_t (&pairs)[4], uint32_t mb, bool gamma_neg,
                                                int& m, double& g) {
  static_assert(Q >= 2, "members must lie above M/2");
  constexpr int kLanes = G / 8;
  const uint32_t em = mb >> 7;
  const uint32_t mm = 0x80u | (mb & 0x7Fu);
  const uint32_t tq = (mm << Q) - mm;                     // (T/u) 2^(q-1)
  const uint32_t tfl = tq >> (Q - 1);                     // floor(T/u)
  const uint32_t tfrac = tq - (tfl << (Q - 1));           // (T/u - floor(T/u)) 2^(q-1)
  const u16x2 e2 = {(unsigned short)(em - 2), (unsigned short)(em - 2)};
  const u16x2 tf2 = {(unsigned short)tfl, (unsigned short)tfl};
  // Two 32-bit accumulators, each a sum over both sets in bits 0-14 plus 2^15 times the
  // sum over the negative set (C_{-1}): one v_dot2_u32_u16 per pair and accumulator,
  // with the multiplier 1 + 2^15 [w_i < 0] per half.  A group sums at most
  // 128 * 128 < 2^15 excess units, so neither field overflows, lanes included.
  uint32_t e_acc = 0, c_acc = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t d = pairs[j];
    const u16x2 mag = __builtin_bit_cast(u16x2, d & 0x7FFF7FFFu);
    const u16x2 p = __builtin_elementwise_sub_sat(mag >> 7, e2);
    const u16x2 v = __builtin_bit_cast(u16x2, (d & 0x007F007Fu) | 0x00800080u) * p;
    const u16x2 dd = __builtin_elementwise_sub_sat(v, tf2);           // Def. 1 membership and excess
    const u16x2 k = __builtin_bit_cast(u16x2, (d & 0x80008000u) | 0x00010001u);
    e_acc = __builtin_amdgcn_udot2(dd, k, e_acc, false);
    c_acc = __builtin_amdgcn_udot2(pk_min1_u16(dd), k, c_acc, false);
  }
  e_acc = group_sum_u32<kLanes>(e_acc);
  c_acc = group_sum_u32<kLanes>(c_acc);
  // differences negative set minus positive set, then oriented by gamma*
  const int dc = 2 * (int)(c_acc >> 15) - (int)(c_acc & 0x7FFFu);
  const int de = 2 * (int)(e_acc >> 15) - (int)(e_acc & 0x7FFFu);
  const int sgn = gamma_neg ? -1 : 1;
  m = sgn * dc;
  const int excess = sgn * ((de << (Q - 1)) - dc * (int)tfrac);   // sum (v - T/u) 2^(q-1), other minus star
  const double two_alpha = (double)__uint_as_float(mb << 16) * (4.0 / (double)(1 << Q));
  g = two_alpha * __builtin_amdgcn_ldexp((double)excess, (int)em - 135 - (Q - 1));
}

}  // namespace ssq
