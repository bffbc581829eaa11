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

}  // namespace ssq
