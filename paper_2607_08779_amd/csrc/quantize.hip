// Group-wise quantize + pack kernel (signed absmax, absmax, min-max grids).
//
// Sec. 3 of the paper: Eq. (2) min-max grid, Eq. (3) absmax grid, Eq. (4)-(5)
// signed absmax grid and its sign rule; Eq. (1) is the quantizer all three use.
// App. B.1: one binary16 scale per group and packed few-bit indices (the Q*_1 layout
// adds a binary16 minimum per group).
//
// Mapping.  The matrix is one flat stream of rows*cols weights (cols is a
// multiple of the group, so no group straddles a row).  Each lane owns a chunk
// of 8 consecutive weights (16 bytes of bf16, one coalesced load); a group of G
// weights is G/8 consecutive lanes of one wavefront, which reduce max/min with
// butterfly shuffles.  Each lane quantizes its 8 weights and packs them into
// 8q bits; neighbouring lanes merge those bits so every store is a dword.
//
// DIAG (signed grid only) also stores each group's sign-rule margin and gain (Sec. 4
// Remark 1, sign_stats.h) from the same registers: one pass over the weights.
#include "sign_stats.h"
#include "ssq_internal.h"

namespace ssq {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 2;   // chunks per thread, loaded before any is processed (1, 4, 8 measured slower)

template <typename In>
struct Loader;

template <>
struct Loader<uint16_t> {  // bf16 bits, 16 bytes per chunk
  static __device__ __forceinline__ void load(const uint16_t* W, int64_t chunk, float (&w)[8]) {
    const u32x4 d = load_stream16(W + 8 * chunk);
    w[0] = bf16_lo(d.x); w[1] = bf16_hi(d.x); w[2] = bf16_lo(d.y); w[3] = bf16_hi(d.y);
    w[4] = bf16_lo(d.z); w[5] = bf16_hi(d.z); w[6] = bf16_lo(d.w); w[7] = bf16_hi(d.w);
  }
};

template <>
struct Loader<float> {  // binary32, 32 bytes per chunk
  static __device__ __forceinline__ void load(const float* W, int64_t chunk, float (&w)[8]) {
    const u32x4 a = load_stream16(W + 8 * chunk);
    const u32x4 b = load_stream16(W + 8 * chunk + 4);
    w[0] = __uint_as_float(a.x); w[1] = __uint_as_float(a.y); w[2] = __uint_as_float(a.z);
    w[3] = __uint_as_float(a.w); w[4] = __uint_as_float(b.x); w[5] = __uint_as_float(b.y);
    w[6] = __uint_as_float(b.z); w[7] = __uint_as_float(b.w);
  }
};

// Store the 8q bits `v` of chunk `chunk` (its bytes start at chunk*q) as whole dwords.
// Every lane must call this (the neighbour exchange is a wavefront shuffle).
// The value of the next lane (DPP row_shl:1; the partners below never cross a 16-lane row).
__device__ __forceinline__ uint32_t next_lane(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x101, 0xF, 0xF, false);
}

template <int Q>
__device__ __forceinline__ void store_codes(uint8_t* codes, int64_t chunk, uint32_t v, bool valid) {
  if constexpr (Q == 4) {
    if (valid) reinterpret_cast<uint32_t*>(codes)[chunk] = v;
  } else if constexpr (Q == 2) {
    const uint32_t next = next_lane(v);
    if (valid && (chunk & 1) == 0) reinterpret_cast<uint32_t*>(codes)[chunk >> 1] = v | (next << 16);
  } else {  // Q == 3: the 24-bit words of four lanes form three dwords
    const uint32_t next = next_lane(v);
    const int j = (int)(chunk & 3);
    if (valid && j < 3)
      reinterpret_cast<uint32_t*>(codes)[(chunk >> 2) * 3 + j] = (v >> (8 * j)) | (next << (24 - 8 * j));
  }
}

template <typename In, int Q, int G, int MODE, bool DIAG = false>
__global__ __launch_bounds__(kThreads) void quantize_kernel(const In* __restrict__ W,
                                                            int64_t total_chunks,
                                                            uint8_t* __restrict__ codes,
                                                            uint16_t* __restrict__ scales,
                                                            void* __restrict__ meta,
                                                            int16_t* __restrict__ margin = nullptr,
                                                            float* __restrict__ gain = nullptr) {
  static_assert(!DIAG || MODE == 0, "the diagnostics describe the signed grid");
  constexpr int kLanesPerGroup = G / 8;
  constexpr float kLo = -(float)(1 << (Q - 1));          // min A_q (signed alphabet)
  constexpr float kHi = (float)((1 << (Q - 1)) - 1);     // max A_q
  constexpr float kTop = (float)((1 << Q) - 1);          // max of the unsigned alphabet
  constexpr float kHalfRange = (float)(1 << (Q - 1));    // 2^(q-1)

  const int64_t base = (int64_t)blockIdx.x * (kThreads * kUnroll) + threadIdx.x;
  float w[kUnroll][8];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t chunk = base + (int64_t)u * kThreads;
    if (chunk < total_chunks) {
      Loader<In>::load(W, chunk, w[u]);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) w[u][i] = 0.0f;
    }
  }

#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t chunk = base + (int64_t)u * kThreads;
    const bool valid = chunk < total_chunks;
    float mx = w[u][0], mn = w[u][0];
#pragma unroll
    for (int i = 1; i < 8; ++i) { mx = fmaxf(mx, w[u][i]); mn = fminf(mn, w[u][i]); }
    mx = group_max<kLanesPerGroup>(mx);            // max_j w_j over the group
    const float nmn = group_max<kLanesPerGroup>(-mn);  // -min_j w_j
    int diag_m = 0;
    double diag_g = 0.0;
    if constexpr (DIAG) {
      // bf16 weights: packed 16-bit statistics unless a group of the wavefront has a
      // tiny or zero maximum (a wave-uniform choice: both exchange values between lanes)
      const uint32_t mb = (__float_as_uint(fmaxf(mx, nmn)) >> 16) & 0x7FFFu;
      if (sizeof(In) == 2 && __builtin_amdgcn_ballot_w64(mb < 0x100u) == 0) {
        uint32_t d[4];
        bf16_pairs_perm(w[u], d);
        sign_stats_bf16<Q, G>(d, mb, mx > nmn, diag_m, diag_g);
      } else
        sign_stats<Q, G>(w[u], mx, nmn, diag_m, diag_g);
    }

    uint32_t packed = 0;
    uint16_t scale_bits = 0;
    uint8_t zero_point = 0;
    uint16_t min_bits = 0;
    if constexpr (MODE == 0 || MODE == 1) {
      // Eq. (3) / Eq. (5): M = ||w||_inf, alpha = M / 2^(q-1) (exact), s = gamma*alpha with
      // gamma = -1 iff the largest magnitude is a positive entry not matched by a negative one.
      const float amax = fmaxf(mx, nmn);
      const bool neg = (MODE == 0) && (mx > nmn);
      const float alpha = amax * (1.0f / kHalfRange);
      const float s = neg ? -alpha : alpha;
      if (amax == 0.0f) {
#pragma unroll
        for (int i = 0; i < 8; ++i) packed |= (uint32_t)(1u << (Q - 1)) << (Q * i);
      } else if (sizeof(In) == 2 && amax >= 0x1p-100f && amax <= 0x1p100f) {
        // bf16 weights: w and M carry 8-bit significands, so the exact quotient w/s is either
        // a half-integer or at least 2^-11 away from every half-integer, while
        // w * (2^(q-1)/M) is within 2^-19 of it.  Snapping that product to the 2^-12 grid
        // (one fma against 3072, whose ulp is 2^-12) lands exactly on the half when the
        // quotient is one and on the correct side otherwise, so rint of the snapped value
        // equals rint(fl32(w/s)) -- the division result -- bit for bit.
        //
        // The snapped value t = 3072 + q' (|q'| <= 2^(q-1), a multiple of 2^-12) plus
        // 1.5*2^23 - 3072 is 1.5*2^23 + q' exactly, rounded once at ulp 1: the low mantissa
        // bits then hold rne(q') = c, and bits - bits(1.5*2^23) + 2^(q-1) is the offset-binary
        // index u in [0, 2^q].  |w| <= M keeps c >= -2^(q-1), so only the top clip can bind.
        float rs = (1.0f / amax) * kHalfRange;
        if (neg) rs = -rs;
        constexpr float kRound = 12582912.0f - 3072.0f;                    // 1.5*2^23 - 3072
        constexpr uint32_t kBias = 0x4B400000u - (1u << (Q - 1));          // bits(1.5*2^23) - 2^(q-1)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float t = __builtin_fmaf(w[u][i], rs, 3072.0f);
          const uint32_t idx = __float_as_uint(t + kRound) - kBias;
          packed |= min(idx, (uint32_t)kTop) << (Q * i);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float c = fminf(fmaxf(rintf(w[u][i] / s), kLo), kHi);   // Eq. (1), z = 0
          packed |= (uint32_t)((int)c + (1 << (Q - 1))) << (Q * i);
        }
      }
      scale_bits = amax == 0.0f ? (uint16_t)0 : f32_to_f16_bits(s);
    } else {
      // Eq. (2).  MODE 2 (u8 zero point): the range widened to contain 0, so the integer
      // zero point fits [0, 2^q-1].  MODE 3 (binary16 minimum, the Q*_1 layout of
      // App. B.1): the group's own range, codes rint((w - min)/s) -- Eq. (1) with the
      // real zero point -min/s -- and the minimum stored beside the scale.
      const float lo_v = MODE == 2 ? fminf(-nmn, 0.0f) : -nmn;
      const float hi_v = MODE == 2 ? fmaxf(mx, 0.0f) : mx;
      const float s = (hi_v - lo_v) / kTop;
      if constexpr (MODE == 3) {       // a minimum that is (or rounds to) a zero is stored as +0
        min_bits = f32_to_f16_bits(lo_v);
        if ((min_bits & 0x7FFFu) == 0) min_bits = 0;
      }
      if (s != 0.0f) {
        // rint(fl32(a/s)) without a division, for the zero point (a = -min') and every
        // weight (a = w, or a = fl32(w - min) for MODE 3).  In both cases |a| <= the
        // range, so |a/s| < 2^q - 1 + 2^-16 < 16.  With r = rcp(s) (within 1 ulp of 1/s;
        // s is normal and far from overflow), t = a*r is within 0.75 * 2^-18 of a/s, and
        // fl32(a/s) within 2^-21 of a/s, so fl32(a/s) lies within 2^-18 of t.  When t is
        // farther than 2^-18 from every half-integer (|t - rint(t)| < 1/2 - 2^-18, an
        // exact difference), rint(t) is rint(fl32(a/s)).  Otherwise the half-integer h
        // next to t decides: if h*s == a exactly (one fma, which cannot underflow for
        // s >= 2^-100) the quotient is h itself, else the value is divided.  Exact
        // half-integer quotients are common with bf16 weights (~0.2 % of weights); those
        // and the rarer near misses branch.
        const bool fast = s >= 0x1p-100f && s <= 0x1p100f;
        const float r = __builtin_amdgcn_rcpf(s);
        auto rint_quotient = [&](float a) {
          const float t = a * r;
          float c = rintf(t);
          if (!fast || __builtin_fabsf(t - c) >= 0.5f - 0x1p-18f) {
            const float h = t > c ? c + 0.5f : c - 0.5f;
            c = fast && __builtin_fmaf(h, s, -a) == 0.0f ? rintf(h) : rintf(a / s);
          }
          return c;
        };
        const float z = MODE == 2 ? fminf(fmaxf(rint_quotient(-lo_v), 0.0f), kTop) : 0.0f;
        float rq[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) rq[i] = rint_quotient(MODE == 2 ? w[u][i] : w[u][i] - lo_v);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float c = fminf(fmaxf(rq[i] + z, 0.0f), kTop);
          packed |= (uint32_t)(int)c << (Q * i);
        }
        zero_point = (uint8_t)(int)z;
        scale_bits = f32_to_f16_bits(s);
      }
    }

    store_codes<Q>(codes, chunk, packed, valid);
    if (valid && (chunk % kLanesPerGroup) == 0) {
      scales[chunk / kLanesPerGroup] = scale_bits;
      if constexpr (MODE == 2) static_cast<uint8_t*>(meta)[chunk / kLanesPerGroup] = zero_point;
      if constexpr (MODE == 3) static_cast<uint16_t*>(meta)[chunk / kLanesPerGroup] = min_bits;
      if constexpr (DIAG) {
        margin[chunk / kLanesPerGroup] = (int16_t)diag_m;
        gain[chunk / kLanesPerGroup] = (float)diag_g;
      }
    }
  }
}

template <typename In, int Q, int G>
hipError_t launch_mode(const In* W, int64_t total_chunks, int mode, uint8_t* codes,
                       uint16_t* scales, void* zp, hipStream_t stream) {
  const int64_t per_block = (int64_t)kThreads * kUnroll;
  const dim3 grid((unsigned)((total_chunks + per_block - 1) / per_block));
  switch (mode) {
    case 0: quantize_kernel<In, Q, G, 0><<<grid, kThreads, 0, stream>>>(W, total_chunks, codes, scales, zp); break;
    case 1: quantize_kernel<In, Q, G, 1><<<grid, kThreads, 0, stream>>>(W, total_chunks, codes, scales, zp); break;
    case 2: quantize_kernel<In, Q, G, 2><<<grid, kThreads, 0, stream>>>(W, total_chunks, codes, scales, zp); break;
    default: quantize_kernel<In, Q, G, 3><<<grid, kThreads, 0, stream>>>(W, total_chunks, codes, scales, zp); break;
  }
  return hipGetLastError();
}

template <typename In, int Q>
hipError_t launch_group(const In* W, int64_t total_chunks, int group, int mode, uint8_t* codes,
                        uint16_t* scales, void* zp, hipStream_t stream) {
  switch (group) {
    case 32: return launch_mode<In, Q, 32>(W, total_chunks, mode, codes, scales, zp, stream);
    case 64: return launch_mode<In, Q, 64>(W, total_chunks, mode, codes, scales, zp, stream);
    default: return launch_mode<In, Q, 128>(W, total_chunks, mode, codes, scales, zp, stream);
  }
}

template <typename In, int Q, int G>
hipError_t launch_diag(const In* W, int64_t total_chunks, uint8_t* codes, uint16_t* scales, int16_t* margin,
                       float* gain, hipStream_t stream) {
  const int64_t per_block = (int64_t)kThreads * kUnroll;
  const dim3 grid((unsigned)((total_chunks + per_block - 1) / per_block));
  quantize_kernel<In, Q, G, 0, true><<<grid, kThreads, 0, stream>>>(W, total_chunks, codes, scales, nullptr,
                                                                   margin, gain);
  return hipGetLastError();
}

template <typename In>
hipError_t launch_diag_any(const In* W, int64_t rows, int64_t cols, int group, int q, uint8_t* codes,
                           uint16_t* scales, int16_t* margin, float* gain, hipStream_t stream) {
  const int64_t total_chunks = rows * cols / 8;
  if (total_chunks == 0) return hipSuccess;
  switch (q * 1000 + group) {
    case 2032: return launch_diag<In, 2, 32>(W, total_chunks, codes, scales, margin, gain, stream);
    case 2064: return launch_diag<In, 2, 64>(W, total_chunks, codes, scales, margin, gain, stream);
    case 2128: return launch_diag<In, 2, 128>(W, total_chunks, codes, scales, margin, gain, stream);
    case 3032: return launch_diag<In, 3, 32>(W, total_chunks, codes, scales, margin, gain, stream);
    case 3064: return launch_diag<In, 3, 64>(W, total_chunks, codes, scales, margin, gain, stream);
    case 3128: return launch_diag<In, 3, 128>(W, total_chunks, codes, scales, margin, gain, stream);
    case 4032: return launch_diag<In, 4, 32>(W, total_chunks, codes, scales, margin, gain, stream);
    case 4064: return launch_diag<In, 4, 64>(W, total_chunks, codes, scales, margin, gain, stream);
    case 4128: return launch_diag<In, 4, 128>(W, total_chunks, codes, scales, margin, gain, stream);
    default: return hipErrorInvalidValue;
  }
}

template <typename In>
hipError_t launch_any(const In* W, int64_t rows, int64_t cols, int group, int q, int mode,
                      uint8_t* codes, uint16_t* scales, void* zp, hipStream_t stream) {
  const int64_t total_chunks = rows * cols / 8;
  if (total_chunks == 0) return hipSuccess;
  switch (q) {
    case 2: return launch_group<In, 2>(W, total_chunks, group, mode, codes, scales, zp, stream);
    case 3: return launch_group<In, 3>(W, total_chunks, group, mode, codes, scales, zp, stream);
    default: return launch_group<In, 4>(W, total_chunks, group, mode, codes, scales, zp, stream);
  }
}

}  // namespace

hipError_t launch_quantize_bf16(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                                int mode, uint8_t* codes, uint16_t* scales, void* zp,
                                hipStream_t stream) {
  return launch_any<uint16_t>(W, rows, cols, group, q, mode, codes, scales, zp, stream);
}

hipError_t launch_quantize_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                               int mode, uint8_t* codes, uint16_t* scales, void* zp,
                               hipStream_t stream) {
  return launch_any<float>(W, rows, cols, group, q, mode, codes, scales, zp, stream);
}

hipError_t launch_quantize_diag_bf16(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                                     uint8_t* codes, uint16_t* scales, int16_t* margin, float* gain,
                                     hipStream_t stream) {
  return launch_diag_any<uint16_t>(W, rows, cols, group, q, codes, scales, margin, gain, stream);
}

hipError_t launch_quantize_diag_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                                    uint8_t* codes, uint16_t* scales, int16_t* margin, float* gain,
                                    hipStream_t stream) {
  return launch_diag_any<float>(W, rows, cols, group, q, codes, scales, margin, gain, stream);
}

}  // namespace ssq
