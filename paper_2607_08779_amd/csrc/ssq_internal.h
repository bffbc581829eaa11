// Internal declarations shared by the libssq translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssq {

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Streaming loads that bypass cache retention (each byte is read once).
__device__ __forceinline__ u32x4 load_stream16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x2 load_stream8(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
}
__device__ __forceinline__ uint32_t load_stream4(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
}

// Codes of one 32-weight block (4q bytes) as q dwords.
template <int Q>
__device__ __forceinline__ void load_block_codes(const uint8_t* p, uint32_t (&d)[Q]) {
  if constexpr (Q == 4) {
    const u32x4 v = load_stream16(p);
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  } else if constexpr (Q == 2) {
    const u32x2 v = load_stream8(p);
    d[0] = v.x; d[1] = v.y;
  } else {
    d[0] = load_stream4(p); d[1] = load_stream4(p + 4); d[2] = load_stream4(p + 8);
  }
}

// Field k (q bits) of a little-endian bit stream held in dwords d[].
template <int Q>
__device__ __forceinline__ uint32_t field(const uint32_t* d, int k) {
  const int bit = k * Q, w = bit >> 5, sh = bit & 31;
  uint32_t v = d[w] >> sh;
  if (sh + Q > 32) v |= d[w + 1] << (32 - sh);
  return v & ((1u << Q) - 1u);
}

__device__ __forceinline__ float bf16_lo(uint32_t d) { return __uint_as_float(d << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t d) { return __uint_as_float(d & 0xFFFF0000u); }

// binary32 -> bfloat16 bits, round half to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  __bf16 h = (__bf16)f;
  return __builtin_bit_cast(uint16_t, h);
}

// binary32 -> binary16 bits, round half to even (v_cvt_f16_f32 in the default mode).
__device__ __forceinline__ uint16_t f32_to_f16_bits(float f) {
  _Float16 h = (_Float16)f;
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t bits) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}

// Butterfly reduction over aligned lane sets of `width` lanes (width a power of two <= 64).
template <int WIDTH>
__device__ __forceinline__ float group_max(float v) {
#pragma unroll
  for (int o = 1; o < WIDTH; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

template <int WIDTH>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int o = 1; o < WIDTH; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Instantiate FN<q, group, has_zp>(args...) for the supported (q, group) pairs and
// return its result from the enclosing function.
#define SSQ_DISPATCH_QGZ(FN, q, group, has_zp, ...)                                          \
  do {                                                                                     \
    switch (q * 1000 + group * 2 + (has_zp ? 1 : 0)) {                                     \
      case 2064: return FN<2, 32, false>(__VA_ARGS__);  case 2065: return FN<2, 32, true>(__VA_ARGS__); \
      case 2128: return FN<2, 64, false>(__VA_ARGS__);  case 2129: return FN<2, 64, true>(__VA_ARGS__); \
      case 2256: return FN<2, 128, false>(__VA_ARGS__); case 2257: return FN<2, 128, true>(__VA_ARGS__); \
      case 3064: return FN<3, 32, false>(__VA_ARGS__);  case 3065: return FN<3, 32, true>(__VA_ARGS__); \
      case 3128: return FN<3, 64, false>(__VA_ARGS__);  case 3129: return FN<3, 64, true>(__VA_ARGS__); \
      case 3256: return FN<3, 128, false>(__VA_ARGS__); case 3257: return FN<3, 128, true>(__VA_ARGS__); \
      case 4064: return FN<4, 32, false>(__VA_ARGS__);  case 4065: return FN<4, 32, true>(__VA_ARGS__); \
      case 4128: return FN<4, 64, false>(__VA_ARGS__);  case 4129: return FN<4, 64, true>(__VA_ARGS__); \
      case 4256: return FN<4, 128, false>(__VA_ARGS__); case 4257: return FN<4, 128, true>(__VA_ARGS__); \
      default: return hipErrorInvalidValue;                                                \
    }                                                                                      \
  } while (0)

// ---------------------------------------------------------------------------
// Host-side launchers (arguments already validated by the C ABI layer)
// ---------------------------------------------------------------------------

hipError_t launch_quantize_bf16(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                                int mode, uint8_t* codes, uint16_t* scales, uint8_t* zp,
                                hipStream_t stream);
hipError_t launch_quantize_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                               int mode, uint8_t* codes, uint16_t* scales, uint8_t* zp,
                               hipStream_t stream);
hipError_t launch_gemv_bf16(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                            const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
                            hipStream_t stream);
hipError_t launch_matmul_f32(const float* x, int64_t M, const uint8_t* codes,
                             const uint16_t* scales, const uint8_t* zp, int64_t N, int64_t K,
                             int group, int q, float* y, hipStream_t stream);
hipError_t launch_gemm_bf16(const uint16_t* x, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, const uint8_t* zp, int64_t N, int64_t K,
                            int group, int q, uint16_t* y, hipStream_t stream);

}  // namespace ssq
