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

// Raw buffer descriptors: base address + byte count (gfx9 word 3).  A load at or past
// the byte count returns zeros, which serves as free predication at ragged edges.
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));
constexpr int kBufferWord3 = 0x00020000;
constexpr int kStream = 2;   // cache policy bits: non-temporal (data read once)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferWord3);
}

// Codes of one 32-weight block (4q bytes) from a buffer, as q dwords.
template <int Q>
__device__ __forceinline__ void buffer_block_codes(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                                   uint32_t (&d)[Q]) {
  if constexpr (Q == 4) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, kStream);
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  } else if constexpr (Q == 2) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, kStream);
    d[0] = v.x; d[1] = v.y;
  } else {
    const u32x3 v = __builtin_amdgcn_raw_buffer_load_b96(r, (int)voff, (int)soff, kStream);
    d[0] = v.x; d[1] = v.y; d[2] = v.z;
  }
}

// (v & mask) | magic in one v_and_or_b32.  gfx9 VOP3 encodings take no literals and
// read one SGPR, so the mask rides in an SGPR and the magic in a VGPR; left to itself
// the compiler emits separate and/or instructions.
__device__ __forceinline__ uint32_t and_or(uint32_t v, uint32_t mask, uint32_t magic) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(v), "s"(mask), "v"(magic));
  return r;
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
// Maximum over aligned groups of WIDTH (4, 8 or 16) lanes, in every lane of the group,
// with DPP moves (no LDS round trip): quad_perm xor 1 and xor 2 make each quad uniform,
// row_half_mirror pairs the two quads of an 8-lane half-row, row_mirror the two halves
// of a 16-lane row.
template <int CTRL>
__device__ __forceinline__ float dpp_max(float v) {
  const int moved = __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false);
  return fmaxf(v, __int_as_float(moved));
}
template <int WIDTH>
__device__ __forceinline__ float group_max(float v) {
  static_assert(WIDTH == 4 || WIDTH == 8 || WIDTH == 16, "group of 4, 8 or 16 lanes");
  v = dpp_max<0xB1>(v);                          // quad_perm [1,0,3,2]
  v = dpp_max<0x4E>(v);                          // quad_perm [2,3,0,1]
  if constexpr (WIDTH >= 8) v = dpp_max<0x141>(v);   // row_half_mirror
  if constexpr (WIDTH >= 16) v = dpp_max<0x140>(v);  // row_mirror
  return v;
}

// Sum over a whole wavefront; the total lands in lane 63.  Row-local DPP steps
// (quad_perm, half-mirror, mirror), then row_bcast:15 / row_bcast:31 carry the row
// sums across the four 16-lane rows.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float v) {
  const int moved = __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xF, false);
  return v + __int_as_float(moved);
}
__device__ __forceinline__ float wave_sum(float v) {
  v = dpp_add<0xB1, 0xF>(v);    // quad_perm [1,0,3,2]
  v = dpp_add<0x4E, 0xF>(v);    // quad_perm [2,3,0,1]
  v = dpp_add<0x141, 0xF>(v);   // row_half_mirror
  v = dpp_add<0x140, 0xF>(v);   // row_mirror
  v = dpp_add<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3
  v = dpp_add<0x143, 0xC>(v);   // row_bcast:31 into rows 2 and 3
  return v;
}

template <int WIDTH>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int o = 1; o < WIDTH; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Per-group metadata stored beside the scales: none (the symmetric formats), an
// integer zero point (u8, the weight reads s*(u - z)) or a binary16 minimum (the Q*_1
// layout of App. B.1, the weight reads s*u + m).
enum : int { kMetaNone = 0, kMetaZp = 1, kMetaMin = 2 };
struct GroupMeta {
  const void* ptr;   // u8 [N, K/group] zero points, u16 [N, K/group] binary16 minimums, or null
  int kind;          // kMetaNone, kMetaZp or kMetaMin
};

// Instantiate FN<q, group, meta kind>(args...) for the supported (q, group) pairs and
// return its result from the enclosing function.
#define SSQ_DISPATCH_QGM_CASE(FN, Q, G, ...)                                                   \
  case Q * 1000 + G * 3 + 0: return FN<Q, G, 0>(__VA_ARGS__);                                \
  case Q * 1000 + G * 3 + 1: return FN<Q, G, 1>(__VA_ARGS__);                                \
  case Q * 1000 + G * 3 + 2: return FN<Q, G, 2>(__VA_ARGS__);
#define SSQ_DISPATCH_QGM(FN, q, group, kind, ...)                                              \
  do {                                                                                       \
    switch (q * 1000 + group * 3 + kind) {                                                   \
      SSQ_DISPATCH_QGM_CASE(FN, 2, 32, __VA_ARGS__) SSQ_DISPATCH_QGM_CASE(FN, 2, 64, __VA_ARGS__)     \
      SSQ_DISPATCH_QGM_CASE(FN, 2, 128, __VA_ARGS__) SSQ_DISPATCH_QGM_CASE(FN, 3, 32, __VA_ARGS__)    \
      SSQ_DISPATCH_QGM_CASE(FN, 3, 64, __VA_ARGS__) SSQ_DISPATCH_QGM_CASE(FN, 3, 128, __VA_ARGS__)    \
      SSQ_DISPATCH_QGM_CASE(FN, 4, 32, __VA_ARGS__) SSQ_DISPATCH_QGM_CASE(FN, 4, 64, __VA_ARGS__)     \
      SSQ_DISPATCH_QGM_CASE(FN, 4, 128, __VA_ARGS__)                                         \
      default: return hipErrorInvalidValue;                                                  \
    }                                                                                        \
  } while (0)

// ---------------------------------------------------------------------------
// Host-side launchers (arguments already validated by the C ABI layer)
// ---------------------------------------------------------------------------

// Quantize modes: 0 signed symmetric, 1 unsigned symmetric, 2 min-max with a u8 zero
// point (`meta` = u8 [rows, cols/group]), 3 min-max with a binary16 minimum (`meta` =
// u16 [rows, cols/group]); `meta` is null for the symmetric modes.
constexpr int kModeAsymMin = 3;
hipError_t launch_quantize_bf16(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                                int mode, uint8_t* codes, uint16_t* scales, void* meta,
                                hipStream_t stream);
hipError_t launch_quantize_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                               int mode, uint8_t* codes, uint16_t* scales, void* meta,
                               hipStream_t stream);
hipError_t launch_gemv_bf16(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                            GroupMeta meta, int64_t N, int64_t K, int group, int q, uint16_t* y,
                            hipStream_t stream);
hipError_t launch_matmul_f32(const float* x, int64_t M, const uint8_t* codes,
                             const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K,
                             int group, int q, float* y, hipStream_t stream);
hipError_t launch_gemm_bf16(const uint16_t* x, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K,
                            int group, int q, uint16_t* y, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);
// Workspace bytes that let the GEMM split its reduction (0 when splitting would not help).
size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

// Layout of a split-reduction workspace, the same for every kernel and shape: arrival
// counters (one u32 per output tile or row block) in the first kSplitCounterBytes, fp32
// partials after them.  Counters always sit in the same bytes, so a workspace that one
// call left with its counters back at zero is valid for any later shape: no call's
// partials can land where another call's counters live.  A plan that would need more
// counters than fit does not split.
constexpr int64_t kSplitCounterBytes = 65536;
constexpr int64_t kMaxSplitCounters = kSplitCounterBytes / 4;


// Token counts 2..kSkinnyMaxM run the skinny-M kernels (weights dequantized once into
// MFMA operands; with a workspace the reduction is split across workgroups).
constexpr int64_t kSkinnyMaxM = 32;
hipError_t launch_skinny_bf16(const uint16_t* x, int64_t M, const uint8_t* codes,
                              const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K,
                              int group, int q, uint16_t* y, void* workspace, size_t workspace_bytes,
                              hipStream_t stream);
size_t skinny_workspace_bytes(int64_t M, int64_t N, int64_t K, int q);

// Sign-rule diagnostics (Sec. 4): per-group margin and gain, optional 3x3 tally.
hipError_t launch_diagnostics_bf16(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                                   int16_t* margin, float* gain, uint64_t* tally);
hipError_t launch_diagnostics_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                                  int16_t* margin, float* gain, uint64_t* tally);

// Signed quantization fused with the sign-rule margin and gain (quantize.hip).
hipError_t launch_quantize_diag_bf16(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                                     uint8_t* codes, uint16_t* scales, int16_t* margin, float* gain,
                                     hipStream_t stream);
hipError_t launch_quantize_diag_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                                    uint8_t* codes, uint16_t* scales, int16_t* margin, float* gain,
                                    hipStream_t stream);

// Q8_0 activations and the integer-dot matmul (q8.hip).
hipError_t launch_quantize_act_q8(const uint16_t* x, int64_t M, int64_t K, int8_t* q, uint16_t* d,
                                  hipStream_t stream);
hipError_t launch_matmul_q8(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K, int group, int q,
                            uint16_t* y, hipStream_t stream);

// GGUF array-of-structures export (export.hip): q in {2, 4}; mins null for Q*_0.
int64_t gguf_block_bytes(int q, bool with_min);
hipError_t launch_export_gguf(const uint8_t* codes, const uint16_t* scales, const uint16_t* mins, int64_t rows,
                              int64_t cols, int group, int q, uint8_t* out, hipStream_t stream);

}  // namespace ssq
