// Weight dequantization for the MFMA kernels (GEMM and skinny-M matmul).
//
// App. B.3 of the paper: the weight a code stands for is s*(u - o), with o = 2^(q-1)
// for the symmetric formats and o = z for the asymmetric one; the Q*_1 layout of
// App. B.1 stores a minimum m instead (s*u + m).  These helpers turn a thread's share
// of a 32-weight block of packed codes into bf16 MFMA operands.
#pragma once

#include "ssq_internal.h"

namespace ssq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float f16_lo(uint32_t p) { return (float)__builtin_bit_cast(_Float16, (uint16_t)p); }
__device__ __forceinline__ float f16_hi(uint32_t p) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(p >> 16)); }

// Dwords of a block's codes one thread loads: its 1/P share (q=3 loads the whole
// 12-byte block, whose halves are not dword aligned).
template <int Q, int P>
struct Part {
  static constexpr int kDwords = Q == 3 ? 3 : Q / P;
  static constexpr int kFields = 32 / P;
};

template <int Q, int P>
__device__ __forceinline__ void load_part(__amdgpu_buffer_rsrc_t r, uint32_t off, int part,
                                          uint32_t (&d)[Part<Q, P>::kDwords]) {
  constexpr int kBytes = 4 * Part<Q, P>::kDwords;
  const uint32_t o = Q == 3 ? off : off + (uint32_t)(part * kBytes);
  if constexpr (kBytes == 16) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)o, 0, kStream);
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  } else if constexpr (kBytes == 12) {
    const u32x3 v = __builtin_amdgcn_raw_buffer_load_b96(r, (int)o, 0, kStream);
    d[0] = v.x; d[1] = v.y; d[2] = v.z;
  } else if constexpr (kBytes == 8) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)o, 0, kStream);
    d[0] = v.x; d[1] = v.y;
  } else {
    d[0] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)o, 0, kStream);
  }
}

// This thread's 32/P weights s*(u - o), natural k order, as bf16 pairs.  Each q-bit
// field is OR-ed into the mantissa of the fp16 constant 1024 (0x6400 | u == 1024 + u),
// two fields per instruction; one v_fma_mix_f32 per weight forms
// (1024 + u)*s - (1024 + o)*s.  Both products are exact in fp32 (11-bit by 11-bit), so
// the result is s*(u - o) exactly; it is rounded to bf16 once.  `so` = -(1024 + o)*s.
template <int Q, int P>
__device__ __forceinline__ void dequant_part(const uint32_t (&d)[Part<Q, P>::kDwords], int part,
                                             float s, float so, uint32_t (&w)[16 / P]) {
  const uint32_t magic = 0x64006400u;
  constexpr int kF = Part<Q, P>::kFields;
  float f[kF];
  if constexpr (Q == 4) {
#pragma unroll
    for (int i = 0; i < kF / 8; ++i) {
      const uint32_t v4 = d[i] >> 4;
      const uint32_t p[4] = {and_or(d[i], 0x000F000Fu, magic), and_or(v4, 0x000F000Fu, magic),
                             and_or(d[i] >> 8, 0x000F000Fu, magic), and_or(v4 >> 8, 0x000F000Fu, magic)};
#pragma unroll
      for (int j = 0; j < 4; ++j) {          // p[j] holds fields j and j + 4 of this dword
        f[8 * i + j] = __builtin_fmaf(f16_lo(p[j]), s, so);
        f[8 * i + j + 4] = __builtin_fmaf(f16_hi(p[j]), s, so);
      }
    }
  } else if constexpr (Q == 2) {
#pragma unroll
    for (int i = 0; i < kF / 16; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {          // fields j and j + 8 of this dword
        const uint32_t p = and_or(d[i] >> (2 * j), 0x00030003u, magic);
        f[16 * i + j] = __builtin_fmaf(f16_lo(p), s, so);
        f[16 * i + j + 8] = __builtin_fmaf(f16_hi(p), s, so);
      }
  } else {
    // 24-bit words of 8 fields (the block has four); this part owns words
    // [4/P * part, 4/P * (part + 1)).  Fields 4..7 of a word move up to bit 16.
    const uint32_t v[4] = {d[0], __builtin_amdgcn_alignbit(d[1], d[0], 24),
                           __builtin_amdgcn_alignbit(d[2], d[1], 16), d[2] >> 8};
#pragma unroll
    for (int i = 0; i < kF / 8; ++i) {
      const uint32_t word = v[(4 / P) * part + i];
      const uint32_t sp = (word & 0xFFFu) | ((word << 4) & 0x0FFF0000u);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t p = and_or(sp >> (3 * j), 0x00070007u, magic);
        f[8 * i + j] = __builtin_fmaf(f16_lo(p), s, so);
        f[8 * i + j + 4] = __builtin_fmaf(f16_hi(p), s, so);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kF / 2; ++k) w[k] = pack_bf16x2(f[2 * k], f[2 * k + 1]);
}

// Constant term `so` of the dequantization (1024 + u)*s + so for each metadata layout:
// -(1024 + o)*s with the offset o = 2^(q-1) (symmetric) or the zero point z (both
// products exact: 11-bit by 11-bit), or m - 1024*s for the binary16 minimum layout
// (one rounding; the weight s*u + m is then within an ulp of fp32).
template <int META, int Q>
__device__ __forceinline__ float dequant_offset(float s, uint32_t meta_bits) {
  if constexpr (META == kMetaMin) {
    return __builtin_fmaf(-1024.0f, s, f16_bits_to_f32(meta_bits));
  } else {
    const float o = META == kMetaZp ? (float)meta_bits : (float)(1 << (Q - 1));
    return -(1024.0f + o) * s;
  }
}

// Load of one group's metadata (zero point u8 or binary16 minimum) at group index gi.
template <int META>
__device__ __forceinline__ uint32_t load_group_meta(__amdgpu_buffer_rsrc_t r, uint32_t gi, bool in) {
  if constexpr (META == kMetaMin) return __builtin_amdgcn_raw_buffer_load_b16(r, in ? gi * 2 : 0x80000000u, 0, 0);
  else if constexpr (META == kMetaZp) return __builtin_amdgcn_raw_buffer_load_b8(r, in ? gi : 0x80000000u, 0, 0);
  else return 0u;
}
template <int META>
constexpr int meta_size() { return META == kMetaMin ? 2 : META == kMetaZp ? 1 : 0; }

// s_waitcnt on the vector-memory counter only (gfx9 encoding: vmcnt in bits 3:0 and
// 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima).  Loads complete in order,
// so vmcnt <= N means everything but the last N loads has landed -- including loads
// that write LDS directly, which the compiler does not track.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | 0x70 | 0xF00 | ((N >> 4) << 14));
}

// Workgroup barrier for LDS only: this wavefront's LDS operations are waited for
// (s_waitcnt lgkmcnt(0), the gfx9 encoding with vmcnt and expcnt at their maxima), then
// s_barrier, written as a memory-clobbering asm statement.  The compiler's own barrier
// (and __syncthreads' fences) also waits for every direct-to-LDS load in flight, i.e.
// the prefetch, and for the global stores.  Callers make sure no LDS location read
// after it is still being written by a load in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);
  asm volatile("s_barrier" ::: "memory");
}

}  // namespace ssq
