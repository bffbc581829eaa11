// Prefill GEMM: y[M,N] = x[M,K] * What[N,K]^T with What dequantized into LDS.
//
// App. B.3 of the paper: What[n,k] = s[n,b] (u[n,k] - o[n,b]).  Prefill is a
// dense contraction, so it runs on bf16 MFMA.  Each workgroup owns a BM x BN
// output tile; per BK-deep step it stages the activation tile and dequantizes
// the weight tile (s*(u - o) is exact in fp32, then rounded to bf16) into LDS,
// and each of its four wavefronts multiplies a 64x64 sub-tile with
// v_mfma_f32_16x16x32_bf16, accumulating in fp32.
//
// MFMA operand layout (16x16x32): lane l supplies row (l % 16) of A and column
// (l % 16) of B, each with 8 consecutive k values starting at 8 * (l / 16).
// Both operands use the same k assignment, so the reduction is correct for any
// internal k order.  Lane l receives D[4 * (l / 16) + r][l % 16], r = 0..3.
#include "ssq_internal.h"

namespace ssq {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kStride = BK + 8;   // LDS row pitch in bf16 elements (144 bytes, 16-byte aligned)

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

template <int Q, int G, bool ZP>
__global__ __launch_bounds__(256) void gemm_kernel(const uint16_t* __restrict__ x, int M,
                                                   const uint8_t* __restrict__ codes,
                                                   const uint16_t* __restrict__ scales,
                                                   const uint8_t* __restrict__ zp, int N, int K,
                                                   uint16_t* __restrict__ y) {
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * kStride];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * kStride];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
  const int nblk = K / 32;
  const int64_t row_bytes = (int64_t)K * Q / 8;
  const int groups_per_row = K / G;

  // Loader roles: thread t stages row (t / 2), 32-wide half (t % 2) of both tiles.
  const int lr = tid >> 1, lh = tid & 1;
  const int64_t am = m0 + lr, bn = n0 + lr;

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  for (int kb = 0; kb < nblk; kb += 2) {
    const int blk = kb + lh;
    // Activation tile: 32 bf16 (64 bytes) per thread.
    {
      uint4 v[4];
      if (am < M && blk < nblk) {
        const uint4* p = reinterpret_cast<const uint4*>(x + am * K + (int64_t)blk * 32);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = p[i];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = uint4{0u, 0u, 0u, 0u};
      }
      uint4* dst = reinterpret_cast<uint4*>(As + lr * kStride + lh * 32);
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = v[i];
    }
    // Weight tile: dequantize one 32-weight block per thread.
    {
      uint32_t w[16];
      if (bn < N && blk < nblk) {
        uint32_t d[Q];
        load_block_codes<Q>(codes + bn * row_bytes + (int64_t)blk * (4 * Q), d);
        const int64_t gi = bn * groups_per_row + blk / (G / 32);
        const float s = f16_bits_to_f32(scales[gi]);
        const float o = ZP ? (float)zp[gi] : (float)(1 << (Q - 1));
        const float so = -s * o;   // exact: o has at most 4 bits, s 11
#pragma unroll
        for (int k = 0; k < 16; ++k)
          w[k] = pack_bf16x2(__builtin_fmaf((float)field<Q>(d, 2 * k), s, so),
                             __builtin_fmaf((float)field<Q>(d, 2 * k + 1), s, so));
      } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) w[k] = 0u;
      }
      uint4* dst = reinterpret_cast<uint4*>(Bs + lr * kStride + lh * 32);
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = uint4{w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 a[4], b[4];
      const int kofs = ks * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = *reinterpret_cast<const bf16x8*>(As + (wm * 64 + i * 16 + (lane & 15)) * kStride + kofs);
        b[i] = *reinterpret_cast<const bf16x8*>(Bs + (wn * 64 + i * 16 + (lane & 15)) * kStride + kofs);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t m = m0 + wm * 64 + i * 16 + 4 * (lane >> 4) + r;
        const int64_t n = n0 + wn * 64 + j * 16 + (lane & 15);
        if (m < M && n < N) y[m * N + n] = f32_to_bf16_bits(acc[i][j][r]);
      }
}

template <int Q, int G, bool ZP>
hipError_t gemm_dispatch(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                         const uint8_t* zp, int64_t N, int64_t K, uint16_t* y, hipStream_t stream) {
  const dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
  gemm_kernel<Q, G, ZP><<<grid, 256, 0, stream>>>(x, (int)M, codes, scales, zp, (int)N, (int)K, y);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const uint16_t* x, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, const uint8_t* zp, int64_t N, int64_t K,
                            int group, int q, uint16_t* y, hipStream_t stream) {
  SSQ_DISPATCH_QGZ(gemm_dispatch, q, group, zp != nullptr, x, M, codes, scales, zp, N, K, y, stream);
}

}  // namespace ssq
