// Decode GEMV (M = 1) over packed few-bit weights, plus the binary32 matmul.
//
// App. B.3 of the paper: with W[n,k] ~ s[n,b] (u[n,k] - o[n,b]) in group b,
//   y[n] = sum_b s[n,b] * ( sum_{k in b} x[k] u[n,k]  -  o[n,b] sum_{k in b} x[k] ).
// The symmetric formats (signed or not -- the sign lives in s) have the
// constant offset o = 2^(q-1); the asymmetric one reads o from zp.
//
// Streaming design (HBM bound).  The unit of work is a block of 32 consecutive
// weights of one row: 4q bytes of codes, loaded by one lane with one vector
// load.  A wavefront owns R rows and its lanes stride over the blocks of those
// rows, so every code byte is read once, coalesced.  Codes become bf16 pairs
// by OR-ing two q-bit fields into the mantissa of the bf16 constant 128
// (0x4300 | u == 128 + u exactly), and v_dot2_f32_bf16 multiplies them with
// activation pairs in fp32.  The 128 + o offset is removed once per block with
// the block's activation sum, and the scale is applied once per block.
#include "ssq_internal.h"

namespace ssq {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr uint32_t kMagic = 0x43004300u;   // bf16 pair (128.0, 128.0)
constexpr uint32_t kOnes = 0x3F803F80u;    // bf16 pair (1.0, 1.0)
constexpr float kMagicValue = 128.0f;

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                         __builtin_bit_cast(bf16x2, b), c, false);
}

// Codes of one 32-weight block: 4q bytes.
template <int Q>
struct Block {
  uint32_t d[Q];
};

template <int Q>
__device__ __forceinline__ Block<Q> load_block(const uint8_t* p) {
  Block<Q> b;
  load_block_codes<Q>(p, b.d);
  return b;
}

// Activation pairs laid out to match the code pairs produced by block_dot.
// For q = 4 and q = 3 every 8 weights form pairs (e_j, e_{j+4}); for q = 2
// every 16 weights form pairs (e_j, e_{j+8}).  xp[] holds 16 bf16 pairs.
template <int Q>
__device__ __forceinline__ void permute_x(const uint32_t (&X)[16], uint32_t (&xp)[16]) {
  constexpr uint32_t kLo = 0x05040100u, kHi = 0x07060302u;
  if constexpr (Q == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        xp[8 * d + j] = __builtin_amdgcn_perm(X[8 * d + 4 + j / 2], X[8 * d + j / 2], (j & 1) ? kHi : kLo);
  } else {
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        xp[4 * d + j] = __builtin_amdgcn_perm(X[4 * d + 2 + j / 2], X[4 * d + j / 2], (j & 1) ? kHi : kLo);
  }
}

// sum_{k in block} x[k] * (128 + u[k]) in fp32.
template <int Q>
__device__ __forceinline__ float block_dot(const Block<Q>& b, const uint32_t (&xp)[16]) {
  float acc = 0.0f;
  if constexpr (Q == 4) {
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc = dot2(((b.d[d] >> (4 * j)) & 0x000F000Fu) | kMagic, xp[4 * d + j], acc);
  } else if constexpr (Q == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc = dot2(((b.d[d] >> (2 * j)) & 0x00030003u) | kMagic, xp[8 * d + j], acc);
  } else {
    // Re-split the 96 bits into four 24-bit words of 8 fields, then move fields 4..7 of
    // each word up to bit 16 so that pairs (e_j, e_{j+4}) share one shift.
    const uint32_t v[4] = {b.d[0] & 0xFFFFFFu, __builtin_amdgcn_alignbit(b.d[1], b.d[0], 24) & 0xFFFFFFu,
                           __builtin_amdgcn_alignbit(b.d[2], b.d[1], 16) & 0xFFFFFFu, b.d[2] >> 8};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t s = (v[w] & 0xFFFu) | ((v[w] << 4) & 0x0FFF0000u);
#pragma unroll
      for (int j = 0; j < 4; ++j) acc = dot2(((s >> (3 * j)) & 0x00070007u) | kMagic, xp[4 * w + j], acc);
    }
  }
  return acc;
}

template <int Q, int G, bool ZP, int R, int U>
__global__ __launch_bounds__(256) void gemv_kernel(const uint16_t* __restrict__ x,
                                                   const uint8_t* __restrict__ codes,
                                                   const uint16_t* __restrict__ scales,
                                                   const uint8_t* __restrict__ zp, int N, int K,
                                                   uint16_t* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int64_t row0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * R;
  if (row0 >= N) return;  // whole wavefront
  const int nblk = K / 32;
  const int64_t row_bytes = (int64_t)K * Q / 8;
  const int groups_per_row = K / G;
  constexpr int kBlocksPerGroup = G / 32;
  constexpr float kSymOffset = kMagicValue + (float)(1 << (Q - 1));

  float yacc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) yacc[r] = 0.0f;

  for (int j0 = lane; j0 < nblk; j0 += 64 * U) {
    Block<Q> cb[U][R];
    float sc[U][R], off[U][R];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + 64 * u;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int64_t row = row0 + r;
        if (j < nblk && row < N) {
          cb[u][r] = load_block<Q>(codes + row * row_bytes + (int64_t)j * (4 * Q));
          const int64_t gi = row * groups_per_row + j / kBlocksPerGroup;
          sc[u][r] = f16_bits_to_f32(scales[gi]);
          off[u][r] = ZP ? kMagicValue + (float)zp[gi] : kSymOffset;
        } else {
#pragma unroll
          for (int i = 0; i < Q; ++i) cb[u][r].d[i] = 0;
          sc[u][r] = 0.0f;
          off[u][r] = 0.0f;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + 64 * u;
      if (j >= nblk) break;
      uint32_t X[16];
      const uint4* xv = reinterpret_cast<const uint4*>(x) + (int64_t)j * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint4 t = xv[i];
        X[4 * i] = t.x; X[4 * i + 1] = t.y; X[4 * i + 2] = t.z; X[4 * i + 3] = t.w;
      }
      float xs = 0.0f;  // sum of the block's activations
#pragma unroll
      for (int i = 0; i < 16; ++i) xs = dot2(X[i], kOnes, xs);
      uint32_t xp[16];
      permute_x<Q>(X, xp);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const float acc = block_dot<Q>(cb[u][r], xp);
        yacc[r] = __builtin_fmaf(sc[u][r], __builtin_fmaf(-off[u][r], xs, acc), yacc[r]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const float v = group_sum<64>(yacc[r]);
    if (lane == 0 && row0 + r < N) y[row0 + r] = f32_to_bf16_bits(v);
  }
}

// ---------------------------------------------------------------------------
// Binary32 matmul: x[M,K] fp32, y[M,N] fp32.  One wavefront per (row n, 4 tokens);
// each lane dequantizes whole 32-weight blocks exactly in fp32.
// ---------------------------------------------------------------------------

constexpr int kF32Tokens = 4;

template <int Q, int G, bool ZP>
__global__ __launch_bounds__(256) void matmul_f32_kernel(const float* __restrict__ x, int M,
                                                         const uint8_t* __restrict__ codes,
                                                         const uint16_t* __restrict__ scales,
                                                         const uint8_t* __restrict__ zp, int N,
                                                         int K, float* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int m0 = blockIdx.y * kF32Tokens;
  if (n >= N) return;
  const int nblk = K / 32;
  const int64_t row_bytes = (int64_t)K * Q / 8;
  float acc[kF32Tokens] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int j = lane; j < nblk; j += 64) {
    const Block<Q> b = load_block<Q>(codes + n * row_bytes + (int64_t)j * (4 * Q));
    const int64_t gi = n * (K / G) + j / (G / 32);
    const float s = f16_bits_to_f32(scales[gi]);
    const float o = ZP ? (float)zp[gi] : (float)(1 << (Q - 1));
    float w[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) w[k] = s * ((float)field<Q>(b.d, k) - o);   // exact in fp32
#pragma unroll
    for (int t = 0; t < kF32Tokens; ++t) {
      if (m0 + t >= M) break;
      const float* xr = x + (int64_t)(m0 + t) * K + (int64_t)j * 32;
      float a = 0.0f;
#pragma unroll
      for (int k = 0; k < 32; ++k) a = __builtin_fmaf(xr[k], w[k], a);
      acc[t] += a;
    }
  }
#pragma unroll
  for (int t = 0; t < kF32Tokens; ++t) {
    const float v = group_sum<64>(acc[t]);
    if (lane == 0 && m0 + t < M) y[(int64_t)(m0 + t) * N + n] = v;
  }
}

template <int Q, int G, bool ZP>
hipError_t gemv_dispatch(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                         const uint8_t* zp, int64_t N, int64_t K, uint16_t* y, hipStream_t stream) {
  constexpr int R = 2, U = 2;
  const dim3 grid((unsigned)((N + 4 * R - 1) / (4 * R)));
  gemv_kernel<Q, G, ZP, R, U><<<grid, 256, 0, stream>>>(x, codes, scales, zp, (int)N, (int)K, y);
  return hipGetLastError();
}

template <int Q, int G, bool ZP>
hipError_t f32_dispatch(const float* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                        const uint8_t* zp, int64_t N, int64_t K, float* y, hipStream_t stream) {
  const dim3 grid((unsigned)((N + 3) / 4), (unsigned)((M + kF32Tokens - 1) / kF32Tokens));
  matmul_f32_kernel<Q, G, ZP><<<grid, 256, 0, stream>>>(x, (int)M, codes, scales, zp, (int)N, (int)K, y);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemv_bf16(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                            const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
                            hipStream_t stream) {
  SSQ_DISPATCH_QGZ(gemv_dispatch, q, group, zp != nullptr, x, codes, scales, zp, N, K, y, stream);
}

hipError_t launch_matmul_f32(const float* x, int64_t M, const uint8_t* codes,
                             const uint16_t* scales, const uint8_t* zp, int64_t N, int64_t K,
                             int group, int q, float* y, hipStream_t stream) {
  SSQ_DISPATCH_QGZ(f32_dispatch, q, group, zp != nullptr, x, M, codes, scales, zp, N, K, y, stream);
}

}  // namespace ssq
