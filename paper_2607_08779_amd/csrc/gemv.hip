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
#include <algorithm>

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

// sum_{k in block} x[k] * (128 + u[k]) in fp32.  `magic` holds kMagic (in a VGPR).
template <int Q>
__device__ __forceinline__ float block_dot(const Block<Q>& b, const uint32_t (&xp)[16], uint32_t magic) {
  float acc = 0.0f;
  if constexpr (Q == 4) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t w4 = b.d[d] >> 4;
      acc = dot2(and_or(b.d[d], 0x000F000Fu, magic), xp[4 * d], acc);
      acc = dot2(and_or(w4, 0x000F000Fu, magic), xp[4 * d + 1], acc);
      acc = dot2(and_or(b.d[d] >> 8, 0x000F000Fu, magic), xp[4 * d + 2], acc);
      acc = dot2(and_or(w4 >> 8, 0x000F000Fu, magic), xp[4 * d + 3], acc);
    }
  } else if constexpr (Q == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc = dot2(and_or(b.d[d] >> (2 * j), 0x00030003u, magic), xp[8 * d + j], acc);
  } else {
    // Re-split the 96 bits into four 24-bit words of 8 fields, then move fields 4..7 of
    // each word up to bit 16 so that pairs (e_j, e_{j+4}) share one shift.
    const uint32_t v[4] = {b.d[0], __builtin_amdgcn_alignbit(b.d[1], b.d[0], 24),
                           __builtin_amdgcn_alignbit(b.d[2], b.d[1], 16), b.d[2] >> 8};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t s = (v[w] & 0xFFFu) | ((v[w] << 4) & 0x0FFF0000u);
#pragma unroll
      for (int j = 0; j < 4; ++j) acc = dot2(and_or(s >> (3 * j), 0x00070007u, magic), xp[4 * w + j], acc);
    }
  }
  return acc;
}

// Work split.  A team of T threads (T = blocks per row rounded up to whole
// wavefronts, at most 1024) owns kRows consecutive rows; thread t takes block t of
// each row (and t + T, ... for rows longer than 1024 blocks).  Short rows pack
// several teams into one 256-thread workgroup.  Each thread issues its activation
// load and its kRows code and scale loads before any arithmetic and consumes them
// in issue order, so many small wavefronts stream and compute concurrently.
// Partial sums meet through a DPP wavefront reduction and LDS.
//
// Every row has its own buffer descriptor whose range is the row (or empty for rows
// past N), and all offsets travel in the range-checked VGPR offset: rows past N read
// zeros and contribute nothing.
#ifndef SSQ_GEMV_ROWS
#define SSQ_GEMV_ROWS 4          // rows per team
#endif
constexpr int kRows = SSQ_GEMV_ROWS;
constexpr int kMaxWaves = 16;

template <int Q, int G, bool ZP>
__global__ __launch_bounds__(1024) void gemv_kernel(const uint16_t* __restrict__ x,
                                                    const uint8_t* __restrict__ codes,
                                                    const uint16_t* __restrict__ scales,
                                                    const uint8_t* __restrict__ zp, int N, int K,
                                                    int team_threads, uint16_t* __restrict__ y) {
  constexpr int kBlocksPerGroup = G / 32;
  constexpr float kSymOffset = kMagicValue + (float)(1 << (Q - 1));
  __shared__ float partial[kMaxWaves][kRows];

  // team_threads is a multiple of 64, so the team index is uniform across a wavefront.
  const int team = __builtin_amdgcn_readfirstlane((int)threadIdx.x / team_threads);
  const int t = (int)threadIdx.x - team * team_threads;
  const int teams = blockDim.x / team_threads;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row0 = ((int64_t)blockIdx.x * teams + team) * kRows;
  const int nblk = K / 32;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)(K / G);
  const uint32_t magic = kMagic;
  const int64_t rows_here = N - row0 < kRows ? (N - row0 > 0 ? N - row0 : 0) : kRows;

  __amdgpu_buffer_rsrc_t rc[kRows], rs[kRows], rz[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    const bool live = r < rows_here;
    const int64_t row = live ? row0 + r : 0;
    rc[r] = make_rsrc(codes + row * row_bytes, live ? row_bytes : 0u);
    rs[r] = make_rsrc(scales + row * groups_per_row, live ? groups_per_row * 2 : 0u);
    rz[r] = make_rsrc(ZP ? zp + row * groups_per_row : zp, ZP && live ? groups_per_row : 0u);
  }
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)K * 2);

  float yacc[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) yacc[r] = 0.0f;

  auto consume = [&](const uint32_t (&X)[16], const Block<Q> (&cb)[kRows], const uint32_t (&sbits)[kRows],
                     const uint32_t (&zbits)[kRows]) {
    float xs = 0.0f;  // sum of the block's activations
#pragma unroll
    for (int i = 0; i < 16; ++i) xs = dot2(X[i], kOnes, xs);
    uint32_t xp[16];
    permute_x<Q>(X, xp);
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const float acc = block_dot<Q>(cb[r], xp, magic);
      const float sc = f16_bits_to_f32(sbits[r]);
      const float off = ZP ? kMagicValue + (float)zbits[r] : kSymOffset;
      yacc[r] = __builtin_fmaf(sc, __builtin_fmaf(-off, xs, acc), yacc[r]);
    }
  };
  auto load_rows = [&](int j, Block<Q> (&cb)[kRows], uint32_t (&sbits)[kRows], uint32_t (&zbits)[kRows]) {
    const uint32_t coff = (uint32_t)j * (4 * Q);
    const uint32_t goff = (uint32_t)(j / kBlocksPerGroup);
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      buffer_block_codes<Q>(rc[r], coff, 0, cb[r].d);
      sbits[r] = __builtin_amdgcn_raw_buffer_load_b16(rs[r], goff * 2, 0, 0);
      zbits[r] = ZP ? __builtin_amdgcn_raw_buffer_load_b8(rz[r], goff, 0, 0) : 0u;
    }
  };

  if (rows_here > 0) {
    for (int j = t; j < nblk; j += team_threads) {
      // Loads first, in consumption order: the activation block, then per row its codes,
      // scale (and zero point).
      uint32_t X[16];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rx, j * 64 + 16 * i, 0, 0);
        X[4 * i] = v.x; X[4 * i + 1] = v.y; X[4 * i + 2] = v.z; X[4 * i + 3] = v.w;
      }
      Block<Q> cb[kRows];
      uint32_t sbits[kRows], zbits[kRows];
      load_rows(j, cb, sbits, zbits);
      consume(X, cb, sbits, zbits);
    }
  }
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    const float v = wave_sum(yacc[r]);
    if (lane == 63) partial[wave][r] = v;
  }
  __syncthreads();
  if (t < kRows) {
    const int64_t row = row0 + t;
    if (row < N) {
      const int waves_per_team = team_threads / 64;
      float v = 0.0f;
      for (int w = 0; w < waves_per_team; ++w) v += partial[team * waves_per_team + w][t];
      y[row] = f32_to_bf16_bits(v);
    }
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
  const int64_t nblk = K / 32;
  const int team = (int)std::min<int64_t>(1024, (nblk + 63) / 64 * 64);
  const int teams = team >= 256 ? 1 : 256 / team;
  const int64_t rows_per_block = (int64_t)teams * kRows;
  const dim3 grid((unsigned)((N + rows_per_block - 1) / rows_per_block));
  gemv_kernel<Q, G, ZP><<<grid, team * teams, 0, stream>>>(x, codes, scales, zp, (int)N, (int)K,
                                                           team, y);
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
