// Q8_0 activations and the integer-dot decode matmul.
//
// Activations (Sec. 5.2, App. C): dynamic Q8_0 per token, blocks of 32, the
// narrow-range symmetric grid {-127, ..., 127}: d = amax / 127 in binary32, codes
// clip(rint(x / d)) from that d, stored scale binary16(d); an all-zero block stores
// d = +0 and codes 0.
//
// Matmul (App. B.3, the integer GEMM term and the row-sum correction): for the
// 32-activation block b inside weight group g,
//   I = sum_{j in b} q_j u_j,  R = sum_{j in b} q_j   (exact integers, v_dot4_i32_i8)
//   y += d_b s_g (I - o_g R)          symmetric offset o = 2^(q-1) or zero point z
//   y += d_b (s_g I + m_g R)          binary16 minimum layout (App. B.1 Q*_1)
// Codes are unsigned q-bit fields (0 .. 2^q - 1), so they are valid signed bytes and
// one signed 4-way byte dot product multiplies them with the activation codes.  The
// product d_b s_g of two binary16 values is exact in binary32 and so is I - o R
// (|I - o R| < 2^17), so each symmetric block term is rounded once, by the fma that
// adds it to the row's partial sum.
#include <algorithm>

#include "ssq_internal.h"
#include "mfma_dequant.h"

namespace ssq {
namespace {

// ---------------------------------------------------------------------------
// Activation quantization: 8 activations per lane, a block is 4 consecutive lanes.
// ---------------------------------------------------------------------------

constexpr int kActThreads = 256;

__global__ __launch_bounds__(kActThreads) void quantize_act_q8_kernel(const uint16_t* __restrict__ x,
                                                                      int64_t total_chunks,
                                                                      uint2* __restrict__ q,
                                                                      uint16_t* __restrict__ d) {
  const int64_t chunk = (int64_t)blockIdx.x * kActThreads + threadIdx.x;
  const bool valid = chunk < total_chunks;      // whole blocks: total_chunks is a multiple of 4
  float w[8];
  if (valid) {
    const u32x4 v = load_stream16(x + 8 * chunk);
    w[0] = bf16_lo(v.x); w[1] = bf16_hi(v.x); w[2] = bf16_lo(v.y); w[3] = bf16_hi(v.y);
    w[4] = bf16_lo(v.z); w[5] = bf16_hi(v.z); w[6] = bf16_lo(v.w); w[7] = bf16_hi(v.w);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = 0.0f;
  }
  float amax = fabsf(w[0]);
#pragma unroll
  for (int i = 1; i < 8; ++i) amax = fmaxf(amax, fabsf(w[i]));
  amax = group_max<4>(amax);
  const float dd = amax / 127.0f;                          // binary32, correctly rounded
  uint32_t packed[2] = {0u, 0u};
  if (amax != 0.0f) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float c = fminf(fmaxf(rintf(w[i] / dd), -127.0f), 127.0f);   // Eq. (1), z = 0
      packed[i >> 2] |= ((uint32_t)(int)c & 0xFFu) << (8 * (i & 3));
    }
  }
  if (valid) {
    q[chunk] = uint2{packed[0], packed[1]};
    if ((chunk & 3) == 0) d[chunk >> 2] = f32_to_f16_bits(amax != 0.0f ? dd : 0.0f);
  }
}

// ---------------------------------------------------------------------------
// Integer dot products of one 32-weight block.
// ---------------------------------------------------------------------------

__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// Activation bytes rearranged to the byte order in which block_idot unpacks the codes:
// q = 4 splits each dword of 8 nibbles into its even and odd fields; q = 2 takes field
// k of every byte, i.e. elements k, k+4, k+8, k+12 of 16 (a 4x4 byte transpose);
// q = 3 takes fields (j, j+1, j+4, j+5) of each 8-field word, j = 0 and 2.
template <int Q>
__device__ __forceinline__ void permute_xq(const uint32_t (&X)[8], uint32_t (&xp)[8]) {
  if constexpr (Q == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xp[2 * i] = __builtin_amdgcn_perm(X[2 * i + 1], X[2 * i], 0x06040200u);
      xp[2 * i + 1] = __builtin_amdgcn_perm(X[2 * i + 1], X[2 * i], 0x07050301u);
    }
  } else if constexpr (Q == 2) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t* x4 = X + 4 * h;
      const uint32_t a = __builtin_amdgcn_perm(x4[1], x4[0], 0x05010400u);   // x0b0 x1b0 x0b1 x1b1
      const uint32_t b = __builtin_amdgcn_perm(x4[1], x4[0], 0x07030602u);   // x0b2 x1b2 x0b3 x1b3
      const uint32_t c = __builtin_amdgcn_perm(x4[3], x4[2], 0x05010400u);
      const uint32_t e = __builtin_amdgcn_perm(x4[3], x4[2], 0x07030602u);
      xp[4 * h + 0] = __builtin_amdgcn_perm(c, a, 0x05040100u);
      xp[4 * h + 1] = __builtin_amdgcn_perm(c, a, 0x07060302u);
      xp[4 * h + 2] = __builtin_amdgcn_perm(e, b, 0x05040100u);
      xp[4 * h + 3] = __builtin_amdgcn_perm(e, b, 0x07060302u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xp[2 * i] = __builtin_amdgcn_perm(X[2 * i + 1], X[2 * i], 0x05040100u);
      xp[2 * i + 1] = __builtin_amdgcn_perm(X[2 * i + 1], X[2 * i], 0x07060302u);
    }
  }
}

// sum_{k in block} q[k] * u[k] with the activation bytes from permute_xq.
template <int Q>
__device__ __forceinline__ int block_idot(const uint32_t (&c)[Q], const uint32_t (&xp)[8]) {
  int acc = 0;
  if constexpr (Q == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc = sdot4(c[i] & 0x0F0F0F0Fu, xp[2 * i], acc);
      acc = sdot4((c[i] >> 4) & 0x0F0F0F0Fu, xp[2 * i + 1], acc);
    }
  } else if constexpr (Q == 2) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc = sdot4((c[h] >> (2 * k)) & 0x03030303u, xp[4 * h + k], acc);
  } else {
    // Four 24-bit words of 8 fields; fields 4..7 of a word move up to bit 16 so that
    // one shift serves fields j and j + 4.
    const uint32_t v[4] = {c[0], __builtin_amdgcn_alignbit(c[1], c[0], 24),
                           __builtin_amdgcn_alignbit(c[2], c[1], 16), c[2] >> 8};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t s = (v[i] & 0xFFFu) | ((v[i] << 4) & 0x0FFF0000u);
      const uint32_t lo = (s & 0x00070007u) | (((s >> 3) & 0x00070007u) << 8);          // f0 f1 f4 f5
      const uint32_t hi = ((s >> 6) & 0x00070007u) | (((s >> 9) & 0x00070007u) << 8);   // f2 f3 f6 f7
      acc = sdot4(lo, xp[2 * i], acc);
      acc = sdot4(hi, xp[2 * i + 1], acc);
    }
  }
  return acc;
}

// ---------------------------------------------------------------------------
// Decode GEMV: the streaming design of the bf16 GEMV (a workgroup owns kRows rows,
// lane i of wavefront w takes block 64 w + i of each row per pass, one vector load
// per block of codes, lanes contiguous) with 32 bytes of activation codes and one
// activation scale per block, loaded by the lane directly: the lanes' 32-byte runs
// are contiguous.  One token per grid row (blockIdx.y); further tokens re-read the
// weights.
// ---------------------------------------------------------------------------

constexpr int kRows = 4;
constexpr int kMaxTeam = 512;
constexpr int kMaxWaves = kMaxTeam / 64;
constexpr uint32_t kOutOfRange = 0x80000000u;

template <int Q, int G, int META>
__global__ __launch_bounds__(kMaxTeam) void gemv_q8_kernel(const int8_t* __restrict__ qx,
                                                           const uint16_t* __restrict__ dx,
                                                           const uint8_t* __restrict__ codes,
                                                           const uint16_t* __restrict__ scales,
                                                           const void* __restrict__ meta, int N, int K,
                                                           int threads, int token0, uint16_t* __restrict__ y) {
  constexpr int kBlocksPerGroup = G / 32;
  constexpr int kMetaSize = META == kMetaZp ? 1 : META == kMetaMin ? 2 : 0;
  __shared__ float partial[kMaxWaves][kRows];

  const int64_t m = token0 + blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int row0 = (int)blockIdx.x * kRows;
  const int rows_here = N - row0 < kRows ? N - row0 : kRows;   // >= 1
  const int nblk = K / 32;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)K / G;

  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes + (int64_t)row0 * row_bytes, (uint32_t)rows_here * row_bytes);
  const __amdgpu_buffer_rsrc_t rs =
      make_rsrc(scales + (int64_t)row0 * groups_per_row, (uint32_t)rows_here * groups_per_row * 2);
  const uint8_t* const mb = static_cast<const uint8_t*>(meta);
  const __amdgpu_buffer_rsrc_t rz =
      make_rsrc(kMetaSize ? mb + (int64_t)row0 * groups_per_row * kMetaSize : mb,
                kMetaSize ? (uint32_t)rows_here * groups_per_row * kMetaSize : 0u);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(qx + m * K, (uint32_t)K);
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(dx + m * nblk, (uint32_t)nblk * 2);

  float yacc[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) yacc[r] = 0.0f;

  for (int jw = wave * 64; jw < nblk; jw += threads) {   // uniform across the wavefront
    const int j = jw + lane;
    const bool live = j < nblk;
    const uint32_t xo = live ? (uint32_t)j * 32 : kOutOfRange;
    const u32x4 xa = __builtin_amdgcn_raw_buffer_load_b128(rx, (int)xo, 0, 0);
    const u32x4 xb = __builtin_amdgcn_raw_buffer_load_b128(rx, (int)xo, 16, 0);
    const uint32_t dbits = __builtin_amdgcn_raw_buffer_load_b16(rd, live ? (int)(j * 2) : (int)kOutOfRange, 0, 0);
    const uint32_t goff = (uint32_t)(j / kBlocksPerGroup);
    uint32_t sbits[kRows], zbits[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const uint32_t gi = r * groups_per_row + goff;
      sbits[r] = __builtin_amdgcn_raw_buffer_load_b16(rs, live ? (int)(gi * 2) : (int)kOutOfRange, 0, 0);
      if constexpr (META == kMetaMin)
        zbits[r] = __builtin_amdgcn_raw_buffer_load_b16(rz, live ? (int)(gi * 2) : (int)kOutOfRange, 0, 0);
      else if constexpr (META == kMetaZp)
        zbits[r] = __builtin_amdgcn_raw_buffer_load_b8(rz, live ? (int)gi : (int)kOutOfRange, 0, 0);
      else
        zbits[r] = 0u;
    }
    uint32_t cb[kRows][Q];
#pragma unroll
    for (int r = 0; r < kRows; ++r)
      buffer_block_codes<Q>(rc, live ? r * row_bytes + (uint32_t)j * (4 * Q) : kOutOfRange, 0, cb[r]);

    const uint32_t X[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
    int rsum = 0;                                           // R: the block's activation-code sum
#pragma unroll
    for (int i = 0; i < 8; ++i) rsum = sdot4(X[i], 0x01010101u, rsum);
    uint32_t xp[8];
    permute_xq<Q>(X, xp);
    const float dsc = f16_bits_to_f32(dbits);
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const int acc = block_idot<Q>(cb[r], xp);
      const float sc = f16_bits_to_f32(sbits[r]);
      if constexpr (META == kMetaMin) {
        const float t = __builtin_fmaf(sc, (float)acc, f16_bits_to_f32(zbits[r]) * (float)rsum);
        yacc[r] = __builtin_fmaf(dsc, t, yacc[r]);
      } else {
        const int o = META == kMetaZp ? (int)zbits[r] : (1 << (Q - 1));
        yacc[r] = __builtin_fmaf(sc * dsc, (float)(acc - o * rsum), yacc[r]);
      }
    }
  }
  // Four row sums at once, as in the bf16 GEMV: swapping lane halves folds the four
  // values of a lane into one; four DPP steps finish each 16-lane row.
  {
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(yacc[0]), __float_as_uint(yacc[1]), false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(yacc[2]), __float_as_uint(yacc[3]), false, false);
    const float s01 = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const float s23 = __uint_as_float(b[0]) + __uint_as_float(b[1]);
    const auto c = __builtin_amdgcn_permlane16_swap(__float_as_uint(s01), __float_as_uint(s23), false, false);
    float v = __uint_as_float(c[0]) + __uint_as_float(c[1]);
    v = dpp_add<0xB1, 0xF>(v);
    v = dpp_add<0x4E, 0xF>(v);
    v = dpp_add<0x141, 0xF>(v);
    v = dpp_add<0x140, 0xF>(v);
    if ((lane & 15) == 0) partial[wave][((lane >> 4) & 1) * 2 + (lane >> 5)] = v;
  }
  __syncthreads();
  if ((int)threadIdx.x < rows_here) {
    const int waves = threads >> 6;
    float v = 0.0f;
    for (int w = 0; w < waves; ++w) v += partial[w][threadIdx.x];
    y[m * N + row0 + threadIdx.x] = f32_to_bf16_bits(v);
  }
}

template <int Q, int G, int META>
hipError_t gemv_q8_dispatch(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, const void* meta, int64_t N, int64_t K, uint16_t* y,
                            hipStream_t stream) {
  const int64_t nblk = K / 32;
  const int64_t passes = (nblk + kMaxTeam - 1) / kMaxTeam;
  const int threads = (int)(((nblk + passes - 1) / passes + 63) / 64 * 64);
  constexpr int64_t kMaxGridY = 65535;
  for (int64_t m0 = 0; m0 < M; m0 += kMaxGridY) {
    const dim3 grid((unsigned)((N + kRows - 1) / kRows), (unsigned)std::min<int64_t>(M - m0, kMaxGridY));
    gemv_q8_kernel<Q, G, META><<<grid, threads, 0, stream>>>(qx, dx, codes, scales, meta, (int)N, (int)K,
                                                             threads, (int)m0, y);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// Batched decode (2 <= M <= 32 tokens per launch): one read of the weights for every
// token, the block terms on integer MFMA (v_mfma_i32_16x16x32_i8).
//
// A workgroup owns 16 weight rows; its W wavefronts take the quads (4 consecutive
// 32-weight blocks) of those rows in turn, quad w, w + W, ..., U quads per round: a round
// issues all its loads (the quads' codes go straight to a wavefront-private LDS slot, the
// activation codes and the weight scales to registers), waits for them, and multiplies.
// Per block and 16-token tile two MFMAs run: the first multiplies the tile's activation
// codes (A: row = token) with a B of constant bytes -o (or the row's -z[n, g]), the
// second with the block's weight codes (B: column = weight row), so the int32
// accumulator ends at I - o R exactly (|I - o R| < 2^17).  The binary16-minimum layout
// multiplies a B of ones into a second accumulator instead, for R.  Lane l holds
// D[4 (l/16) + r][l % 16], r = 0..3: tokens 4 (l/16) + r of weight row n0 + l % 16, and
// adds the block's term d[t, b] s[n, g] (I - o R) (or d (s I + m R)) in fp32, as the
// one-token kernel does.  The token scales d of the launch's tokens are staged in LDS,
// transposed to [block][token], so that a lane reads its four with one 8-byte load.
//
// Operand order.  Lane group c = l/16 of an MFMA supplies 8 consecutive k of the block:
// fields 8c..8c+7, q bytes at byte q*c of the block.  They are unpacked into bytes in
// a permuted k order (pairs of nibbles, fields of a 2-bit byte, ...), and the activation
// bytes of the same 8 k are permuted to match with two v_perm_b32; an MFMA sums over
// whichever k each operand slot stands for as long as A and B agree.
// The wavefronts' partial sums meet in LDS (wavefront order) at the end.
// ---------------------------------------------------------------------------

typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kSkinnyMaxWaves = 16;
constexpr int kSkinnyMaxK = 32768;       // token-scale staging: K/32 x 32 binary16 in LDS

template <int MT>
struct SkinnyQ8 {
  static constexpr int kTokens = 16 * MT;            // token rows of the A tiles
  static constexpr int kRounds = MT == 1 ? 4 : 2;    // quads per wavefront per round (U)
  static constexpr int kSlot = 1024;                 // LDS per quad: 16 rows x 16q bytes
};

// 8 fields (8q bits, fields at q-bit steps from bit 0) as 8 bytes, in the k order
// matched by act_pair<Q>: q = 4 [0 2 4 6 | 1 3 5 7], q = 2 [0 4 2 6 | 1 5 3 7],
// q = 3 [0 1 4 5 | 2 3 6 7].
template <int Q>
__device__ __forceinline__ int64_t code_bytes(uint32_t v) {
  uint32_t lo, hi;
  if constexpr (Q == 4) {
    lo = v & 0x0F0F0F0Fu;
    hi = (v >> 4) & 0x0F0F0F0Fu;
  } else if constexpr (Q == 2) {
    const uint32_t x = ((v << 12) & 0x0FFF0000u) | (v & 0xFFFFu);   // fields 2..7 also from bit 16
    lo = x & 0x03030303u;
    hi = (x >> 2) & 0x03030303u;
  } else {
    const uint32_t s = (v & 0xFFFu) | ((v << 4) & 0x0FFF0000u);      // fields 4..7 from bit 16
    lo = (s & 0x00070007u) | (((s >> 3) & 0x00070007u) << 8);
    hi = ((s >> 6) & 0x00070007u) | (((s >> 9) & 0x00070007u) << 8);
  }
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// 8 activation bytes (natural order, X0 = bytes 0..3) in code_bytes<Q>'s order.
template <int Q>
__device__ __forceinline__ int64_t act_pair(uint32_t x0, uint32_t x1) {
  constexpr uint32_t kLo = Q == 4 ? 0x06040200u : Q == 2 ? 0x06020400u : 0x05040100u;
  constexpr uint32_t kHi = Q == 4 ? 0x07050301u : Q == 2 ? 0x07030501u : 0x07060302u;
  const uint32_t lo = __builtin_amdgcn_perm(x1, x0, kLo), hi = __builtin_amdgcn_perm(x1, x0, kHi);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

template <int Q, int G, int META, int MT>
__global__ __launch_bounds__(1024) void skinny_q8_kernel(const int8_t* __restrict__ qx,
                                                         const uint16_t* __restrict__ dx, int M,
                                                         const uint8_t* __restrict__ codes,
                                                         const uint16_t* __restrict__ scales,
                                                         const void* __restrict__ meta, int N, int K,
                                                         int token0, uint16_t* __restrict__ y) {
  using S = SkinnyQ8<MT>;
  constexpr int TT = S::kTokens, U = S::kRounds;
  constexpr int kBPG = G / 32;                                     // blocks per group
  constexpr int kGroupsPerQuad = 4 / kBPG > 0 ? 4 / kBPG : 1;     // distinct groups of a quad
  constexpr int kMetaSize = META == kMetaZp ? 1 : META == kMetaMin ? 2 : 0;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int W = (int)blockDim.x >> 6;
  const int n0 = (int)blockIdx.x * 16;
  const int rows_here = N - n0 < 16 ? N - n0 : 16;
  const int nblk = K / 32, nq = (nblk + 3) / 4;
  const int Mc = M - token0 < TT ? M - token0 : TT;                // tokens of this launch
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t gpr = (uint32_t)(K / G);                          // groups per row
  uint16_t* const dsh = reinterpret_cast<uint16_t*>(lds);
  uint8_t* const slots = lds + (((size_t)nblk * TT * 2 + 15) & ~(size_t)15);
  uint8_t* const myslots = slots + (size_t)wave * U * S::kSlot;

  // Token scales of the launch, transposed to [block][token]; tokens past M read 0.
  // Thread b takes block b (the launch gives at least as many threads as blocks): its
  // TT loads go out together, then two (four) 16-byte LDS stores.
  // Tokens past M lie past the descriptor's range and read 0 (no branches, so the loads
  // go out together).
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(dx + (int64_t)token0 * nblk, (uint32_t)(Mc * nblk * 2));
  for (int b = (int)threadIdx.x; b < nblk; b += (int)blockDim.x) {
    uint32_t h[TT / 2];
#pragma unroll
    for (int t2 = 0; t2 < TT / 2; ++t2) {
      const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(rd, (2 * t2 * nblk + b) * 2, 0, 0);
      const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(rd, ((2 * t2 + 1) * nblk + b) * 2, 0, 0);
      h[t2] = lo | (hi << 16);
    }
#pragma unroll
    for (int v = 0; v < TT / 8; ++v)
      *reinterpret_cast<u32x4*>(dsh + b * TT + 8 * v) = u32x4{h[4 * v], h[4 * v + 1], h[4 * v + 2], h[4 * v + 3]};
  }
  __syncthreads();

  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes + (int64_t)n0 * row_bytes, (uint32_t)rows_here * row_bytes);
  // (base and range made explicitly wavefront-uniform: left alone, the compiler keeps
  // this descriptor in vector registers and wraps every load in a loop over lanes)
  const uint64_t xa0 = reinterpret_cast<uintptr_t>(qx + (int64_t)token0 * K);
  const uint64_t xa1 = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(xa0 >> 32)) << 32) |
                       (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)xa0);
  const __amdgpu_buffer_rsrc_t rx =
      make_rsrc(reinterpret_cast<const int8_t*>(xa1), (uint32_t)__builtin_amdgcn_readfirstlane(Mc * K));
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(scales + (int64_t)n0 * gpr, (uint32_t)rows_here * gpr * 2);
  const uint8_t* const mb = static_cast<const uint8_t*>(meta);
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(kMetaSize ? mb + (int64_t)n0 * gpr * kMetaSize : mb,
                                              kMetaSize ? (uint32_t)rows_here * gpr * kMetaSize : 0u);

  const int n = lane & 15, c = lane >> 4;          // B column (weight row) and k chunk
  // code DMA: lane l < 16q fetches 16 bytes, piece l % q of row l / q's quad
  const int dma_row = lane / Q, dma_piece = lane % Q;
  constexpr uint32_t kOff = kOutOfRange;

  float yacc[MT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) yacc[mt][r] = 0.0f;

  for (int i0 = 0; wave + W * i0 < nq; i0 += U) {                 // rounds (uniform)
    uint32_t xa[U][4][MT][2];      // activation bytes: lane (t = l%16, c): 8 bytes of block j, chunk c
    uint32_t sb[U][kGroupsPerQuad], zb[U][kGroupsPerQuad];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = wave + W * (i0 + u);
      const bool vq = s < nq;
      const uint32_t coff = vq && lane < 16 * Q ? (uint32_t)dma_row * row_bytes + (uint32_t)s * (16 * Q) + 16u * dma_piece
                                                : kOff;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (__attribute__((address_space(3))) void*)(myslots + u * S::kSlot), 16,
                                               coff, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int b = 4 * s + j;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const uint32_t xo = vq && b < nblk ? (uint32_t)(mt * 16 + n) * (uint32_t)K + 32u * b + 8u * c : kOff;
          const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rx, (int)xo, 0, 0);
          xa[u][j][mt][0] = v.x;
          xa[u][j][mt][1] = v.y;
        }
      }
#pragma unroll
      for (int gq = 0; gq < kGroupsPerQuad; ++gq) {
        const int b = 4 * s + gq * kBPG;
        const uint32_t gi = (uint32_t)n * gpr + (uint32_t)(b / kBPG);
        const bool ok = vq && b < nblk;
        sb[u][gq] = __builtin_amdgcn_raw_buffer_load_b16(rs, ok ? (int)(gi * 2) : (int)kOff, 0, 0);
        if constexpr (META == kMetaMin)
          zb[u][gq] = __builtin_amdgcn_raw_buffer_load_b16(rz, ok ? (int)(gi * 2) : (int)kOff, 0, 0);
        else if constexpr (META == kMetaZp)
          zb[u][gq] = __builtin_amdgcn_raw_buffer_load_b8(rz, ok ? (int)gi : (int)kOff, 0, 0);
        else
          zb[u][gq] = 0u;
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // every load of the round goes out before the wait
    wait_vmcnt<0>();                  // this round's loads, the direct-to-LDS codes included
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // Every quad slot of the round is multiplied, also those past the wavefront's last
    // quad (their operands read zeros): a branch here would let the compiler sink the
    // round's scale loads past the wait, into the multiply.
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = wave + W * (i0 + u);
      const uint8_t* const slot = myslots + u * S::kSlot + n * (16 * Q);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int b = 4 * s + j;
        const int gq = j / kBPG < kGroupsPerQuad ? j / kBPG : kGroupsPerQuad - 1;
        // this lane's 8 fields of block j: q bytes at byte q*c of the block
        uint32_t v;
        if constexpr (Q == 4) {
          v = *reinterpret_cast<const uint32_t*>(slot + 16 * j + 4 * c);
        } else if constexpr (Q == 2) {
          v = *reinterpret_cast<const uint16_t*>(slot + 8 * j + 2 * c);
        } else {
          const int byte = 12 * j + 3 * c;
          const uint32_t* const w32 = reinterpret_cast<const uint32_t*>(slot + (byte & ~3));
          v = __builtin_amdgcn_alignbit(w32[1], w32[0], 8 * (byte & 3));
        }
        const int64_t bq = code_bytes<Q>(v);
        int64_t bo;                   // the offset operand: bytes -o, -z[n, g] or ones
        if constexpr (META == kMetaMin) {
          bo = 0x0101010101010101ll;
        } else if constexpr (META == kMetaZp) {
          const uint32_t nz = __builtin_amdgcn_perm(0u, (0u - zb[u][gq]) & 0xFFu, 0x00000000u);
          bo = (int64_t)(((uint64_t)nz << 32) | nz);
        } else {
          constexpr uint32_t kNo = (0x100u - (1u << (Q - 1))) * 0x01010101u;
          bo = (int64_t)(((uint64_t)kNo << 32) | kNo);
        }
        const float sc = f16_bits_to_f32(sb[u][gq]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int64_t a = act_pair<Q>(xa[u][j][mt][0], xa[u][j][mt][1]);
          const i32x4 zero = {0, 0, 0, 0};
          i32x4 acc, accr;
          if constexpr (META == kMetaMin) {
            accr = __builtin_amdgcn_mfma_i32_16x16x32_i8(a, bo, zero, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x32_i8(a, bq, zero, 0, 0, 0);
          } else {
            acc = __builtin_amdgcn_mfma_i32_16x16x32_i8(a, bo, zero, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x32_i8(a, bq, acc, 0, 0, 0);
          }
          // token scales of tokens 16 mt + 4c .. +3 for block b
          const u32x2 dd = *reinterpret_cast<const u32x2*>(dsh + (b < nblk ? b : 0) * TT + mt * 16 + 4 * c);
          const uint32_t dpair[2] = {dd.x, dd.y};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float dsc = f16_bits_to_f32((dpair[r >> 1] >> (16 * (r & 1))) & 0xFFFFu);
            if constexpr (META == kMetaMin) {
              const float t = __builtin_fmaf(sc, (float)acc[r], f16_bits_to_f32(zb[u][gq]) * (float)accr[r]);
              yacc[mt][r] = __builtin_fmaf(dsc, t, yacc[mt][r]);
            } else {
              yacc[mt][r] = __builtin_fmaf(sc * dsc, (float)acc[r], yacc[mt][r]);
            }
          }
        }
      }
    }
  }
  // The wavefronts' partial sums, in wavefront order: part[w][t][n] over the idle slots
  // and staging (every wavefront is past its last LDS read after the barrier).
  __syncthreads();
  float* const part = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) part[(wave * TT + mt * 16 + 4 * c + r) * 16 + n] = yacc[mt][r];
  __syncthreads();
  for (int i = (int)threadIdx.x; i < Mc * 16; i += (int)blockDim.x) {
    const int t = i >> 4, nn = i & 15;
    if (nn >= rows_here) continue;
    float v = 0.0f;
    for (int w = 0; w < W; ++w) v += part[(w * TT + t) * 16 + nn];
    y[(int64_t)(token0 + t) * N + n0 + nn] = f32_to_bf16_bits(v);
  }
}

template <int Q, int G, int META, int MT>
hipError_t skinny_q8_launch(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, const void* meta, int64_t N, int64_t K, int64_t token0,
                            uint16_t* y, hipStream_t stream) {
  using S = SkinnyQ8<MT>;
  const int64_t nblk = K / 32, nq = (nblk + 3) / 4;
  const int waves = (int)std::min<int64_t>(kSkinnyMaxWaves, nq);
  const size_t stage = ((size_t)nblk * S::kTokens * 2 + 15) & ~(size_t)15;
  const size_t slots = (size_t)waves * S::kRounds * S::kSlot;
  const size_t part = (size_t)waves * S::kTokens * 16 * 4;
  const size_t lds = std::max(stage + slots, part);
  skinny_q8_kernel<Q, G, META, MT><<<dim3((unsigned)((N + 15) / 16)), (unsigned)(64 * waves), lds, stream>>>(
      qx, dx, (int)M, codes, scales, meta, (int)N, (int)K, (int)token0, y);
  return hipGetLastError();
}

// Tokens in launches of up to 32 (two 16-token tiles) or 16, each reading the weights once;
// the one-token kernel for M = 1 and for rows longer than the token-scale staging holds.
template <int Q, int G, int META>
hipError_t matmul_q8_dispatch(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                              const uint16_t* scales, const void* meta, int64_t N, int64_t K, uint16_t* y,
                              hipStream_t stream) {
  if (M == 1 || K > kSkinnyMaxK) return gemv_q8_dispatch<Q, G, META>(qx, dx, M, codes, scales, meta, N, K, y, stream);
  for (int64_t m0 = 0; m0 < M; m0 += 32) {
    const hipError_t e = M - m0 > 16
        ? skinny_q8_launch<Q, G, META, 2>(qx, dx, M, codes, scales, meta, N, K, m0, y, stream)
        : skinny_q8_launch<Q, G, META, 1>(qx, dx, M, codes, scales, meta, N, K, m0, y, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_quantize_act_q8(const uint16_t* x, int64_t M, int64_t K, int8_t* q, uint16_t* d,
                                  hipStream_t stream) {
  const int64_t total_chunks = M * K / 8;
  if (total_chunks == 0) return hipSuccess;
  const int64_t blocks = (total_chunks + kActThreads - 1) / kActThreads;
  quantize_act_q8_kernel<<<dim3((unsigned)blocks), kActThreads, 0, stream>>>(x, total_chunks,
                                                                              reinterpret_cast<uint2*>(q), d);
  return hipGetLastError();
}

hipError_t launch_matmul_q8(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K, int group, int q,
                            uint16_t* y, hipStream_t stream) {
  SSQ_DISPATCH_QGM(matmul_q8_dispatch, q, group, meta.kind, qx, dx, M, codes, scales, meta.ptr, N, K, y, stream);
}

}  // namespace ssq
