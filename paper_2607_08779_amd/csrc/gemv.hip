// Decode GEMV (M = 1) over packed few-bit weights, plus the binary32 matmul.
//
// App. B.3 of the paper: with W[n,k] ~ s[n,b] (u[n,k] - o[n,b]) in group b,
//   y[n] = sum_b s[n,b] * ( sum_{k in b} x[k] u[n,k]  -  o[n,b] sum_{k in b} x[k] ).
// The symmetric formats (signed or not -- the sign lives in s) have the
// constant offset o = 2^(q-1); the asymmetric one reads o from zp.  The Q*_1 layout
// of App. B.1 stores a minimum m instead (W ~ s*u + m), which contributes
// m * sum_{k in b} x[k] per block.
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

// q = 2 fields at mantissa bits 2-3 and 4-5 are OR-ed into the bf16 constants 32 and 8
// instead of 128: with exponent 134 - 2c the field at bits 2c..2c+1 adds exactly u, so
// the pair needs no shift.  The fields of a dword then fall into three offset classes
// c (base 128, 32 or 8) by their position j in the dword's 8 pairs.
constexpr uint32_t kMagicQ2[3] = {0x43004300u, 0x42004200u, 0x41004100u};
constexpr float kBaseQ2[3] = {128.0f, 32.0f, 8.0f};
constexpr int kClassQ2[8] = {0, 1, 2, 0, 0, 1, 2, 0};

// sum_{k in block} x[k] * (base(k) + u[k]) in fp32, base 128 except for q = 2 (above).
// `magic` holds kMagic (in a VGPR).
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
    // pair j of the dword holds fields (j, j + 8): bits 2j of each half-word
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const uint32_t w = b.d[d], w6 = w >> 6, w8 = w >> 8, w14 = w >> 14;
      acc = dot2(and_or(w, 0x00030003u, magic), xp[8 * d + 0], acc);
      acc = dot2(and_or(w, 0x000C000Cu, kMagicQ2[1]), xp[8 * d + 1], acc);
      acc = dot2(and_or(w, 0x00300030u, kMagicQ2[2]), xp[8 * d + 2], acc);
      acc = dot2(and_or(w6, 0x00030003u, magic), xp[8 * d + 3], acc);
      acc = dot2(and_or(w8, 0x00030003u, magic), xp[8 * d + 4], acc);
      acc = dot2(and_or(w8, 0x000C000Cu, kMagicQ2[1]), xp[8 * d + 5], acc);
      acc = dot2(and_or(w8, 0x00300030u, kMagicQ2[2]), xp[8 * d + 6], acc);
      acc = dot2(and_or(w14, 0x00030003u, magic), xp[8 * d + 7], acc);
    }
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

// y + (one block's term of a row sum), from acc = sum_k x_k (base_k + u_k) (block_dot),
// xs = sum_k x_k and xb = sum_k base_k x_k over the block, the block's scale bits and
// its zero point or minimum bits.
template <int Q, int META>
__device__ __forceinline__ float add_block_term(float y, float acc, float xs, float xb, uint32_t sbits,
                                                uint32_t zbits) {
  const float sc = f16_bits_to_f32(sbits);
  if constexpr (META == kMetaMin) {    // s * sum x u + m * sum x
    y = __builtin_fmaf(sc, acc - xb, y);
    return __builtin_fmaf(f16_bits_to_f32(zbits), xs, y);
  } else if constexpr (Q == 2) {
    const float o = META == kMetaZp ? (float)zbits : (float)(1 << (Q - 1));
    return __builtin_fmaf(sc, __builtin_fmaf(-o, xs, acc - xb), y);
  } else {
    const float off = META == kMetaZp ? kMagicValue + (float)zbits : kMagicValue + (float)(1 << (Q - 1));
    return __builtin_fmaf(sc, __builtin_fmaf(-off, xs, acc), y);
  }
}

// The block sums xs and xb of one block's activations, and its pairs permuted for
// block_dot (q = 2 pairs carry three bases, the others base 128 throughout).
template <int Q>
__device__ __forceinline__ void block_x(const uint32_t (&X)[16], uint32_t (&xp)[16], float& xs, float& xb) {
  permute_x<Q>(X, xp);
  if constexpr (Q == 2) {
    float cs[3] = {0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < 16; ++i) cs[kClassQ2[i & 7]] = dot2(xp[i], kOnes, cs[kClassQ2[i & 7]]);
    xs = cs[0] + cs[1] + cs[2];
    xb = __builtin_fmaf(kBaseQ2[2], cs[2], __builtin_fmaf(kBaseQ2[1], cs[1], kBaseQ2[0] * cs[0]));
  } else {
    xs = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) xs = dot2(X[i], kOnes, xs);
    xb = kMagicValue * xs;
  }
}

// The 16 bf16 code pairs of a block in the order block_dot multiplies them (for
// several tokens the pairs are formed once and dotted with each token's activations).
template <int Q>
__device__ __forceinline__ void block_pairs(const Block<Q>& b, uint32_t magic, uint32_t (&w)[16]) {
  if constexpr (Q == 4) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t w4 = b.d[d] >> 4;
      w[4 * d] = and_or(b.d[d], 0x000F000Fu, magic);
      w[4 * d + 1] = and_or(w4, 0x000F000Fu, magic);
      w[4 * d + 2] = and_or(b.d[d] >> 8, 0x000F000Fu, magic);
      w[4 * d + 3] = and_or(w4 >> 8, 0x000F000Fu, magic);
    }
  } else if constexpr (Q == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const uint32_t v = b.d[d], v6 = v >> 6, v8 = v >> 8, v14 = v >> 14;
      w[8 * d + 0] = and_or(v, 0x00030003u, magic);
      w[8 * d + 1] = and_or(v, 0x000C000Cu, kMagicQ2[1]);
      w[8 * d + 2] = and_or(v, 0x00300030u, kMagicQ2[2]);
      w[8 * d + 3] = and_or(v6, 0x00030003u, magic);
      w[8 * d + 4] = and_or(v8, 0x00030003u, magic);
      w[8 * d + 5] = and_or(v8, 0x000C000Cu, kMagicQ2[1]);
      w[8 * d + 6] = and_or(v8, 0x00300030u, kMagicQ2[2]);
      w[8 * d + 7] = and_or(v14, 0x00030003u, magic);
    }
  } else {
    const uint32_t v[4] = {b.d[0], __builtin_amdgcn_alignbit(b.d[1], b.d[0], 24),
                           __builtin_amdgcn_alignbit(b.d[2], b.d[1], 16), b.d[2] >> 8};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t sp = (v[i] & 0xFFFu) | ((v[i] << 4) & 0x0FFF0000u);
#pragma unroll
      for (int j = 0; j < 4; ++j) w[4 * i + j] = and_or(sp >> (3 * j), 0x00070007u, magic);
    }
  }
}

// Work split.  A workgroup of T threads (T a whole number of wavefronts, at most 512)
// owns kRows consecutive rows; wavefront w takes 64 consecutive blocks of each row per
// pass (lane i block 64w + i), and passes repeat T blocks further on until the row
// ends.  Partial sums meet through a DPP wavefront reduction and LDS.  Every wavefront
// of the grid is resident at once for the decode shapes, so the whole matrix is in
// flight from the start; per-wavefront set-up is kept to a few scalar instructions,
// because the CU's one scalar unit serves all of its wavefronts as they start.
//
// Operand movement.  The codes are loaded one block per lane (4q contiguous bytes,
// lanes contiguous).  A lane also needs its block's 64 bytes of activations and one
// scale per row, but loading those per lane would stride the activation loads by 64
// bytes and spend a load instruction per row on two-byte scales.  Instead the
// wavefront loads its 4 KB activation span with four fully contiguous 1 KB loads and
// its kRows rows of scales (and zero points) with a single load, writes them to a
// wavefront-private LDS area and reads back what each lane needs.  The activation
// chunks are stored swizzled so that both the stores and the 64-byte-strided reads
// hit distinct LDS banks.  The single scale load needs the rows' scale runs 16-byte
// aligned; otherwise (VS = false) every lane loads its scale per row directly.
//
// One buffer descriptor covers the workgroup's live rows of codes (scales, zero
// points) and one the activations; loads past a descriptor's range return zeros.
// Lanes past the end of a row point their loads out of range, so rows and blocks
// beyond the matrix contribute exact zeros.
constexpr int kRows = 4;          // rows per workgroup (the folded reduction assumes four)
constexpr int kMaxTeam = 512;
constexpr int kMaxWaves = kMaxTeam / 64;
constexpr int kXChunks = 256;    // 16-byte activation chunks of one pass: 64 blocks x 64 bytes
constexpr uint32_t kOutOfRange = 0x80000000u;

template <int G, int META>
struct Stage {
  static constexpr int kBlocksPerGroup = G / 32;
  static constexpr int kScaleBytes = 128 / kBlocksPerGroup;   // one row's scales for 64 blocks
  static constexpr int kMetaSize = META == kMetaZp ? 1 : META == kMetaMin ? 2 : 0;  // bytes per group
  static constexpr int kZpBytes = 64 / kBlocksPerGroup * kMetaSize;    // one row's metadata
  static constexpr int kScaleChunks = kRows * kScaleBytes / 16;
  static constexpr int kZpChunks = kRows * kZpBytes / 16;
  static constexpr int kWaveChunks = kXChunks + kScaleChunks + kZpChunks;
  static constexpr int kWaveBytes = kWaveChunks * 16;
  static_assert(kScaleChunks <= 64 && kZpChunks <= 64, "one load instruction per wavefront");
};

// LDS chunk holding piece p (16 bytes) of block b of a pass.
__device__ __forceinline__ int x_slot(int b, int p) { return 4 * b + (p ^ ((b >> 2) & 3)); }

// Four wavefront sums at once: swapping lane halves (32 apart, then 16 apart) folds the
// four values of a lane into one, leaving in 16-lane row R the partials of value
// fold4_row(16 R); four DPP steps then finish each 16-lane row, whose lane 0 (lane 16R)
// holds the sum.
__device__ __forceinline__ float fold4_sum(float v0, float v1, float v2, float v3) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0), __float_as_uint(v1), false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v2), __float_as_uint(v3), false, false);
  const float s01 = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const float s23 = __uint_as_float(b[0]) + __uint_as_float(b[1]);
  const auto c = __builtin_amdgcn_permlane16_swap(__float_as_uint(s01), __float_as_uint(s23), false, false);
  float v = __uint_as_float(c[0]) + __uint_as_float(c[1]);
  v = dpp_add<0xB1, 0xF>(v);    // quad_perm [1,0,3,2]
  v = dpp_add<0x4E, 0xF>(v);    // quad_perm [2,3,0,1]
  v = dpp_add<0x141, 0xF>(v);   // row_half_mirror
  v = dpp_add<0x140, 0xF>(v);   // row_mirror
  return v;
}
__device__ __forceinline__ int fold4_row(int lane) { return ((lane >> 4) & 1) * 2 + (lane >> 5); }

// Orders LDS stores of some lanes before loads of others within one wavefront.
__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// T tokens (1 or 2) share each unpacked block; token t's activations start at x + t*K
// and its outputs at y + t*N.
template <int Q, int G, int META, bool VS, int T = 1>
__global__ __launch_bounds__(kMaxTeam) void gemv_kernel(const uint16_t* __restrict__ x,
                                                        const uint8_t* __restrict__ codes,
                                                        const uint16_t* __restrict__ scales,
                                                        const void* __restrict__ meta, int N, int K,
                                                        uint16_t* __restrict__ y, int threads) {
  using S = Stage<G, META>;
  constexpr bool ZP = META != kMetaNone;                   // any per-group metadata
  constexpr int kMetaSize = S::kMetaSize;
  const uint8_t* const zp = static_cast<const uint8_t*>(meta);
  constexpr int kBlocksPerGroup = S::kBlocksPerGroup;
  __shared__ float partial[kMaxWaves][kRows * T];
  extern __shared__ u32x4 stage[];
  constexpr int kWaveChunks = T * kXChunks + S::kScaleChunks + S::kZpChunks;

  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int row0 = (int)blockIdx.x * kRows;
  const int rows_here = N - row0 < kRows ? N - row0 : kRows;   // >= 1
  const int nblk = K / 32;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)K / G;
  const uint32_t magic = kMagic;
  u32x4* const xw = stage + wave * kWaveChunks;
  const uint8_t* const sw = reinterpret_cast<const uint8_t*>(xw + T * kXChunks);
  const uint8_t* const zw = sw + S::kScaleChunks * 16;

  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes + (int64_t)row0 * row_bytes, (uint32_t)rows_here * row_bytes);
  const __amdgpu_buffer_rsrc_t rs =
      make_rsrc(scales + (int64_t)row0 * groups_per_row, (uint32_t)rows_here * groups_per_row * 2);
  const __amdgpu_buffer_rsrc_t rz =
      make_rsrc(ZP ? zp + (int64_t)row0 * groups_per_row * kMetaSize : zp,
                ZP ? (uint32_t)rows_here * groups_per_row * kMetaSize : 0u);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)T * K * 2);

  float yacc[T][kRows];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int r = 0; r < kRows; ++r) yacc[t][r] = 0.0f;

  auto consume = [&](const uint32_t (&X)[T][16], const Block<Q> (&cb)[kRows], const uint32_t (&sbits)[kRows],
                     const uint32_t (&zbits)[kRows]) {
    uint32_t xp[T][16];
    // xs: sum of the block's activations; xb: sum of base(k) x[k], the constant part of
    // block_dot (128 xs except for q = 2, whose pairs carry three bases)
    float xs[T], xb[T];
#pragma unroll
    for (int t = 0; t < T; ++t) block_x<Q>(X[t], xp[t], xs[t], xb[t]);
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      float acc[T];
      if constexpr (T == 1) {
        acc[0] = block_dot<Q>(cb[r], xp[0], magic);
      } else {
        uint32_t w[16];
        block_pairs<Q>(cb[r], magic, w);
#pragma unroll
        for (int t = 0; t < T; ++t) {
          acc[t] = 0.0f;
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[t] = dot2(w[i], xp[t][i], acc[t]);
        }
      }
#pragma unroll
      for (int t = 0; t < T; ++t) yacc[t][r] = add_block_term<Q, META>(yacc[t][r], acc[t], xs[t], xb[t], sbits[r], zbits[r]);
    }
  };

  // Passes are uniform across the wavefront.
  for (int jw = wave * 64; jw < nblk; jw += threads) {
    const int j = jw + lane;
    const bool live = j < nblk;
    // Loads first: activations, scales (and zero points), then the codes of each row.
    u32x4 xq[T][4];
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        xq[t][i] = __builtin_amdgcn_raw_buffer_load_b128(rx, t * K * 2 + jw * 64 + 1024 * i + 16 * lane, 0, 0);
    u32x4 sq = {0, 0, 0, 0}, zq = {0, 0, 0, 0};
    uint32_t sbits[kRows], zbits[kRows];
    if constexpr (VS) {
      constexpr int kPer = S::kScaleBytes / 16;   // chunks per row
      const uint32_t in_row = (uint32_t)(jw / kBlocksPerGroup) * 2 + 16 * (lane % kPer);
      const uint32_t off = in_row < groups_per_row * 2 ? (lane / kPer) * groups_per_row * 2 + in_row : kOutOfRange;
      if (lane < S::kScaleChunks) sq = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
      if constexpr (ZP) {
        constexpr int kZPer = S::kZpBytes / 16;
        const uint32_t zin = (uint32_t)(jw / kBlocksPerGroup) * kMetaSize + 16 * (lane % kZPer);
        const uint32_t zoff = zin < groups_per_row * kMetaSize
                                  ? (lane / kZPer) * groups_per_row * kMetaSize + zin : kOutOfRange;
        if (lane < S::kZpChunks) zq = __builtin_amdgcn_raw_buffer_load_b128(rz, zoff, 0, 0);
      }
    } else {
      const uint32_t goff = (uint32_t)(j / kBlocksPerGroup);
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        sbits[r] = __builtin_amdgcn_raw_buffer_load_b16(rs, live ? (r * groups_per_row + goff) * 2 : kOutOfRange, 0, 0);
        if constexpr (META == kMetaMin)
          zbits[r] = __builtin_amdgcn_raw_buffer_load_b16(rz, live ? (r * groups_per_row + goff) * 2 : kOutOfRange, 0, 0);
        else
          zbits[r] = ZP ? __builtin_amdgcn_raw_buffer_load_b8(rz, live ? r * groups_per_row + goff : kOutOfRange, 0, 0) : 0u;
      }
    }
    Block<Q> cb[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r)
      buffer_block_codes<Q>(rc, live ? r * row_bytes + (uint32_t)j * (4 * Q) : kOutOfRange, 0, cb[r].d);

    // Through LDS: chunk c = 64 i + lane of the pass is piece c % 4 of block c / 4.
    wave_sync_lds();   // the previous pass's reads are done
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) xw[t * kXChunks + x_slot(16 * i + (lane >> 2), lane & 3)] = xq[t][i];
    if constexpr (VS) {
      if (lane < S::kScaleChunks) xw[T * kXChunks + lane] = sq;
      if constexpr (ZP) if (lane < S::kZpChunks) xw[T * kXChunks + S::kScaleChunks + lane] = zq;
    }
    wave_sync_lds();
    uint32_t X[T][16];
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const u32x4 v = xw[t * kXChunks + x_slot(lane, p)];
        X[t][4 * p] = v.x; X[t][4 * p + 1] = v.y; X[t][4 * p + 2] = v.z; X[t][4 * p + 3] = v.w;
      }
    if constexpr (VS) {
      const int g = lane / kBlocksPerGroup;
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        sbits[r] = *reinterpret_cast<const uint16_t*>(sw + r * S::kScaleBytes + 2 * g);
        if constexpr (META == kMetaMin)
          zbits[r] = *reinterpret_cast<const uint16_t*>(zw + r * S::kZpBytes + 2 * g);
        else
          zbits[r] = ZP ? zw[r * S::kZpBytes + g] : 0u;
      }
    }
    consume(X, cb, sbits, zbits);
  }
  static_assert(kRows == 4, "the folded reduction handles four rows");
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const float v = fold4_sum(yacc[t][0], yacc[t][1], yacc[t][2], yacc[t][3]);
    if ((lane & 15) == 0) partial[wave][t * kRows + fold4_row(lane)] = v;
  }
  __syncthreads();
  if constexpr (T == 1) {
    if ((int)threadIdx.x < rows_here) {
      const int waves = threads >> 6;
      float v = 0.0f;
      for (int w = 0; w < waves; ++w) v += partial[w][threadIdx.x];
      y[row0 + threadIdx.x] = f32_to_bf16_bits(v);
    }
  } else if ((int)threadIdx.x < kRows * T) {
    const int t = (int)threadIdx.x / kRows, r = (int)threadIdx.x % kRows;
    if (r < rows_here) {
      const int waves = threads >> 6;
      float v = 0.0f;
      for (int w = 0; w < waves; ++w) v += partial[w][t * kRows + r];
      y[(int64_t)t * N + row0 + r] = f32_to_bf16_bits(v);
    }
  }
}

// ---------------------------------------------------------------------------
// Activation-stationary decode GEMV (M = 1, K <= 16 x 2048), for matrices with many
// rows per resident workgroup.
//
// The workgroup has C = ceil(K / 2048) wavefronts; wavefront w owns blocks 64w..64w+63
// of every row (lane i: block 64w + i).  It loads its 4 KB of activations once (four
// contiguous 1 KB loads, redistributed through LDS), forms their pairs and block sums
// once, and keeps them in registers while the workgroup walks a run of PER 4-row
// groups.  The codes, scales (and zero points or minimums) of group i+1 are in flight
// while group i is multiplied.  After a group the wavefront folds its four rows' lane
// partials into four sums and parks them in LDS; when the run is done the workgroup
// adds the C wavefronts' sums of each row in wavefront order and stores y.  Per
// 32-weight block and row a lane spends the unpack and 16 dot2 of block_dot plus the
// scale step; the per-pass activation work of the pass-looping kernel (its LDS round
// trip, pair permutation and block sums, and its re-read of x for every 4 rows) is
// paid once per run of up to 32 rows.
// ---------------------------------------------------------------------------

constexpr int kStatMaxWaves = 16;      // K <= 16 x 64 blocks
constexpr int kStatMaxGroups = 8;      // 4-row groups per workgroup
constexpr int kCUs = 256;              // MI355X compute units
// Two groups in registers (69 VGPRs at q = 4: seven wavefronts per SIMD), and the grid
// sized for 28 resident wavefronts per CU.  Deeper rings (three or four groups) were
// measured slower: the registers they take cost more wavefronts than they add loads.
constexpr int kStatDepth = 2;
constexpr int kStatWavesPerCU = 28;

template <int Q>
struct StatGroup {
  Block<Q> cb[kRows];
  uint32_t s[kRows];
  uint32_t z[kRows];
};

// A lane's load offsets for its block j in the four rows of a group, the same for every
// group (each group gets descriptors of its own, see stat_rsrc); past the row's blocks
// they point out of range.
struct StatOffsets {
  uint32_t c[kRows], s[kRows], z[kRows];
};

template <int Q, int G, int META>
__device__ __forceinline__ StatOffsets stat_offsets(bool live, int j, uint32_t row_bytes, uint32_t groups_per_row) {
  constexpr int kMetaSize = META == kMetaZp ? 1 : META == kMetaMin ? 2 : 0;
  const uint32_t g = (uint32_t)(j / (G / 32));
  StatOffsets o;
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    o.c[r] = live ? (uint32_t)r * row_bytes + (uint32_t)j * (4 * Q) : kOutOfRange;
    o.s[r] = live ? ((uint32_t)r * groups_per_row + g) * 2 : kOutOfRange;
    o.z[r] = live ? ((uint32_t)r * groups_per_row + g) * kMetaSize : kOutOfRange;
  }
  return o;
}

// Descriptor over rows 4i.. of the workgroup's run (rows_here rows from `base`, `stride`
// bytes each): scalar arithmetic only; groups past the run get an empty range.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t stat_rsrc(const void* base, uint32_t stride, int i, int rows_here) {
  const int left = rows_here - 4 * i;
  return make_rsrc(static_cast<const uint8_t*>(base) + (int64_t)(4 * i) * stride, left > 0 ? (uint32_t)left * stride : 0u);
}

// Loads of row group i of the workgroup's run (rows 4i..4i+3).
template <int Q, int G, int META>
__device__ __forceinline__ void stat_issue(StatGroup<Q>& st, int i, const StatOffsets& o, int rows_here,
                                           uint32_t row_bytes, uint32_t groups_per_row, const uint8_t* cbase,
                                           const uint16_t* sbase, const uint8_t* zbase) {
  constexpr int kMetaSize = META == kMetaZp ? 1 : META == kMetaMin ? 2 : 0;
  const __amdgpu_buffer_rsrc_t rc = stat_rsrc(cbase, row_bytes, i, rows_here);
  const __amdgpu_buffer_rsrc_t rs = stat_rsrc(sbase, groups_per_row * 2, i, rows_here);
  const __amdgpu_buffer_rsrc_t rz = stat_rsrc(zbase, kMetaSize ? groups_per_row * kMetaSize : 0u, i,
                                              kMetaSize ? rows_here : 0);
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    buffer_block_codes<Q>(rc, o.c[r], 0, st.cb[r].d);
    st.s[r] = __builtin_amdgcn_raw_buffer_load_b16(rs, o.s[r], 0, 0);
    if constexpr (META == kMetaMin)
      st.z[r] = __builtin_amdgcn_raw_buffer_load_b16(rz, o.z[r], 0, 0);
    else if constexpr (META == kMetaZp)
      st.z[r] = __builtin_amdgcn_raw_buffer_load_b8(rz, o.z[r], 0, 0);
    else
      st.z[r] = 0u;
  }
}

template <int Q, int META>
__device__ __forceinline__ float stat_rows(const StatGroup<Q>& st, const uint32_t (&xp)[16], float xs, float xb,
                                           uint32_t magic) {
  float v[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r)
    v[r] = add_block_term<Q, META>(0.0f, block_dot<Q>(st.cb[r], xp, magic), xs, xb, st.s[r], st.z[r]);
  return fold4_sum(v[0], v[1], v[2], v[3]);
}

template <int Q, int G, int META, int D, int PER>
__global__ __launch_bounds__(1024) void gemv_stat_kernel(const uint16_t* __restrict__ x,
                                                         const uint8_t* __restrict__ codes,
                                                         const uint16_t* __restrict__ scales,
                                                         const void* __restrict__ meta, int N, int K,
                                                         int groups_per_wg, uint16_t* __restrict__ y) {
  static_assert(PER <= kStatMaxGroups && D >= 2, "run length and ring depth");
  constexpr int kMetaSize = META == kMetaZp ? 1 : META == kMetaMin ? 2 : 0;
  __shared__ float part[kStatMaxGroups][kStatMaxWaves][kRows];
  const uint8_t* const zp = static_cast<const uint8_t*>(meta);

  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int waves = (int)blockDim.x >> 6;
  const int nblk = K / 32;
  const int j = wave * 64 + lane;
  const bool live = j < nblk;
  const int g0 = (int)blockIdx.x * groups_per_wg;
  const int groups_total = (N + kRows - 1) / kRows;
  const int ng = groups_total - g0 < groups_per_wg ? groups_total - g0 : groups_per_wg;   // >= 1
  const int row0 = g0 * kRows;
  const int rows_here = N - row0 < ng * kRows ? N - row0 : ng * kRows;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)K / G;
  const uint32_t magic = kMagic;

  // the run's operands; each group's loads go through descriptors over its own rows, so
  // rows past N and blocks past the row read as zeros and the offsets stay constant
  const uint8_t* const cbase = codes + (int64_t)row0 * row_bytes;
  const uint16_t* const sbase = scales + (int64_t)row0 * groups_per_row;
  const uint8_t* const zbase = kMetaSize ? zp + (int64_t)row0 * groups_per_row * kMetaSize : zp;
  const StatOffsets off = stat_offsets<Q, G, META>(live, j, row_bytes, groups_per_row);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)K * 2);

  // The wavefront's 4 KB of activations: four contiguous 1 KB loads, then through a
  // wavefront-private LDS area to the lane that owns each block (chunk c = 64 i + lane is
  // piece c % 4 of block c / 4; chunks past K read zeros).
  extern __shared__ u32x4 xstage[];
  u32x4* const xw = xstage + wave * kXChunks;
  u32x4 xq[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    xq[i] = __builtin_amdgcn_raw_buffer_load_b128(rx, wave * 4096 + 1024 * i + 16 * lane, 0, 0);
  // A ring of D groups in registers: while group i is multiplied, groups i+1..i+D-1
  // are in flight.  The run is unrolled at compile time (PER groups, groups past the
  // workgroup's ng read zeros without touching memory: their rows lie past the
  // descriptors), so every wait is for exactly the group about to be consumed; a loop
  // or a data-dependent branch would make the compiler drain every load in flight.
  StatGroup<Q> st[D];
#pragma unroll
  for (int d = 0; d < D - 1 && d < PER; ++d)
    stat_issue<Q, G, META>(st[d], d, off, rows_here, row_bytes, groups_per_row, cbase, sbase, zbase);
#pragma unroll
  for (int i = 0; i < 4; ++i) xw[x_slot(16 * i + (lane >> 2), lane & 3)] = xq[i];
  wave_sync_lds();
  uint32_t X[16];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const u32x4 v = xw[x_slot(lane, p)];
    X[4 * p] = v.x; X[4 * p + 1] = v.y; X[4 * p + 2] = v.z; X[4 * p + 3] = v.w;
  }
  uint32_t xp[16];
  float xs, xb;
  block_x<Q>(X, xp, xs, xb);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (i + D - 1 < PER)
      stat_issue<Q, G, META>(st[(i + D - 1) % D], i + D - 1, off, rows_here, row_bytes, groups_per_row, cbase,
                             sbase, zbase);
    const float v = stat_rows<Q, META>(st[i % D], xp, xs, xb, magic);
    if (i < ng && (lane & 15) == 0) part[i][wave][fold4_row(lane)] = v;
  }
  __syncthreads();
  for (int t = (int)threadIdx.x; t < rows_here; t += (int)blockDim.x) {
    float v = 0.0f;
    for (int w = 0; w < waves; ++w) v += part[t / kRows][w][t % kRows];
    y[row0 + t] = f32_to_bf16_bits(v);
  }
}

template <int Q, int G, int META, int PER>
void gemv_stat_launch(const uint16_t* x, const uint8_t* codes, const uint16_t* scales, const void* meta,
                      int64_t N, int64_t K, uint16_t* y, hipStream_t stream) {
  const int64_t waves = (K / 32 + 63) / 64;
  const int64_t groups = (N + kRows - 1) / kRows;
  const dim3 grid((unsigned)((groups + PER - 1) / PER));
  gemv_stat_kernel<Q, G, META, kStatDepth, PER><<<grid, (unsigned)(64 * waves), (size_t)waves * kXChunks * 16, stream>>>(
      x, codes, scales, meta, (int)N, (int)K, PER, y);
}

// Runs of PER = 4 or 8 row groups per workgroup: 4 while that fits the matrix into one
// round of resident workgroups, else 8.  Returns false (nothing launched) for matrices
// that one round covers with runs of two groups or fewer: there every wavefront of the
// pass-looping kernel has its loads in flight from the start, and that kernel measured
// faster (its activation work per row is higher, but it runs twice the wavefronts).
template <int Q, int G, int META>
bool gemv_stat_dispatch(const uint16_t* x, const uint8_t* codes, const uint16_t* scales, const void* meta,
                        int64_t N, int64_t K, uint16_t* y, hipStream_t stream) {
  const int64_t waves = (K / 32 + 63) / 64;
  if (waves > kStatMaxWaves) return false;
  const int64_t groups = (N + kRows - 1) / kRows;
  const int64_t slots = kCUs * std::max<int64_t>(1, kStatWavesPerCU / waves);
  if (groups <= 2 * slots) return false;
  if (groups <= 4 * slots) gemv_stat_launch<Q, G, META, 4>(x, codes, scales, meta, N, K, y, stream);
  else gemv_stat_launch<Q, G, META, 8>(x, codes, scales, meta, N, K, y, stream);
  return true;
}

// ---------------------------------------------------------------------------
// Binary32 matmul: x[M,K] fp32, y[M,N] fp32.  One wavefront per (row n, 4 tokens);
// each lane dequantizes whole 32-weight blocks exactly in fp32.
// ---------------------------------------------------------------------------

constexpr int kF32Tokens = 4;

template <int Q, int G, int META>
__global__ __launch_bounds__(256) void matmul_f32_kernel(const float* __restrict__ x, int M,
                                                         const uint8_t* __restrict__ codes,
                                                         const uint16_t* __restrict__ scales,
                                                         const void* __restrict__ meta, int N,
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
    // weight = s*u - s*o, or s*u + m for the minimum layout
    const float so = META == kMetaMin ? f16_bits_to_f32(static_cast<const uint16_t*>(meta)[gi])
                   : META == kMetaZp ? -s * (float)static_cast<const uint8_t*>(meta)[gi]
                                     : -s * (float)(1 << (Q - 1));
    float w[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) w[k] = __builtin_fmaf(s, (float)field<Q>(b.d, k), so);
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

template <int Q, int G, int META, int T = 1>
hipError_t gemv_dispatch(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                         const void* meta, int64_t N, int64_t K, uint16_t* y, hipStream_t stream) {
  using S = Stage<G, META>;
  const int64_t nblk = K / 32;
  const int64_t passes = (nblk + kMaxTeam - 1) / kMaxTeam;
  const int threads = (int)(((nblk + passes - 1) / passes + 63) / 64 * 64);
  const dim3 grid((unsigned)((N + kRows - 1) / kRows));
  const size_t lds = (size_t)(threads / 64) * (T * kXChunks + S::kScaleChunks + S::kZpChunks) * 16;
  // One load per wavefront covers the rows' scales (and zero points or minimums) when
  // every row's run of them starts 16-byte aligned.
  const int64_t groups = K / G;
  const bool vs = reinterpret_cast<uintptr_t>(scales) % 16 == 0 && (groups * 2) % 16 == 0 &&
                  (S::kMetaSize == 0 ||
                   (reinterpret_cast<uintptr_t>(meta) % 16 == 0 && (groups * S::kMetaSize) % 16 == 0));
  if (vs)
    gemv_kernel<Q, G, META, true, T><<<grid, threads, lds, stream>>>(x, codes, scales, meta, (int)N, (int)K, y,
                                                                     threads);
  else
    gemv_kernel<Q, G, META, false, T><<<grid, threads, lds, stream>>>(x, codes, scales, meta, (int)N, (int)K, y,
                                                                      threads);
  return hipGetLastError();
}

template <int Q, int G, int META>
hipError_t f32_dispatch(const float* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                        const void* meta, int64_t N, int64_t K, float* y, hipStream_t stream) {
  const dim3 grid((unsigned)((N + 3) / 4), (unsigned)((M + kF32Tokens - 1) / kF32Tokens));
  matmul_f32_kernel<Q, G, META><<<grid, 256, 0, stream>>>(x, (int)M, codes, scales, meta, (int)N, (int)K, y);
  return hipGetLastError();
}

// One token: the activation-stationary kernel where it applies (gemv_stat_dispatch),
// else the pass-looping kernel.
template <int Q, int G, int META>
hipError_t gemv1_dispatch(const uint16_t* x, const uint8_t* codes, const uint16_t* scales, const void* meta,
                          int64_t N, int64_t K, uint16_t* y, hipStream_t stream) {
  if (gemv_stat_dispatch<Q, G, META>(x, codes, scales, meta, N, K, y, stream)) return hipGetLastError();
  return gemv_dispatch<Q, G, META>(x, codes, scales, meta, N, K, y, stream);
}

}  // namespace

hipError_t launch_gemv_bf16(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                            GroupMeta meta, int64_t N, int64_t K, int group, int q, uint16_t* y,
                            hipStream_t stream) {
  SSQ_DISPATCH_QGM(gemv1_dispatch, q, group, meta.kind, x, codes, scales, meta.ptr, N, K, y, stream);
}

// Two tokens through one pass over the weights (M = 2).
template <int Q, int G, int META>
hipError_t gemv2_dispatch(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                          const void* meta, int64_t N, int64_t K, uint16_t* y, hipStream_t stream) {
  return gemv_dispatch<Q, G, META, 2>(x, codes, scales, meta, N, K, y, stream);
}

hipError_t launch_gemv2_bf16(const uint16_t* x, const uint8_t* codes, const uint16_t* scales,
                             GroupMeta meta, int64_t N, int64_t K, int group, int q, uint16_t* y,
                             hipStream_t stream) {
  SSQ_DISPATCH_QGM(gemv2_dispatch, q, group, meta.kind, x, codes, scales, meta.ptr, N, K, y, stream);
}

hipError_t launch_matmul_f32(const float* x, int64_t M, const uint8_t* codes,
                             const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K,
                             int group, int q, float* y, hipStream_t stream) {
  SSQ_DISPATCH_QGM(f32_dispatch, q, group, meta.kind, x, M, codes, scales, meta.ptr, N, K, y, stream);
}

}  // namespace ssq
