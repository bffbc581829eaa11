// Skinny-M matmul (batched decode, 2 <= M <= 32): y[M,N] = x[M,K] * What[N,K]^T.
//
// App. B.3 of the paper: What[n,k] = s[n,b] (u[n,k] - o[n,b]).  With a handful of
// tokens the product is bound by streaming the packed weights, as the GEMV is, but a
// per-token dot product would repeat the unpacking M times.  Here every weight is
// dequantized once (s*(u - o), exact in fp32, rounded to bf16) straight into the B
// operand of v_mfma_f32_16x16x32_bf16, and the tokens share it through the matrix
// cores: one MFMA per 16 tokens per 512 weights.  Nothing is staged in LDS except
// the final cross-wavefront sums.
//
// A workgroup owns 16 consecutive weight rows and the whole reduction; its
// wavefronts split K into contiguous ranges of 128-wide super-blocks.  For the MFMA,
// lane l works on weight row l % 16 and on the super-block's 32-weight block l / 16,
// and holds the 32 activations of token l % 16 at the same k.  The super-block's
// four MFMAs take chunk t (8 k values) of each lane's block.  The MFMA reduces over
// whatever k each lane supplies, so operands that agree on the assignment give the
// exact product.
//
// Loads do not use that layout: lane L reads row (or token) L / 4, piece L % 4, so
// four neighbouring lanes cover one contiguous 64-byte span and the texture unit
// serves a quad per access (with one row per lane it serves one lane per cycle, which
// halves throughput).  A ds_bpermute per dword then moves each value to its MFMA lane,
// and for the activations a 4x4 transpose across the four 16-lane rows
// (v_permlane32_swap / v_permlane16_swap) turns "chunk c of block j" into "chunk j of
// block c".
#include <algorithm>

#include "mfma_dequant.h"
#include "ssq_internal.h"

namespace ssq {
namespace {

constexpr int kMaxWaves = 16;
constexpr uint32_t kOutOfRange = 0x80000000u;   // past every buffer's size: loads return 0

template <int Q, int G, int META, int MB>
__global__ __launch_bounds__(1024) void skinny_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const void* __restrict__ meta, int M, int N, int K, uint16_t* __restrict__ y) {
  __shared__ float red[kMaxWaves][MB * 256];   // per wave: its partial D tiles, lane order

  const int tid = threadIdx.x, lane = tid & 63;
  // wave-uniform (scalar) so the super-block loop and its range tests stay in SGPRs and
  // out-of-range loads are chosen by a scalar select, not by branching around them
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int waves = (int)(blockDim.x >> 6);
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int nblk = K / 32, nsb = (nblk + 3) / 4;
  const int per = (nsb + waves - 1) / waves;
  const int sb_begin = std::min(nsb, wave * per);
  const int sb_end = std::min(nsb, sb_begin + per);
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)(K / G);

  // Descriptors over this workgroup's rows (rows past N read zeros) and over x (tokens
  // past M read zeros; M*K*2 < 2^28 for M <= 32).
  const uint32_t rows = (uint32_t)std::min<int64_t>(16, N - n0);
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes + n0 * row_bytes, rows * row_bytes);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(scales + n0 * groups_per_row, rows * groups_per_row * 2);
  constexpr bool ZP = META != kMetaNone;
  constexpr int kMetaSize = meta_size<META>();
  const uint8_t* const zp = static_cast<const uint8_t*>(meta);
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(ZP ? zp + n0 * groups_per_row * kMetaSize : zp,
                                              ZP ? rows * groups_per_row * kMetaSize : 0);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)M * (uint32_t)K * 2);

  struct Slot {
    uint32_t d[Part<Q, 1>::kDwords];
    uint32_t s, z;
    u32x4 a[MB][4];
  };
  // Loads of super-block sb; a slot past this wave's range issues the same loads out of
  // range (they return zeros and move no data), so every iteration waits on a fixed count.
  // load layout: lane -> (row lrow, piece lpiece); MFMA layout: lane l takes the value
  // loaded by lane 4*(l%16) + l/16 (byte address `perm` for ds_bpermute)
  const int lrow = lane >> 2, lpiece = lane & 3;
  const int perm = (4 * (lane & 15) + (lane >> 4)) * 4;
  auto load = [&](int sb, bool valid, Slot& t) {
    const int blk = 4 * sb + lpiece;
    const bool in = valid & (blk < nblk);
    load_part<Q, 1>(rc, in ? (uint32_t)lrow * row_bytes + (uint32_t)blk * (4 * Q) : kOutOfRange, 0, t.d);
    const uint32_t gi = (uint32_t)lrow * groups_per_row + (uint32_t)(blk / (G / 32));
    t.s = __builtin_amdgcn_raw_buffer_load_b16(rs, in ? gi * 2 : kOutOfRange, 0, 0);
    if constexpr (ZP) t.z = load_group_meta<META>(rz, gi, in);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint32_t m = (uint32_t)(mb * 16 + lrow);
      // block j of the super-block, chunk lpiece of it: 16 tokens x 64 contiguous bytes
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool inj = valid & (4 * sb + j < nblk);
        const uint32_t off = inj ? (m * (uint32_t)K + (uint32_t)(128 * sb + 32 * j + 8 * lpiece)) * 2 : kOutOfRange;
        t.a[mb][j] = __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, kStream);
      }
    }
    // keep the loads where they are issued: the scheduler would otherwise move them
    // down next to their use, which removes the prefetch distance
    __builtin_amdgcn_sched_barrier(0);
  };

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  auto compute = [&](Slot& t) {
    // to the MFMA layout: codes, scale and zero point of (row l%16, block l/16); token
    // l%16's chunk l/16 of block j in register j
#pragma unroll
    for (int i = 0; i < Part<Q, 1>::kDwords; ++i) t.d[i] = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)t.d[i]);
    t.s = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)t.s);
    if constexpr (ZP) t.z = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)t.z);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) t.a[mb][j][e] = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)t.a[mb][j][e]);
    // 4x4 transpose across the four 16-lane rows: register j of row c holds chunk c of
    // block j; afterwards register j of row c holds chunk j of block c.
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        auto p02 = __builtin_amdgcn_permlane32_swap(t.a[mb][0][e], t.a[mb][2][e], false, false);
        auto p13 = __builtin_amdgcn_permlane32_swap(t.a[mb][1][e], t.a[mb][3][e], false, false);
        auto p01 = __builtin_amdgcn_permlane16_swap(p02[0], p13[0], false, false);
        auto p23 = __builtin_amdgcn_permlane16_swap(p02[1], p13[1], false, false);
        t.a[mb][0][e] = p01[0]; t.a[mb][1][e] = p01[1];
        t.a[mb][2][e] = p23[0]; t.a[mb][3][e] = p23[1];
      }
    const float s = f16_bits_to_f32(t.s);
    uint32_t w[16];
    dequant_part<Q, 1>(t.d, 0, s, dequant_offset<META, Q>(s, ZP ? t.z : 0u), w);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bf16x8 b = __builtin_bit_cast(bf16x8, u32x4{w[4 * j], w[4 * j + 1], w[4 * j + 2], w[4 * j + 3]});
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, t.a[mb][j]), b, acc[mb], 0, 0, 0);
    }
  };

  // Register slots used in turn: no copies (which would wait for the prefetch) and no
  // early exit between a load and its use (the compiler would sink the load past it).
  // A slot past the range holds zeros (scale 0), so computing it adds nothing.
  Slot s0, s1;
  load(sb_begin, sb_begin < sb_end, s0);
  for (int sb = sb_begin; sb < sb_end; sb += 2) {
    load(sb + 1, sb + 1 < sb_end, s1);
    compute(s0);
    load(sb + 2, sb + 2 < sb_end, s0);
    compute(s1);
  }

  // Cross-wavefront reduction: lane l of a wave holds D[4*(l/16) + r][l % 16] of each
  // 16-token block; sum the waves' tiles in wave order and write bf16.
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][mb * 256 + r * 64 + lane] = acc[mb][r];
  __syncthreads();
  for (int t = tid; t < MB * 256; t += (int)blockDim.x) {
    float sum = 0.0f;
    for (int w = 0; w < waves; ++w) sum += red[w][t];
    const int mb = t >> 8, r = (t >> 6) & 3, l = t & 63;
    const int m = mb * 16 + 4 * (l >> 4) + r;
    const int64_t n = n0 + (l & 15);
    if (m < M && n < N) y[(int64_t)m * N + n] = f32_to_bf16_bits(sum);
  }
}

// ---------------------------------------------------------------------------
// Split variant (caller workspace).  The kernel above re-reads every activation once
// per 16 weight rows (for M = 16 tokens at K = 14336: 117 MB from L2 against 29 MB of
// codes), which bounds it.  Here a workgroup owns 128 weight rows and one slice of K;
// each 16-token x 128-k activation chunk is loaded once into LDS and read by all eight
// wavefronts, and the slices of a row block meet in the workspace.
// ---------------------------------------------------------------------------
constexpr int kSplitWaves = 8;                 // 16 weight rows each
constexpr int kSplitRows = 16 * kSplitWaves;
constexpr int kChunk = 8;                      // super-blocks whose loads are in flight at once
constexpr int kSplitTargetWorkgroups = 512;    // two per CU
static_assert(kChunk == kSplitWaves, "wavefront w stages super-block w of a chunk");
constexpr int kSplitMaxSplits = 64;

typedef __attribute__((address_space(3))) void* lds_ptr_t;

struct SplitPlan {
  int64_t row_blocks;
  int splits;
  int mb;
  int64_t workspace;
};

// Enough workgroups to fill the chip and, where the split count allows, at most one
// chunk of super-blocks per slice (its loads then all go out before any arithmetic).
SplitPlan split_plan(int64_t M, int64_t N, int64_t K) {
  SplitPlan p{};
  p.row_blocks = (N + kSplitRows - 1) / kSplitRows;
  p.mb = M > 16 ? 2 : 1;
  const int64_t nsb = (K / 32 + 3) / 4;
  int64_t s = std::max<int64_t>(kSplitTargetWorkgroups / std::max<int64_t>(p.row_blocks, 1),
                                (nsb + kChunk - 1) / kChunk);
  s = std::min<int64_t>(s, std::min<int64_t>(nsb, kSplitMaxSplits));
  if (p.row_blocks > kMaxSplitCounters) s = 1;
  p.splits = (int)std::max<int64_t>(s, 1);
  p.workspace = p.splits > 1 ? kSplitCounterBytes + p.row_blocks * p.splits * kSplitWaves * p.mb * 256 * 4 : 0;
  return p;
}

template <int Q, int G, int META, int MB>
__global__ __launch_bounds__(64 * kSplitWaves) void skinny_split_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const void* __restrict__ meta, int M, int N, int K, int splits, int per, uint16_t* __restrict__ y,
    float* __restrict__ partials, unsigned int* __restrict__ counters) {
  constexpr int kStage = MB * 16 * 128 * 2;    // MB*16 tokens x 128 k, bf16
  __shared__ __attribute__((aligned(1024))) uint8_t xs[kChunk * kStage];
  __shared__ unsigned int arrived;

  // Grid: x = row block, y = slice of K (`per` super-blocks each).
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rb = (int)blockIdx.x, split = (int)blockIdx.y;
  const int64_t n0 = (int64_t)rb * kSplitRows + wave * 16;      // this wavefront's rows
  const int nblk = K / 32, nsb = (nblk + 3) / 4;
  const int sb_begin = std::min(nsb, split * per);
  const int nsteps = std::min(nsb, sb_begin + per) - sb_begin;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)(K / G);

  const uint32_t rows = (uint32_t)std::max<int64_t>(0, std::min<int64_t>(16, N - n0));
  const int64_t nb = rows ? n0 : 0;
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes + nb * row_bytes, rows * row_bytes);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(scales + nb * groups_per_row, rows * groups_per_row * 2);
  constexpr bool ZP = META != kMetaNone;
  constexpr int kMetaSize = meta_size<META>();
  const uint8_t* const zp = static_cast<const uint8_t*>(meta);
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(ZP ? zp + nb * groups_per_row * kMetaSize : zp,
                                              ZP ? rows * groups_per_row * kMetaSize : 0);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)M * (uint32_t)K * 2);

  // Activation chunk of a super-block in LDS (one stage per super-block of the chunk):
  // token block mb at mb*4 KB, token m at m*256, the 16-byte piece q (k = 128*sb + 8q)
  // at position q ^ m, so that the 16 lanes that read one MFMA operand row group hit 16
  // distinct bank groups.  Wavefront w fetches the stage of super-block w of the chunk,
  // 1 KB per load (tokens 4j..4j+3 of block mb): lane L takes position L%16 of token
  // 4j + L/16, i.e. piece (L%16) ^ m -- four neighbouring lanes read one aligned 64 bytes.
  const int d_m = lane >> 4;                   // + 4j
  auto issue_x = [&](int c0) {
    const int st = c0 + wave;
    const int sb = sb_begin + st;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = 4 * j + d_m;
        const int q = (lane & 15) ^ m;
        const bool in = (st < nsteps) & (4 * sb + (q >> 2) < nblk);
        const uint32_t off = ((uint32_t)(mb * 16 + m) * (uint32_t)K + (uint32_t)sb * 128 + 8 * q) * 2;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rx, (lds_ptr_t)(xs + wave * kStage + mb * 4096 + j * 1024), 16, in ? off : kOutOfRange, 0, 0, 0);
      }
  };
  constexpr int kXLoads = 4 * MB;

  // Codes: lane L loads row L/4, block L%4 of the super-block (quad-contiguous), and
  // ds_bpermute hands lane l the codes of row l%16, block l/16.
  const int lrow = lane >> 2, lpiece = lane & 3;
  const int perm = (4 * (lane & 15) + (lane >> 4)) * 4;
  struct Slot {
    uint32_t d[Part<Q, 1>::kDwords];
    uint32_t s, z;
  };
  auto issue_w = [&](int st, Slot& t) {
    const int blk = 4 * (sb_begin + st) + lpiece;
    const bool in = (st < nsteps) & (blk < nblk);
    load_part<Q, 1>(rc, in ? (uint32_t)lrow * row_bytes + (uint32_t)blk * (4 * Q) : kOutOfRange, 0, t.d);
    const uint32_t gi = (uint32_t)lrow * groups_per_row + (uint32_t)(blk / (G / 32));
    t.s = __builtin_amdgcn_raw_buffer_load_b16(rs, in ? gi * 2 : kOutOfRange, 0, 0);
    if constexpr (ZP) t.z = load_group_meta<META>(rz, gi, in);
  };
  constexpr int kWLoads = 2 + (ZP ? 1 : 0);     // vector loads of issue_w

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  const int am = lane & 15, ac = lane >> 4;     // MFMA operand row and 32-k block
  auto compute = [&](Slot& t, int stage) {
#pragma unroll
    for (int i = 0; i < Part<Q, 1>::kDwords; ++i) t.d[i] = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)t.d[i]);
    t.s = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)t.s);
    if constexpr (ZP) t.z = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)t.z);
    const float s = f16_bits_to_f32(t.s);
    uint32_t w[16];
    dequant_part<Q, 1>(t.d, 0, s, dequant_offset<META, Q>(s, ZP ? t.z : 0u), w);
    const uint8_t* xb = xs + stage * kStage + am * 256;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bf16x8 b = __builtin_bit_cast(bf16x8, u32x4{w[4 * j], w[4 * j + 1], w[4 * j + 2], w[4 * j + 3]});
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(xb + mb * 4096 + (((4 * ac + j) ^ am) << 4));
        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[mb], 0, 0, 0);
      }
    }
  };

  // Per chunk of up to kChunk super-blocks: every load of the chunk is issued first
  // (activations into LDS, then the codes of each super-block into its own register
  // slot; past the slice they are out of range and return zeros), the activations are
  // waited for and published with one barrier, and the super-blocks are then computed
  // in order as their codes land.  The barrier also keeps the compiler from moving the
  // code loads down to their (conditional) uses.
  for (int c0 = 0; c0 < nsteps; c0 += kChunk) {
    Slot sl[kChunk];
    issue_x(c0);
#pragma unroll
    for (int i = 0; i < kChunk; ++i) issue_w(c0 + i, sl[i]);
    wait_vmcnt<kChunk * kWLoads>();            // this wave's activation loads have landed
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kChunk; ++i)
      if (c0 + i < nsteps) compute(sl[i], i);
    if (c0 + kChunk < nsteps) __syncthreads();   // the next chunk reuses the stages
  }

  if (splits > 1) {
    // Same protocol as the split GEMM: write-through partials, arrival count, the last
    // workgroup of the row block sums the slices in slice order and resets the count.
    // Partials: [row block][slice][wavefront][token block][lane] x 4 floats, stored and
    // loaded 16 bytes per lane with device-scope coherence (sc1: written through to
    // memory, read past the non-coherent L2).
    constexpr int kSc1 = 16;
    constexpr uint32_t kSliceBytes = kSplitWaves * MB * 256 * 4;
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(partials + (int64_t)rb * splits * (kSliceBytes / 4),
                                                (uint32_t)splits * kSliceBytes);
    const uint32_t mine = (uint32_t)wave * (MB * 1024) + (uint32_t)lane * 16;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[mb]), rp,
                                             (uint32_t)split * kSliceBytes + mine + mb * 1024, 0, kSc1);
    wait_vmcnt<0>();
    __syncthreads();
    if (tid == 0) arrived = atomicAdd(&counters[rb], 1u);
    __syncthreads();
    if (arrived != (unsigned int)(splits - 1)) return;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // Sixteen slices per round trip: all loads of a round are issued before any add (a
    // slice index past the count reloads slice 0 and is added as zero).
    constexpr int kBatch = 16;
    for (int o0 = 0; o0 < splits; o0 += kBatch) {
      f32x4 v[kBatch][MB];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const uint32_t o = o0 + i < splits ? (uint32_t)(o0 + i) : 0u;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          v[i][mb] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rp, o * kSliceBytes + mine + mb * 1024, 0, kSc1));
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const bool live = o0 + i < splits;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[mb][e] += live ? v[i][mb][e] : 0.0f;
      }
    }
    if (tid == 0) __hip_atomic_store(&counters[rb], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = mb * 16 + 4 * (lane >> 4) + r;
      const int64_t n = n0 + (lane & 15);
      if (m < M && n < N) y[(int64_t)m * N + n] = f32_to_bf16_bits(acc[mb][r]);
    }
}

// ---------------------------------------------------------------------------
// Activation-stationary variant (q = 2 or 4; K a multiple of a wavefront's range).
//
// A wavefront owns one range of KB 32-weight blocks (512 k for one 16-token block, 256
// for two) and holds that range's activations in registers for the whole launch, as
// MFMA A operands.  A workgroup of four wavefronts covers four consecutive ranges (a
// slice of K) and walks a run of 16-row tiles.  Each wavefront moves its part of a tile
// (codes, scales, and zero points or minimums) from HBM into its own LDS stage with
// direct-to-LDS loads; the next tile's stage fills while the current one is computed.
//
// The scale is applied after the product (App. B.3).  For block b of row n,
//   sum_k x[m,k] s (u - o)  =  s * sum_k x[m,k] (128 + u)  -  s (128 + o) * xs[m,b],
// with xs[m,b] = sum_{k in b} x[m,k].  OR-ing a code into the bf16 constant 128
// (0x4300 | u == 128 + u) gives the first factor exactly, two weights per v_and_or;
// one bf16 MFMA per block takes the sum over k, and one fma per output applies s.  The
// second term is a product over blocks of xs[m,b] (formed once per wavefront) with a
// per-row coefficient c[n,b] = -s (128 + o) (zero point: o = z; minimum layout, where
// the weight is s*u + m: c = m - 128 s), added by fp32 MFMAs (16x16x4, four blocks
// each).  No weight is rounded: the dequantizing kernels round s (u - o) to bf16.
//
// LDS: a tile's codes sit row by row with one spare 16-byte slot per row (row pitch
// 16 (CPR + 1) bytes for CPR chunks of codes), so the 16 rows that one MFMA operand
// read touches fall into distinct bank groups; the loads fill the pitch directly (a
// load lane's slot p holds chunk p % (CPR + 1) of row p / (CPR + 1), the spare slots
// read out of range).
//
// Reduction: per tile the four wavefronts' partials meet in LDS (in wavefront order)
// and the sum goes to y, or, when K spans several slices, to the workspace; the last
// workgroup of a run to arrive adds the slices in slice order.
// ---------------------------------------------------------------------------
constexpr int kStatWaves = 4;

template <int Q, int G, int META, int MB>
struct StatLayout {
  static constexpr int kBlocks = MB == 1 ? 16 : 8;                 // KB: blocks of a range
  static constexpr int kRowBytes = kBlocks * 4 * Q;                // a row's codes in a range
  static constexpr int kChunks = kRowBytes / 16;                   // CPR
  static constexpr int kPitch = 16 * (kChunks + 1);                // LDS row pitch
  static constexpr int kCodeLoads = (16 * (kChunks + 1) + 63) / 64;
  static constexpr int kStageBytes = kCodeLoads * 1024;
  static constexpr int kGroups = kBlocks * 32 / G;                 // groups of a row in a range
  static constexpr int kMetaSize = META == kMetaZp ? 1 : META == kMetaMin ? 2 : 0;
  static constexpr int kScaleRow = 2 * kGroups;                    // bytes: 4 .. 32
  static constexpr int kMetaRow = kMetaSize * kGroups;             // bytes: 0 .. 32
  static constexpr int kScaleWords = kScaleRow / 4;
  static constexpr int kMetaWords = kMetaRow >= 4 ? kMetaRow / 4 : 1;
};

// One row's `B` bytes of scales or metadata into dwords (B = 32, 16, 8, 4, 2 or 1; the
// offset is a multiple of B, so every load is naturally aligned).
template <int B>
__device__ __forceinline__ void load_row_bytes(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t* d) {
  if constexpr (B >= 16) {
#pragma unroll
    for (int i = 0; i < B / 16; ++i) {
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(off + 16 * i), 0, 0);
      d[4 * i] = v.x; d[4 * i + 1] = v.y; d[4 * i + 2] = v.z; d[4 * i + 3] = v.w;
    }
  } else if constexpr (B == 8) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
    d[0] = v.x; d[1] = v.y;
  } else if constexpr (B == 4) {
    d[0] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
  } else if constexpr (B == 2) {
    d[0] = __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
  } else {
    d[0] = __builtin_amdgcn_raw_buffer_load_b8(r, (int)off, 0, 0);
  }
}

// Field g (`bits` wide) of a little-endian word array, g = g0 + dg with g0 known at
// compile time and dg <= 3 a lane's offset: a 64-bit window starting at g0's dword.
// (Called from fully unrolled loops: g0, and with it every index, folds to a constant.)
template <int BITS>
__device__ __forceinline__ uint32_t row_field(const uint32_t* w, int nwords, int g0, int dg) {
  const int kw = g0 * BITS / 32, kb = g0 * BITS % 32;
  const uint64_t win = (uint64_t)w[kw] | ((uint64_t)(kw + 1 < nwords ? w[kw + 1] : 0u) << 32);
  return (uint32_t)(win >> (kb + BITS * dg)) & ((1u << BITS) - 1u);
}

struct StatPlan {
  bool ok;
  int slices;
  int tiles_per_run;
  int64_t runs;
  int64_t workspace;
};

// Ranges of KB blocks per wavefront, four per workgroup (one slice of K), and runs of an
// even number of row tiles (the kernel takes them in pairs), sized so that the grid
// stays within three resident workgroups per CU.  One 16-token block (M <= 16): with
// two, the dequantizing split kernel measured faster.
StatPlan stat_plan(int64_t M, int64_t N, int64_t K, int q) {
  StatPlan p{};
  constexpr int mb = 1;
  constexpr int64_t range = 32 * 16;
  if ((q != 2 && q != 4) || M < 3 || M > 16 || K % range != 0 || N < 1) return p;
  const int64_t ranges = K / range;
  p.slices = (int)((ranges + kStatWaves - 1) / kStatWaves);
  const int64_t tiles = (N + 15) / 16;
  constexpr int64_t kResident = 3 * 256;
  int64_t r = std::max<int64_t>(2, (p.slices * tiles + kResident - 1) / kResident);
  r += r & 1;
  p.tiles_per_run = (int)r;
  p.runs = (tiles + r - 1) / r;
  if (p.runs > kMaxSplitCounters || p.runs > 65535) return p;
  p.workspace = p.slices > 1 ? kSplitCounterBytes + p.runs * p.slices * r * mb * 256 * 4 : 0;
  p.ok = true;
  return p;
}

// Sum of the eight bf16 activations of a dword quad (fp32).  The dwords are copied out
// of the vector first: a bit cast applied to a vector element (`a[i]`) reads element 0
// whatever i is (hipcc generates a single dword load for all four).
__device__ __forceinline__ float quad_sum(const u32x4 a) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  constexpr uint32_t kOne = 0x3F803F80u;
  const uint32_t d[4] = {a.x, a.y, a.z, a.w};
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2, d[i]), __builtin_bit_cast(bf2, kOne), s, false);
  return s;
}

// Lane (m, c) = (l % 16, l / 16) holds q_t = partial of block 4i + t for t < 4 (its own
// 8 activations of each block); returns the full block sum of block 4i + c for token m:
// halves of the wavefront exchange (lanes l, l ^ 32), then 16-lane rows (l, l ^ 16).
__device__ __forceinline__ float scatter_block_sums(float q0, float q1, float q2, float q3) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(q0), __float_as_uint(q2), false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(q1), __float_as_uint(q3), false, false);
  const float u = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const float v = __uint_as_float(b[0]) + __uint_as_float(b[1]);
  const auto d = __builtin_amdgcn_permlane16_swap(__float_as_uint(u), __float_as_uint(v), false, false);
  return __uint_as_float(d[0]) + __uint_as_float(d[1]);
}

// The four bf16 pairs (128 + u) of the 8 codes in `w` (q = 4: 8 nibbles; q = 2: 8
// fields in the low 16 bits), paired (e0, e4), (e1, e5), (e2, e6), (e3, e7).
template <int Q>
__device__ __forceinline__ u32x4 stat_pairs(uint32_t w, uint32_t magic) {
  if constexpr (Q == 2) w = __builtin_amdgcn_perm(0u, w, 0x0C010C00u);   // bytes {b0, 0, b1, 0}
  constexpr uint32_t kMask = Q == 4 ? 0x000F000Fu : 0x00030003u;
  return u32x4{and_or(w, kMask, magic), and_or(w >> Q, kMask, magic), and_or(w >> (2 * Q), kMask, magic),
               and_or(w >> (3 * Q), kMask, magic)};
}

template <int Q, int G, int META, int MB>
struct StatArgs {
  const uint8_t* codes;
  const uint16_t* scales;
  const uint8_t* meta;
  int N, kb0, tile0;
  bool active;
  uint32_t row_bytes, gpr;
};

// A tile's scales and metadata in registers: lane (n, c) holds row n's groups of the
// wavefront's range.
template <int Q, int G, int META, int MB>
struct StatRow {
  using L = StatLayout<Q, G, META, MB>;
  uint32_t s[L::kScaleWords];
  uint32_t z[L::kMetaWords];
};

// Loads of tile t (rows 16t.. of the run): its codes into a wavefront's LDS stage with
// direct-to-LDS loads (offsets `coff`), its scales and metadata into registers.
template <int Q, int G, int META, int MB>
__device__ __forceinline__ void stat_issue(const StatArgs<Q, G, META, MB>& a, int t, bool in_run, uint8_t* stage,
                                           const uint32_t (&coff)[StatLayout<Q, G, META, MB>::kCodeLoads], int n,
                                           StatRow<Q, G, META, MB>& row) {
  using L = StatLayout<Q, G, META, MB>;
  const int64_t n0 = (int64_t)(a.tile0 + t) * 16;
  const int rows = (int)std::max<int64_t>(0, std::min<int64_t>(16, a.N - n0));
  // the same loads for every tile (past the run or past N they move nothing), so the
  // count of loads in flight is the same on every pass of the loop
  const bool live = in_run && a.active && rows > 0;
  const int64_t g0 = a.kb0 / (G / 32);
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(a.codes + n0 * a.row_bytes + (int64_t)a.kb0 * 4 * Q,
                                              live ? (uint32_t)rows * a.row_bytes - (uint32_t)a.kb0 * 4 * Q : 0u);
#pragma unroll
  for (int i = 0; i < L::kCodeLoads; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (lds_ptr_t)(stage + 1024 * i), 16, (int)coff[i], 0, 0, 0);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.scales + n0 * a.gpr + g0,
                                              live ? ((uint32_t)rows * a.gpr - (uint32_t)g0) * 2 : 0u);
  load_row_bytes<L::kScaleRow>(rs, (uint32_t)n * a.gpr * 2, row.s);
  if constexpr (L::kMetaSize > 0) {
    const __amdgpu_buffer_rsrc_t rz =
        make_rsrc(a.meta + (n0 * a.gpr + g0) * L::kMetaSize,
                  live ? ((uint32_t)rows * a.gpr - (uint32_t)g0) * L::kMetaSize : 0u);
    load_row_bytes<L::kMetaRow>(rz, (uint32_t)n * a.gpr * L::kMetaSize, row.z);
  } else {
    row.z[0] = 0u;
  }
}

// One tile from a stage: acc[mb] = this wavefront's range's share of the 16 x 16 output
// block (tokens 16 mb + 4 (l / 16) + r, row l % 16 in lane l, register r).
template <int Q, int G, int META, int MB>
__device__ __forceinline__ void stat_compute(const uint8_t* stage, const StatRow<Q, G, META, MB>& row,
                                             const bf16x8 (&A)[StatLayout<Q, G, META, MB>::kBlocks][MB],
                                             const float (&XS)[StatLayout<Q, G, META, MB>::kBlocks / 4][MB],
                                             int n, int c, f32x4 (&acc)[MB]) {
  using L = StatLayout<Q, G, META, MB>;
  constexpr int KB = L::kBlocks, GB = G / 32;
  const uint32_t magic = 0x43004300u;
  const uint32_t* const sv = row.s;
  // The block-sum term first: lane (n, c) supplies the coefficient of row n, block
  // 4i + c, and the fp32 MFMAs start acc from it (C = 0), so no MFMA reads a register
  // that a VALU instruction has just written.
  const int gc = c / GB;
  float coef[KB / 4];
#pragma unroll
  for (int i = 0; i < KB / 4; ++i) {
    const float s = f16_bits_to_f32(row_field<16>(row.s, L::kScaleWords, 4 * i / GB, gc));
    if constexpr (META == kMetaMin) {
      const float m = f16_bits_to_f32(row_field<16>(row.z, L::kMetaWords, 4 * i / GB, gc));
      coef[i] = __builtin_fmaf(-128.0f, s, m);
    } else if constexpr (META == kMetaZp) {
      const float z = (float)row_field<8>(row.z, L::kMetaWords, 4 * i / GB, gc);
      coef[i] = -(128.0f + z) * s;
    } else {
      coef[i] = -(128.0f + (float)(1 << (Q - 1))) * s;
    }
  }
  const uint8_t* crow = stage + n * L::kPitch + c * Q;
  uint32_t wv[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) {
    if constexpr (Q == 4) wv[j] = *reinterpret_cast<const uint32_t*>(crow + 16 * j);
    else wv[j] = *reinterpret_cast<const uint16_t*>(crow + 8 * j);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    acc[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(XS[0][mb], coef[0], f32x4{0.0f, 0.0f, 0.0f, 0.0f}, 0, 0, 0);
#pragma unroll
    for (int i = 1; i < KB / 4; ++i) acc[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(XS[i][mb], coef[i], acc[mb], 0, 0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
  // Group g's product accumulates in d[g % kRing] and is scaled kLag groups later.  A
  // VALU read of an MFMA result a few instructions after the MFMA, as the scheduler
  // places it on its own, was measured to return the register's previous contents (the
  // wait the compiler inserts is too short here), so every block's MFMA and every
  // group's scaling sit between scheduling barriers and a result is read three groups
  // (at least 3 x 12 instructions) after it is written; the last groups, and acc, after
  // a fixed wait.
  constexpr int kLag = 3, kRing = kLag + 1, kG = KB / GB;
  f32x4 d[kRing][MB];
  auto scale_group = [&](int g, const f32x4 (&dg)[MB]) {
    const float s = (g & 1) ? f16_hi(sv[g >> 1]) : f16_lo(sv[g >> 1]);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[mb][r] = __builtin_fmaf(s, dg[mb][r], acc[mb][r]);
  };
#pragma unroll
  for (int j = 0; j < KB; ++j) {
    const bf16x8 b = __builtin_bit_cast(bf16x8, stat_pairs<Q>(wv[j], magic));
    const int g = j / GB, slot = g % kRing;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      d[slot][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[j][mb], b,
                                                            j % GB == 0 ? f32x4{0.0f, 0.0f, 0.0f, 0.0f} : d[slot][mb],
                                                            0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (j % GB == GB - 1 && g >= kLag) {
      scale_group(g - kLag, d[(g - kLag) % kRing]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int g = kG > kLag ? kG - kLag : 0; g < kG; ++g) scale_group(g, d[g % kRing]);
}

template <int Q, int G, int META, int MB>
__global__ __launch_bounds__(64 * kStatWaves) void skinny_stat_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const void* __restrict__ meta, int M, int N, int K, int R, uint16_t* __restrict__ y,
    float* __restrict__ partials, unsigned int* __restrict__ counters) {
  using L = StatLayout<Q, G, META, MB>;
  constexpr int KB = L::kBlocks;
  constexpr int kPart = MB * 256;               // floats of one wavefront's tile partial
  // Each stage its own LDS object: the compiler then waits for exactly the loads of the
  // stage it reads.
  __shared__ __attribute__((aligned(1024))) uint8_t stage0[kStatWaves * L::kStageBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t stage1[kStatWaves * L::kStageBytes];
  __shared__ __attribute__((aligned(16))) float part[kStatWaves * kPart];
  __shared__ unsigned int arrived;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int slices = (int)gridDim.x, slice = (int)blockIdx.x, run = (int)blockIdx.y;
  const int n = lane & 15, c = lane >> 4;
  StatArgs<Q, G, META, MB> a;
  a.codes = codes; a.scales = scales; a.meta = static_cast<const uint8_t*>(meta);
  a.N = N;
  a.kb0 = (slice * kStatWaves + wave) * KB;
  a.active = a.kb0 < K / 32;
  a.tile0 = run * R;
  a.row_bytes = (uint32_t)K * Q / 8;
  a.gpr = (uint32_t)(K / G);
  uint8_t* const st0 = stage0 + wave * L::kStageBytes;
  uint8_t* const st1 = stage1 + wave * L::kStageBytes;

  // Code load lanes' offsets, the same for every tile (each tile gets descriptors of its own).
  uint32_t coff[L::kCodeLoads];
#pragma unroll
  for (int i = 0; i < L::kCodeLoads; ++i) {
    const int p = 64 * i + lane, row = p / (L::kChunks + 1), ch = p % (L::kChunks + 1);
    coff[i] = row < 16 && ch < L::kChunks ? (uint32_t)row * a.row_bytes + 16 * ch : kOutOfRange;
  }

  // The range's activations: lane (m, c) holds 8 values of token 16 mb + m, chunk c of
  // each block, paired (x0, x4), (x1, x5), (x2, x6), (x3, x7) like the code pairs.
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)M * (uint32_t)K * 2);
  u32x4 xr[KB][MB];
#pragma unroll
  for (int j = 0; j < KB; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint32_t off = ((uint32_t)(16 * mb + n) * (uint32_t)K + 32 * (uint32_t)(a.kb0 + j) + 8 * c) * 2;
      xr[j][mb] = __builtin_amdgcn_raw_buffer_load_b128(rx, a.active ? (int)off : (int)kOutOfRange, 0, 0);
    }
  StatRow<Q, G, META, MB> row0, row1;
  stat_issue<Q, G, META, MB>(a, 0, true, st0, coff, n, row0);

  bf16x8 A[KB][MB];
  float XS[KB / 4][MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    float q[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const u32x4 v = xr[j][mb];
      constexpr uint32_t kLo = 0x05040100u, kHi = 0x07060302u;
      const u32x4 pr{__builtin_amdgcn_perm(v.z, v.x, kLo), __builtin_amdgcn_perm(v.z, v.x, kHi),
                     __builtin_amdgcn_perm(v.w, v.y, kLo), __builtin_amdgcn_perm(v.w, v.y, kHi)};
      A[j][mb] = __builtin_bit_cast(bf16x8, pr);
      q[j] = quad_sum(v);
    }
#pragma unroll
    for (int i = 0; i < KB / 4; ++i) XS[i][mb] = scatter_block_sums(q[4 * i], q[4 * i + 1], q[4 * i + 2], q[4 * i + 3]);
  }

  // Partial stores: [run][slice][tile][kPart] floats, written through (sc1) for the
  // workgroup that adds the slices; with one slice y is written directly.  Both stores
  // are issued for every element (the unused one, and those of a tile outside the run,
  // out of range), so every pass of the loop issues the same memory operations.
  constexpr int kSc1 = 16;
  const __amdgpu_buffer_rsrc_t rp =
      make_rsrc(partials + ((int64_t)run * slices + slice) * R * kPart, slices > 1 ? (uint32_t)R * kPart * 4 : 0u);
  const __amdgpu_buffer_rsrc_t ry = make_rsrc(y, slices > 1 ? 0u : (uint32_t)M * (uint32_t)N * 2);
  auto finish_tile = [&](int t) {
    // the four wavefronts' partials of tile t, in wavefront order
    const bool in_run = t >= 0 && t < R;
    const int64_t n0 = (int64_t)(a.tile0 + t) * 16;
#pragma unroll
    for (int e0 = 0; e0 < kPart; e0 += 64 * kStatWaves) {
      const int e = e0 + tid;
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < kStatWaves; ++w) v += part[w * kPart + e];
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), rp, in_run ? (t * kPart + e) * 4 : (int)kOutOfRange,
                                            0, kSc1);
      const int mb = e >> 8, l = (e & 255) >> 2, r = e & 3;
      const int m = 16 * mb + 4 * (l >> 4) + r;
      const int64_t row = n0 + (l & 15);
      const bool out = in_run && m < M && row < N;
      __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_bits(v), ry,
                                            out ? (int)(((uint32_t)m * (uint32_t)N + (uint32_t)row) * 2) : (int)kOutOfRange,
                                            0, 0);
    }
  };
  auto park = [&](const f32x4 (&acc)[MB]) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) *reinterpret_cast<f32x4*>(part + wave * kPart + mb * 256 + 4 * lane) = acc[mb];
  };

  // Tiles in pairs (R is even): the loads of tile t+1 are in flight while tile t is
  // computed, and every pass issues the same loads and stores (so the compiler waits for
  // the current tile's, not the next one's).  Barriers, for LDS only (no load writes
  // `part`): after a tile's `part` is written (it is read by all), and after it is read
  // (it is written again).
  f32x4 acc[MB];
  for (int t = 0; t < R; t += 2) {
    lds_barrier();
    finish_tile(t - 1);
    lds_barrier();
    stat_issue<Q, G, META, MB>(a, t + 1, true, st1, coff, n, row1);
    stat_compute<Q, G, META, MB>(st0, row0, A, XS, n, c, acc);
    park(acc);
    lds_barrier();
    finish_tile(t);
    lds_barrier();
    stat_issue<Q, G, META, MB>(a, t + 2, t + 2 < R, st0, coff, n, row0);
    stat_compute<Q, G, META, MB>(st1, row1, A, XS, n, c, acc);
    park(acc);
  }
  lds_barrier();
  finish_tile(R - 1);

  if (slices > 1) {
    // Arrival count per run; the last workgroup adds the slices in slice order.
    wait_vmcnt<0>();
    __syncthreads();
    if (tid == 0) arrived = atomicAdd(&counters[run], 1u);
    __syncthreads();
    if (arrived != (unsigned int)(slices - 1)) return;
    const __amdgpu_buffer_rsrc_t rall = make_rsrc(partials + (int64_t)run * slices * R * kPart,
                                                  (uint32_t)slices * R * kPart * 4);
    const int total = R * kPart;
    for (int e4 = 4 * tid; e4 < total; e4 += 4 * 64 * kStatWaves) {
      constexpr int kLoads = 8;
      f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int s0 = 0; s0 < slices; s0 += kLoads) {
        f32x4 v[kLoads];
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
          const uint32_t sl = s0 + i < slices ? (uint32_t)(s0 + i) : 0u;
          v[i] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                               rall, (int)((sl * (uint32_t)total + (uint32_t)e4) * 4), 0, kSc1));
        }
#pragma unroll
        for (int i = 0; i < kLoads; ++i)
          if (s0 + i < slices) sum += v[i];
      }
      const int t = e4 / kPart, e = e4 % kPart;
      const int64_t n0 = (int64_t)(a.tile0 + t) * 16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int mb = e >> 8, l = (e & 255) >> 2;
        const int m = 16 * mb + 4 * (l >> 4) + r;
        const int64_t row = n0 + (l & 15);
        if (m < M && row < N) y[(int64_t)m * N + row] = f32_to_bf16_bits(sum[r]);
      }
    }
    if (tid == 0) __hip_atomic_store(&counters[run], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int Q, int G, int META>
bool skinny_stat_launch(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                        const void* zp, int64_t N, int64_t K, uint16_t* y, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  if constexpr (Q == 3) {
    return false;
  } else {
    const StatPlan p = stat_plan(M, N, K, Q);
    if (!p.ok) return false;
    if (reinterpret_cast<uintptr_t>(scales) % 16 != 0 || reinterpret_cast<uintptr_t>(zp) % 16 != 0) return false;
    if (p.slices > 1 && (workspace == nullptr || (int64_t)workspace_bytes < p.workspace)) return false;
    unsigned int* counters = static_cast<unsigned int*>(workspace);
    float* partials = p.slices > 1 ? reinterpret_cast<float*>(static_cast<char*>(workspace) + kSplitCounterBytes)
                                   : nullptr;
    const dim3 grid((unsigned)p.slices, (unsigned)p.runs), block(64 * kStatWaves);
    skinny_stat_kernel<Q, G, META, 1><<<grid, block, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N, (int)K,
                                                                  p.tiles_per_run, y, partials, counters);
    return true;
  }
}

template <int Q, int G, int META>
hipError_t skinny_dispatch(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                           const void* zp, int64_t N, int64_t K, uint16_t* y, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  if (skinny_stat_launch<Q, G, META>(x, M, codes, scales, zp, N, K, y, workspace, workspace_bytes, stream))
    return hipGetLastError();
  const SplitPlan p = split_plan(M, N, K);
  if (p.splits > 1 && workspace != nullptr && (int64_t)workspace_bytes >= p.workspace) {
    unsigned int* counters = static_cast<unsigned int*>(workspace);
    float* partials = reinterpret_cast<float*>(static_cast<char*>(workspace) + kSplitCounterBytes);
    const int64_t nsb = (K / 32 + 3) / 4;
    const int per = (int)((nsb + p.splits - 1) / p.splits);
    const dim3 grid((unsigned)p.row_blocks, (unsigned)p.splits), block(64 * kSplitWaves);
    if (p.mb == 1)
      skinny_split_kernel<Q, G, META, 1><<<grid, block, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N, (int)K,
                                                                   p.splits, per, y, partials, counters);
    else
      skinny_split_kernel<Q, G, META, 2><<<grid, block, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N, (int)K,
                                                                   p.splits, per, y, partials, counters);
    return hipGetLastError();
  }
  const int64_t nsb = (K / 32 + 3) / 4;
  const int waves = (int)std::min<int64_t>(kMaxWaves, nsb);
  const dim3 grid((unsigned)((N + 15) / 16)), block((unsigned)(64 * waves));
  if (M <= 16)
    skinny_kernel<Q, G, META, 1><<<grid, block, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N, (int)K, y);
  else
    skinny_kernel<Q, G, META, 2><<<grid, block, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N, (int)K, y);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_skinny_bf16(const uint16_t* x, int64_t M, const uint8_t* codes,
                              const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K,
                              int group, int q, uint16_t* y, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  if (M < 2 || M > kSkinnyMaxM) return hipErrorInvalidValue;
  SSQ_DISPATCH_QGM(skinny_dispatch, q, group, meta.kind, x, M, codes, scales, meta.ptr, N, K, y, workspace,
                   workspace_bytes, stream);
}

size_t skinny_workspace_bytes(int64_t M, int64_t N, int64_t K, int q) {
  // the larger of the two split layouts: which kernel runs also depends on alignment
  const StatPlan sp = stat_plan(M, N, K, q);
  return (size_t)std::max<int64_t>(split_plan(M, N, K).workspace, sp.ok ? sp.workspace : 0);
}

}  // namespace ssq
