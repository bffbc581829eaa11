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

template <int Q, int G, int META>
hipError_t skinny_dispatch(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                           const void* zp, int64_t N, int64_t K, uint16_t* y, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
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

size_t skinny_workspace_bytes(int64_t M, int64_t N, int64_t K) { return (size_t)split_plan(M, N, K).workspace; }

}  // namespace ssq
