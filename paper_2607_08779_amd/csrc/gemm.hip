// Prefill GEMM: y[M,N] = x[M,K] * What[N,K]^T with What dequantized into LDS.
//
// App. B.3 of the paper: What[n,k] = s[n,b] (u[n,k] - o[n,b]).  Prefill is a
// dense contraction, so it runs on bf16 MFMA.  Each workgroup owns a BM x BN
// output tile; per BK-deep step it stages the activation tile and dequantizes
// the weight tile (s*(u - o) is exact in fp32, then rounded to bf16) into one of
// two LDS buffers while its four wavefronts multiply the other buffer's 64x64
// sub-tiles with v_mfma_f32_16x16x32_bf16 (fp32 accumulation).  The next step's
// global loads are issued before the current step's MFMAs; one barrier per step.
//
// MFMA operand layout (16x16x32): lane l supplies row (l % 16) of A and column
// (l % 16) of B, each with 8 consecutive k values starting at 8 * (l / 16).
// Both operands use the same k assignment, so the reduction is correct for any
// internal k order.  Lane l receives D[4 * (l / 16) + r][l % 16], r = 0..3.
#include <algorithm>
#include <type_traits>

#include "ssq_internal.h"

namespace ssq {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kTileBytes = BM * BK * 2;     // one 128 x 64 bf16 tile: 128 rows of 128 bytes
constexpr int kAStages = 3, kBStages = 2;   // 80 KB of LDS: two workgroups per CU

// Byte offset of 16-byte chunk c (8 bf16 along k) of row r in a tile.  The chunk index
// is XOR-swizzled with the row, so the 16 rows an MFMA operand read touches at one k
// offset fall in 8 different chunk columns (no padding needed).
__device__ __forceinline__ uint32_t swz(int r, int c) { return (uint32_t)(r * 128 + ((c ^ (r & 7)) << 4)); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float f16_lo(uint32_t p) { return (float)__builtin_bit_cast(_Float16, (uint16_t)p); }
__device__ __forceinline__ float f16_hi(uint32_t p) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(p >> 16)); }

// 32 weights s*(u - o) of one block as 16 bf16 pairs (natural k order).  Each q-bit
// field is OR-ed into the mantissa of the fp16 constant 1024 (0x6400 | u == 1024 + u),
// two fields per instruction; one v_fma_mix_f32 per weight then forms
// (1024 + u)*s - (1024 + o)*s.  Both products are exact in fp32 (11-bit by 11-bit), so
// the result is s*(u - o) exactly; it is rounded to bf16 once.  `so` = -(1024 + o)*s.
template <int Q>
__device__ __forceinline__ void dequant_block(const uint32_t (&d)[Q], float s, float so, uint32_t (&w)[16]) {
  const uint32_t magic = 0x64006400u;
  float f[32];
  if constexpr (Q == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
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
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {          // fields j and j + 8 of this dword
        const uint32_t p = and_or(d[i] >> (2 * j), 0x00030003u, magic);
        f[16 * i + j] = __builtin_fmaf(f16_lo(p), s, so);
        f[16 * i + j + 8] = __builtin_fmaf(f16_hi(p), s, so);
      }
  } else {
    // Four 24-bit words of 8 fields; fields 4..7 of each word moved up to bit 16.
    const uint32_t v[4] = {d[0], __builtin_amdgcn_alignbit(d[1], d[0], 24),
                           __builtin_amdgcn_alignbit(d[2], d[1], 16), d[2] >> 8};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t sp = (v[i] & 0xFFFu) | ((v[i] << 4) & 0x0FFF0000u);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t p = and_or(sp >> (3 * j), 0x00070007u, magic);
        f[8 * i + j] = __builtin_fmaf(f16_lo(p), s, so);
        f[8 * i + j + 4] = __builtin_fmaf(f16_hi(p), s, so);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 16; ++k) w[k] = pack_bf16x2(f[2 * k], f[2 * k + 1]);
}

// Tile order: workgroups are dealt round-robin to the 8 XCDs.  When the tile count
// divides evenly, XCD x takes a contiguous run of tiles enumerated weight-panel
// major (all M tiles of one N tile together), so a weight panel's codes are fetched
// once per XCD and shared through its L2.
__device__ __forceinline__ void tile_of(int t, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  if (total % 8 == 0) t = (t % 8) * (total / 8) + t / 8;
  tn = t / tiles_m;
  tm = t % tiles_m;
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// ---------------------------------------------------------------------------
// Split reduction (host side).  When the output has too few tiles to occupy the CUs
// twice over, the K steps of each tile are divided among `splits` workgroups whose fp32
// partial tiles meet in a caller-provided workspace: [counters: one u32 per tile,
// padded to 256 bytes][partials: tiles x splits x BM x BN fp32].
// ---------------------------------------------------------------------------
constexpr int64_t kTargetWorkgroups = 512;   // two resident workgroups per CU
constexpr int kMinStepsPerSplit = 16;

int64_t counter_bytes(int64_t tiles) { return (tiles * 4 + 255) / 256 * 256; }

int desired_splits(int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const int64_t steps = (K / 32 + 1) / 2;
  int64_t s = kTargetWorkgroups / tiles;
  s = std::min<int64_t>(s, steps / kMinStepsPerSplit);
  s = std::min<int64_t>(s, 8);
  return (int)std::max<int64_t>(s, 1);
}

int64_t workspace_for(int64_t M, int64_t N, int64_t K, int splits) {
  if (splits <= 1) return 0;
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  return counter_bytes(tiles) + tiles * splits * BM * BN * 4;
}

int gemm_splits(int64_t M, int64_t N, int64_t K, const void* workspace, size_t bytes) {
  const int s = desired_splits(M, N, K);
  if (s <= 1 || workspace == nullptr || (int64_t)bytes < workspace_for(M, N, K, s)) return 1;
  return s;
}

// s_waitcnt on the vector-memory counter only (gfx9 encoding: vmcnt in bits 3:0 and
// 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima).  Loads complete in order,
// so vmcnt <= N means everything but the last N loads has landed -- including loads
// that write LDS directly, which the compiler does not track.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | 0x70 | 0xF00 | ((N >> 4) << 14));
}

template <int Q, int G, bool ZP>
__global__ __launch_bounds__(256) void gemm_kernel(const uint16_t* __restrict__ x, int M,
                                                   const uint8_t* __restrict__ codes,
                                                   const uint16_t* __restrict__ scales,
                                                   const uint8_t* __restrict__ zp, int N, int K,
                                                   uint16_t* __restrict__ y, int splits,
                                                   float* __restrict__ partials,
                                                   unsigned int* __restrict__ counters) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[(kAStages + kBStages) * kTileBytes];
  uint8_t* const As = smem;
  uint8_t* const Bs = smem + kAStages * kTileBytes;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int tiles = tiles_m * tiles_n;
  const int tile_id = (int)blockIdx.x % tiles;   // splits of one tile share no operand data
  const int split = (int)blockIdx.x / tiles;
  int tm, tn;
  tile_of(tile_id, tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int nblk = K / 32;
  const int total_steps = (nblk + 1) / 2;
  // This workgroup's slice of the reduction: steps [s_begin, s_begin + nsteps).
  const int per_split = (total_steps + splits - 1) / splits;
  const int s_begin = split * per_split;
  const int nsteps = total_steps - s_begin < per_split ? total_steps - s_begin : per_split;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)(K / G);
  constexpr float kSymOffset = (float)(1 << (Q - 1));
  constexpr int kLoadsPerStep = 4 + 2 + (ZP ? 1 : 0);

  // Buffer descriptors relative to the tile's first row; rows past M or N read zeros.
  const uint32_t rows_a = (uint32_t)(M - m0 < BM ? M - m0 : BM);
  const uint32_t rows_b = (uint32_t)(N - n0 < BN ? N - n0 : BN);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(x + m0 * K, rows_a * (uint32_t)K * 2);
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes + n0 * row_bytes, rows_b * row_bytes);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(scales + n0 * groups_per_row, rows_b * groups_per_row * 2);
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(ZP ? zp + n0 * groups_per_row : zp, ZP ? rows_b * groups_per_row : 0);

  // Activation tile: 16 wavefront loads of 1 KB straight into LDS.  Wave w issues loads
  // 4w..4w+3; load j fills tile rows 8j..8j+7, lane i writing 16 bytes at 16*i, which
  // is row 8j + i/8, swizzled chunk i%8 -- so lane i fetches logical chunk (i%8)^(row%8).
  uint32_t a_off[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = 8 * (4 * wave + j) + (lane >> 3);
    const int c = (lane & 7) ^ (r & 7);
    a_off[j] = (uint32_t)r * K * 2 + c * 16;
  }
  auto issue_a = [&](int lstep, int stage) {
    const int step = s_begin + lstep;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = (lane & 7) ^ ((8 * (4 * wave + j) + (lane >> 3)) & 7);
      // chunks past K (odd block count, last step) read out of range -> zeros
      const uint32_t off = step * 64 + c * 8 < K ? a_off[j] + (uint32_t)step * 128 : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ra, (lds_ptr_t)(As + stage * kTileBytes + (4 * wave + j) * 1024), 16, off, 0, 0, 0);
    }
  };

  // Weight tile: thread t dequantizes 32-weight block (t % 2) of row t / 2.
  const int lr = tid >> 1, lh = tid & 1;
  const uint32_t c_off = (uint32_t)lr * row_bytes + lh * (4 * Q);
  uint32_t c_reg[2][Q], s_reg[2], z_reg[2];
  auto issue_b = [&](int lstep, int slot) {
    const int step = s_begin + lstep;
    const int blk = 2 * step + lh;
    const bool in = blk < nblk;
    uint32_t d[Q];
    buffer_block_codes<Q>(rc, in ? c_off + (uint32_t)step * (8 * Q) : 0x80000000u, 0, d);
#pragma unroll
    for (int i = 0; i < Q; ++i) c_reg[slot][i] = d[i];
    const uint32_t gi = (uint32_t)lr * groups_per_row + (uint32_t)(blk / (G / 32));
    s_reg[slot] = __builtin_amdgcn_raw_buffer_load_b16(rs, in ? gi * 2 : 0x80000000u, 0, 0);
    if constexpr (ZP) z_reg[slot] = __builtin_amdgcn_raw_buffer_load_b8(rz, in ? gi : 0x80000000u, 0, 0);
  };
  auto store_b = [&](int slot, int stage) {
    const float s = f16_bits_to_f32(s_reg[slot]);
    const float o = ZP ? (float)z_reg[slot] : kSymOffset;
    uint32_t w[16];
    dequant_block<Q>(c_reg[slot], s, -(1024.0f + o) * s, w);   // exact: 11-bit times 11-bit
    uint8_t* dst = Bs + stage * kTileBytes;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      *reinterpret_cast<uint4*>(dst + swz(lr, lh * 4 + e)) = uint4{w[4 * e], w[4 * e + 1], w[4 * e + 2], w[4 * e + 3]};
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  auto mfma_step = [&](int step) {
    const uint8_t* at = As + (step % kAStages) * kTileBytes;
    const uint8_t* bt = Bs + (step % kBStages) * kTileBytes;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 a[4], b[4];
      const int c = ks * 4 + (lane >> 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = *reinterpret_cast<const bf16x8*>(at + swz(wm * 64 + i * 16 + (lane & 15), c));
        b[i] = *reinterpret_cast<const bf16x8*>(bt + swz(wn * 64 + i * 16 + (lane & 15), c));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // Step s: issue loads for s+2, multiply stage s, dequantize codes of s+1, then wait
  // for this wave's activation loads of s+1 and barrier.  Slots are static (the loop is
  // unrolled by two) so the code registers never need dynamic indexing.
  auto step_body = [&](int s, auto slot_c) {
    constexpr int kSlot = decltype(slot_c)::value;
    const bool ahead = s + 2 < nsteps;
    if (ahead) {
      issue_a(s + 2, (s + 2) % kAStages);
      issue_b(s + 2, kSlot);
    }
    mfma_step(s);
    if (s + 1 < nsteps) store_b(1 - kSlot, (s + 1) % kBStages);
    if (ahead) wait_vmcnt<kLoadsPerStep>();
    else wait_vmcnt<0>();
    __syncthreads();
  };

  issue_a(0, 0);
  issue_b(0, 0);
  if (nsteps > 1) {
    issue_a(1, 1);
    issue_b(1, 1);
  }
  store_b(0, 0);
  if (nsteps > 1) wait_vmcnt<kLoadsPerStep>();
  else wait_vmcnt<0>();
  __syncthreads();
  for (int s = 0; s < nsteps; s += 2) {
    step_body(s, std::integral_constant<int, 0>{});
    if (s + 1 < nsteps) step_body(s + 1, std::integral_constant<int, 1>{});
  }

  if (splits > 1) {
    // Split reduction: publish this slice's fp32 partial tile in the lane order of the
    // accumulators (coalesced), then count arrivals; the last arriving workgroup sums
    // all slices in a fixed order, writes y and resets the counter so the workspace
    // stays reusable.
    float* mine = partials + ((int64_t)tile_id * splits + split) * (BM * BN) + wave * 4096 + lane;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) mine[((i * 4 + j) * 4 + r) * 64] = acc[i][j][r];
    __threadfence();                       // release the partial to the whole device
    // The tile buffers are idle after the main loop; their first word carries the arrival
    // count to the whole workgroup (a separate shared variable would push LDS past 80 KB
    // and halve the workgroups per CU).
    unsigned int* arrived = reinterpret_cast<unsigned int*>(smem);
    __syncthreads();
    if (tid == 0) *arrived = atomicAdd(&counters[tile_id], 1u);
    __syncthreads();
    if (*arrived != (unsigned int)(splits - 1)) return;   // uniform across the workgroup
    __threadfence();                       // acquire the other slices' partials
    // Sum every slice (this one included) in slice order, so the result does not depend
    // on which workgroup arrived last.
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int o = 0; o < splits; ++o) {
      const float* part = partials + ((int64_t)tile_id * splits + o) * (BM * BN) + wave * 4096 + lane;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[i][j][r] += __builtin_nontemporal_load(part + ((i * 4 + j) * 4 + r) * 64);
    }
    if (tid == 0) counters[tile_id] = 0u;
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
                         const uint8_t* zp, int64_t N, int64_t K, uint16_t* y, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const int splits = gemm_splits(M, N, K, workspace, workspace_bytes);
  unsigned int* counters = static_cast<unsigned int*>(workspace);
  float* partials = splits > 1 ? reinterpret_cast<float*>(static_cast<char*>(workspace) + counter_bytes(tiles))
                               : nullptr;
  gemm_kernel<Q, G, ZP><<<dim3((unsigned)(tiles * splits)), 256, 0, stream>>>(
      x, (int)M, codes, scales, zp, (int)N, (int)K, y, splits, partials, counters);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const uint16_t* x, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, const uint8_t* zp, int64_t N, int64_t K,
                            int group, int q, uint16_t* y, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  SSQ_DISPATCH_QGZ(gemm_dispatch, q, group, zp != nullptr, x, M, codes, scales, zp, N, K, y,
                   workspace, workspace_bytes, stream);
}

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  return (size_t)workspace_for(M, N, K, desired_splits(M, N, K));
}

}  // namespace ssq
