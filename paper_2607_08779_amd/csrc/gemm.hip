// Prefill GEMM: y[M,N] = x[M,K] * What[N,K]^T with What dequantized into LDS.
//
// App. B.3 of the paper: What[n,k] = s[n,b] (u[n,k] - o[n,b]).  Prefill is a
// dense contraction, so it runs on bf16 MFMA.  A workgroup of 2*WM wavefronts owns
// a (64*WM) x 128 output tile, each wavefront a 64x64 sub-tile of
// v_mfma_f32_16x16x32_bf16 (fp32 accumulation).  Per 64-deep step the activation
// tile and the weight codes are loaded into registers several steps ahead; one step
// ahead the activations are written to an LDS ring and the codes dequantized
// (s*(u - o), exact in fp32, rounded to bf16) into a second one; one barrier per step.
// WM=4 uses the full 160 KB of LDS (one workgroup per CU, a four-stage activation
// ring); WM=2 fits two workgroups per CU.
//
// MFMA operand layout (16x16x32): lane l supplies row (l % 16) of A and column
// (l % 16) of B, each with 8 consecutive k values starting at 8 * (l / 16).
// Both operands use the same k assignment, so the reduction is correct for any
// internal k order.  Lane l receives D[4 * (l / 16) + r][l % 16], r = 0..3.
#include <algorithm>
#include <type_traits>
#include <utility>

#include "ssq_internal.h"
#include "mfma_dequant.h"

namespace ssq {
namespace {


constexpr int BN = 128, BK = 64;
constexpr int kBTileBytes = BN * BK * 2;     // 16 KB: 128 rows of 128 bytes
constexpr int kBStages = 2;

template <int WM>
struct Cfg {
  static constexpr int BM = 64 * WM;                    // output rows per tile
  static constexpr int kWaves = 2 * WM;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kAStages = WM == 2 ? 3 : 4;      // 80 KB or 160 KB of LDS in total
  static constexpr int kAhead = kAStages - 1;           // steps of loads in flight
  static constexpr int kATileBytes = BM * BK * 2;
  static constexpr int kParts = kThreads / 256;         // threads per 32-weight block
  static constexpr int kLds = kAStages * kATileBytes + kBStages * kBTileBytes;
};

// Byte offset of 16-byte chunk c (8 bf16 along k) of row r in a tile.  The chunk index
// is XOR-swizzled with r/2: an MFMA operand read touches 16 consecutive rows at one k
// offset, and LDS serves 16 lanes of a 16-byte read per cycle across 256 bytes of banks,
// so two neighbouring 128-byte rows share a bank line; r/2 sends each pair to its own
// eighth of it (no padding needed).
__device__ __forceinline__ uint32_t swz(int r, int c) { return (uint32_t)(r * 128 + ((c ^ ((r >> 1) & 7)) << 4)); }

// Work order.  Workgroups are dealt round-robin to the 8 XCDs (blockIdx % 8), each XCD
// with its own L2.  When the work items divide evenly, XCD x takes a contiguous run of
// them.  Without a split the items are output tiles in N-panel-major order (all M
// tiles of one weight panel together), so a weight panel's codes are fetched once per
// XCD and shared through its L2.  With a split the K slices of one tile come first,
// then the N tiles of one M tile: an XCD then holds one activation tile (or a few)
// against a run of weight panels, and the slices of a tile meet on one XCD.  Both
// orders were chosen by measurement on the Llama3-8B MLP shapes.
__device__ __forceinline__ void work_item(int b, int tiles_m, int tiles_n, int splits, int& tm, int& tn,
                                          int& split) {
  const int items = tiles_m * tiles_n * splits;
  if (items % 8 == 0) b = (b % 8) * (items / 8) + b / 8;
  // split fastest, then the inner tile index, then the outer one
  const bool n_inner = splits > 1;
  const int inner_count = n_inner ? tiles_n : tiles_m;
  split = b % splits;
  const int rest = b / splits;
  const int inner = rest % inner_count, outer = rest / inner_count;
  tm = n_inner ? outer : inner;
  tn = n_inner ? inner : outer;
}

// ---------------------------------------------------------------------------
// Split reduction (host side).  When the output has too few tiles to give every CU
// a workgroup, the K steps of each tile are divided among `splits` workgroups whose
// fp32 partial tiles meet in a caller-provided workspace: [counters: one u32 per
// tile, in the fixed counter region][partials: tiles x splits x BM x BN fp32].
// ---------------------------------------------------------------------------
constexpr int kMinStepsPerSplit = 16;



struct Plan {
  int wm;            // wave rows (tile height 64*wm)
  int64_t tiles;
  int splits;
  int64_t workspace; // bytes needed when splits > 1
};

Plan plan_for(int64_t M, int64_t N, int64_t K) {
  Plan p{};
  p.wm = M > 128 ? 4 : 2;                                 // 256-row tiles unless M is small
  const int64_t bm = 64 * p.wm;
  p.tiles = ((M + bm - 1) / bm) * ((N + BN - 1) / BN);
  const int64_t steps = (K / 32 + 1) / 2;
  // enough workgroups to fill every CU (one per CU at wm=4, two at wm=2)
  int64_t s = (p.wm == 4 ? 256 : 512) / p.tiles;
  s = std::min<int64_t>(s, steps / kMinStepsPerSplit);
  s = std::min<int64_t>(s, 8);
  if (p.tiles > kMaxSplitCounters) s = 1;
  p.splits = (int)std::max<int64_t>(s, 1);
  p.workspace = p.splits > 1 ? kSplitCounterBytes + p.tiles * p.splits * bm * BN * 4 : 0;
  return p;
}

template <int Q, int G, int META, int WM>
__global__ __launch_bounds__(Cfg<WM>::kThreads) void gemm_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const void* __restrict__ meta, int M, int N, int K, int splits, uint16_t* __restrict__ y,
    float* __restrict__ partials, unsigned int* __restrict__ counters) {
  using C = Cfg<WM>;
  constexpr int BM = C::BM, P = C::kParts, S = C::kAStages, D = C::kAhead;
  // Activation stages: one LDS object each, named with compile-time indices only.
  __shared__ __attribute__((aligned(1024))) uint8_t A0[C::kATileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t A1[C::kATileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t A2[C::kATileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t Bs[kBStages * kBTileBytes];
  auto a_tile = [&](auto stage) -> uint8_t* {
    constexpr int i = decltype(stage)::value;
    static_assert(i < S, "stage index");
    if constexpr (i == 0) return A0;
    else if constexpr (i == 1) return A1;
    else if constexpr (i == 2) return A2;
    else {
      __shared__ __attribute__((aligned(1024))) uint8_t A3[C::kATileBytes];
      return A3;
    }
  };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar offsets
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int tiles = tiles_m * tiles_n;
  int tm, tn, split;
  work_item((int)blockIdx.x, tiles_m, tiles_n, splits, tm, tn, split);
  const int tile_id = tm * tiles_n + tn;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int nblk = K / 32;
  const int total_steps = (nblk + 1) / 2;
  // This workgroup's slice of the reduction: steps [s_begin, s_begin + nsteps).
  const int per_split = (total_steps + splits - 1) / splits;
  const int s_begin = split * per_split;
  const int nsteps = total_steps - s_begin < per_split ? total_steps - s_begin : per_split;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)(K / G);
  constexpr bool ZP = META != kMetaNone;
  constexpr int kMetaSize = meta_size<META>();
  const uint8_t* const zp = static_cast<const uint8_t*>(meta);
  constexpr int kLoadsPerStep = 4 + 2 + (ZP ? 1 : 0);

  // Buffer descriptors relative to the tile's first row; rows past M or N read zeros.
  const uint32_t rows_a = (uint32_t)(M - m0 < BM ? M - m0 : BM);
  const uint32_t rows_b = (uint32_t)(N - n0 < BN ? N - n0 : BN);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(x + m0 * K, rows_a * (uint32_t)K * 2);
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes + n0 * row_bytes, rows_b * row_bytes);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(scales + n0 * groups_per_row, rows_b * groups_per_row * 2);
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(ZP ? zp + n0 * groups_per_row * kMetaSize : zp,
                                              ZP ? rows_b * groups_per_row * kMetaSize : 0);

  // Activation tile: BM/8 wavefront loads of 1 KB straight into LDS, four per wave.
  // Load j fills tile rows 8j..8j+7, lane i writing 16 bytes at 16*i, which is row
  // 8j + i/8, swizzled chunk i%8 -- so lane i fetches logical chunk (i%8)^((row/2)%8).
  uint32_t a_off[4];
  int a_chunk[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = 8 * (4 * wave + j) + (lane >> 3);
    a_chunk[j] = (lane & 7) ^ ((r >> 1) & 7);
    a_off[j] = (uint32_t)r * K * 2 + a_chunk[j] * 16;
  }
  // Activations go through registers: loaded D steps ahead, written to their stage one
  // step before use (every wait is then one the compiler places on a register it needs).
  u32x4 a_reg[S][4];
  auto issue_a = [&](int lstep, int slot) {
    const int step = s_begin + lstep;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // chunks past this slice or past K (odd block count, last step) read zeros
      const bool in = (lstep < nsteps) & (step * 64 + a_chunk[j] * 8 < K);
      const uint32_t off = in ? a_off[j] + (uint32_t)step * 128 : 0x80000000u;
      a_reg[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(ra, off, 0, kStream);
    }
  };
  auto store_a = [&](int slot, auto stage) {
    uint8_t* const at = a_tile(stage);
#pragma unroll
    for (int j = 0; j < 4; ++j) *reinterpret_cast<u32x4*>(at + (4 * wave + j) * 1024 + lane * 16) = a_reg[slot][j];
  };

  // Weight tile: P threads share each 32-weight block; block (t/P) % 2 of row t/(2P).
  const int bid = tid / P, part = tid % P;
  const int lr = bid >> 1, lh = bid & 1;
  const uint32_t c_off = (uint32_t)lr * row_bytes + lh * (4 * Q);
  uint32_t c_reg[S][Part<Q, P>::kDwords], s_reg[S], z_reg[S];
  auto issue_b = [&](int lstep, int slot) {
    const int step = s_begin + lstep;
    const int blk = 2 * step + lh;
    const bool in = (lstep < nsteps) & (blk < nblk);
    uint32_t d[Part<Q, P>::kDwords];
    load_part<Q, P>(rc, in ? c_off + (uint32_t)step * (8 * Q) : 0x80000000u, part, d);
#pragma unroll
    for (int i = 0; i < Part<Q, P>::kDwords; ++i) c_reg[slot][i] = d[i];
    const uint32_t gi = (uint32_t)lr * groups_per_row + (uint32_t)(blk / (G / 32));
    s_reg[slot] = __builtin_amdgcn_raw_buffer_load_b16(rs, in ? gi * 2 : 0x80000000u, 0, 0);
    if constexpr (ZP) z_reg[slot] = load_group_meta<META>(rz, gi, in);
  };
  auto store_b = [&](int slot, int stage) {
    const float s = f16_bits_to_f32(s_reg[slot]);
    uint32_t w[16 / P];
    dequant_part<Q, P>(c_reg[slot], part, s, dequant_offset<META, Q>(s, ZP ? z_reg[slot] : 0u), w);
    uint8_t* dst = Bs + stage * kBTileBytes;
#pragma unroll
    for (int e = 0; e < 4 / P; ++e)
      *reinterpret_cast<uint4*>(dst + swz(lr, lh * 4 + (4 / P) * part + e)) =
          uint4{w[4 * e], w[4 * e + 1], w[4 * e + 2], w[4 * e + 3]};
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  auto mfma_step = [&](int step, auto stage) {
    const uint8_t* at = a_tile(stage);
    const uint8_t* bt = Bs + (step % kBStages) * kBTileBytes;
    // LLVM's MFMA/DS-read interleaving strategy for this loop shape (measured ~7 % faster)
    __builtin_amdgcn_iglp_opt(1);
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

  // Step s (position p = s % S in a group of S steps): issue the loads of step s+D into
  // slot (p+D) % S, multiply stage p, dequantize the codes of step s+1 and write its
  // activations (slot (p+1) % S) to its weight and activation stages, barrier.  Every
  // step issues and stores unconditionally -- past the slice the loads are out of range
  // and return zeros -- and the loop runs whole groups of S steps (static stages and
  // slots) with no exit between a load and its use; the last nsteps % S steps follow.
  // Stage (p+1) % S was last read S-1 steps ago, before an earlier barrier; the barrier
  // publishes step s+1's tiles.
  auto step_body = [&](int s, auto pos) {
    constexpr int p = decltype(pos)::value;
    constexpr int kLoad = (p + D) % S;
    constexpr int kNext = (p + 1) % S;
    issue_a(s + D, kLoad);
    issue_b(s + D, kLoad);
    __builtin_amdgcn_sched_barrier(0);       // the loads go out first
    mfma_step(s, pos);
    store_b(kNext, (s + 1) % kBStages);
    store_a(kNext, std::integral_constant<int, kNext>{});
    __syncthreads();
  };

  [&]<int... L>(std::integer_sequence<int, L...>) {
    ((issue_a(L, L), issue_b(L, L)), ...);
  }(std::make_integer_sequence<int, D>{});
  store_b(0, 0);
  store_a(0, std::integral_constant<int, 0>{});
  __syncthreads();
  int s = 0;
  for (; s + S <= nsteps; s += S) {
    [&]<int... L>(std::integer_sequence<int, L...>) {
      (step_body(s + L, std::integral_constant<int, L>{}), ...);
    }(std::make_integer_sequence<int, S>{});
  }
  [&]<int... L>(std::integer_sequence<int, L...>) {
    ((s + L < nsteps ? step_body(s + L, std::integral_constant<int, L>{}) : void()), ...);
  }(std::make_integer_sequence<int, S - 1>{});

  if (splits > 1) {
    // Split reduction: publish this slice's fp32 partial tile in the lane order of the
    // accumulators (coalesced), then count arrivals; the last arriving workgroup sums
    // all slices in a fixed order, writes y and resets the counter so the workspace
    // stays reusable.
    //
    // Coherence across XCDs: the partials are written and read only with device-scope
    // atomic stores and loads (sc1), which write through to memory and read from it
    // rather than from this XCD's L2.  A store's vmcnt is released only once memory has
    // acknowledged it, so after the wait below every partial of this slice is visible
    // device-wide before the arrival count (a device-coherent RMW) is bumped, and the
    // last workgroup's loads, issued after it has read the count, see them.  A general
    // device-scope fence would instead write back the whole L2 of the XCD in every
    // workgroup (tens of microseconds once many fp32 partials are dirty in it).
    float* mine = partials + ((int64_t)tile_id * splits + split) * (BM * BN) + wave * 4096 + lane;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          __hip_atomic_store(mine + ((i * 4 + j) * 4 + r) * 64, acc[i][j][r], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    wait_vmcnt<0>();                       // every partial store acknowledged by memory
    // The tile buffers are idle after the main loop; their first word carries the arrival
    // count to the whole workgroup (a separate shared variable would push LDS past the
    // per-CU budget the ring sizes are chosen for).
    unsigned int* arrived = reinterpret_cast<unsigned int*>(Bs);
    __syncthreads();
    if (tid == 0) *arrived = atomicAdd(&counters[tile_id], 1u);
    __syncthreads();
    if (*arrived != (unsigned int)(splits - 1)) return;   // uniform across the workgroup
    // Sum every slice (this one included) in slice order, so the result does not depend
    // on which workgroup arrived last.
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int o = 0; o < splits; ++o) {
      const float* part_o = partials + ((int64_t)tile_id * splits + o) * (BM * BN) + wave * 4096 + lane;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            acc[i][j][r] += __hip_atomic_load(part_o + ((i * 4 + j) * 4 + r) * 64, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
    }
    if (tid == 0) __hip_atomic_store(&counters[tile_id], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

template <int Q, int G, int META>
hipError_t gemm_dispatch(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                         const void* zp, int64_t N, int64_t K, uint16_t* y, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  const Plan p = plan_for(M, N, K);
  const bool split = p.splits > 1 && workspace != nullptr && (int64_t)workspace_bytes >= p.workspace;
  const int splits = split ? p.splits : 1;
  unsigned int* counters = static_cast<unsigned int*>(workspace);
  float* partials = split ? reinterpret_cast<float*>(static_cast<char*>(workspace) + kSplitCounterBytes)
                          : nullptr;
  const dim3 grid((unsigned)(p.tiles * splits));
  if (p.wm == 4)
    gemm_kernel<Q, G, META, 4><<<grid, Cfg<4>::kThreads, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N,
                                                                   (int)K, splits, y, partials, counters);
  else
    gemm_kernel<Q, G, META, 2><<<grid, Cfg<2>::kThreads, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N,
                                                                   (int)K, splits, y, partials, counters);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const uint16_t* x, int64_t M, const uint8_t* codes,
                            const uint16_t* scales, GroupMeta meta, int64_t N, int64_t K,
                            int group, int q, uint16_t* y, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  SSQ_DISPATCH_QGM(gemm_dispatch, q, group, meta.kind, x, M, codes, scales, meta.ptr, N, K, y,
                   workspace, workspace_bytes, stream);
}

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) { return (size_t)plan_for(M, N, K).workspace; }

}  // namespace ssq
