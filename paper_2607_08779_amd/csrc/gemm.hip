// Prefill GEMM: y[M,N] = x[M,K] * What[N,K]^T on bf16 MFMA.
//
// App. B.3 of the paper: What[n,k] = s[n,b] (u[n,k] - o[n,b]).  Prefill is a dense
// contraction, so it runs on v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
//
// Work split.  A wavefront owns a 128 (M) x 64 (N) output tile: 4 x 2 MFMA tiles of
// 32 x 32, 128 fp32 accumulators per lane.  Only the activations and the packed weights
// go through LDS; each wavefront dequantizes its own 64 weight rows straight into MFMA B
// operands, so dequantized weights never cost LDS bandwidth.  A workgroup holds two
// K-groups of 2*WM wavefronts (WM x 2 wave tiles: a (128*WM) x 128 output tile; WM = 2
// unless M <= 128): K-group g
// takes the 64-deep steps of parity g, so two wavefronts share each SIMD without
// doubling the tile, and their accumulators meet in LDS at the end.  A "window" is one
// step per K-group: its activation tiles (two stages) and its weight stage are read from
// one half of their LDS rings while the next window's are loaded straight into the
// other half (direct-to-LDS buffer loads, shared by the workgroup); one barrier per
// window.  On gfx950 the matrix cores and the vector ALU of a SIMD do not run at the
// same time (measured: an MFMA stream and a VALU stream take the sum of their times, in
// one wavefront or in two), so the dequantization arithmetic adds to the MFMA time.
//
// Reduction order inside a step.  Lane l covers weight row l % 32 of an MFMA tile;
// lanes 0-31 take the step's first 32-weight block, lanes 32-63 the second.  MFMA j
// (j = 0..3) of the step consumes weights 8j..8j+7 of each lane's block, so one lane
// dequantizes exactly one block per 32-row tile (one 4q-byte code load).  The
// activation operand follows the same assignment: lane l supplies row l % 32 of its
// M tile at k = 64 s + 32 (l / 32) + 8 j + (0..7).  An MFMA sums over whatever k each
// operand slot stands for, as long as A and B agree, so this order is exact.
//
// MFMA layouts (32x32x16 bf16): A lane l = row l % 32, 8 consecutive k of half l / 32;
// B lane l = column l % 32, the same k; D register r of lane l = row 8 (r / 4) +
// 4 (l / 32) + r % 4, column l % 32.
#include <algorithm>
#include <type_traits>
#include <utility>

#include "ssq_internal.h"
#include "mfma_dequant.h"

namespace ssq {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BN = 128;                  // output columns per workgroup tile
constexpr int kStages = 4;               // activation ring: two windows of two steps

template <int WM>
struct Cfg {
  static constexpr int BM = 128 * WM;                   // output rows per workgroup tile
  static constexpr int kGroupWaves = 2 * WM;            // wavefronts per K-group
  static constexpr int kWaves = 2 * kGroupWaves;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kStageBytes = BM * 128;          // BM rows x 64 bf16
  static constexpr int kLds = kStages * kStageBytes;    // 128 KB (WM = 2) or 64 KB (WM = 1)
  // b128 activation loads per thread per window: two stages of BM x 8 chunks
  static constexpr int kALoads = 2 * BM * 8 / kThreads;
  static_assert(kALoads == 8, "each thread stages 128 bytes of a window's activations");
  // The K-groups swap halves of their accumulators through LDS after the main loop.
  static_assert(kWaves * 64 * 64 * 4 <= kLds, "exchange fits the activation ring");
};

// Byte offset of 16-byte chunk c (8 bf16 along k) of row r in an activation stage.  The
// chunk index is XOR-swizzled with r/2: an operand read touches 16 consecutive rows at
// one k offset per LDS cycle, and 256 bytes of banks span two 128-byte rows, so r/2
// sends each row pair to its own sixteenth of the banks (no padding needed).
__device__ __forceinline__ uint32_t swz(int r, int c) { return (uint32_t)(r * 128 + ((c ^ ((r >> 1) & 7)) << 4)); }

// 8 weights s*(u - o) of slice j (weights 8j..8j+7) of a 32-weight block held in q
// dwords, natural order, as four bf16 pairs.  Each q-bit field is OR-ed into the
// mantissa of the fp16 constant 1024 (0x6400 | u == 1024 + u), two fields per
// instruction; one v_fma_mix_f32 per weight forms (1024 + u)*s + so with
// so = -(1024 + o)*s (or m - 1024 s), both products exact in fp32, so the weight is
// s*(u - o) exactly; it is rounded to bf16 once.
template <int Q>
__device__ __forceinline__ bf16x8 dequant_slice(const uint32_t (&d)[Q], int j, float s, float so) {
  const uint32_t magic = 0x64006400u;
  uint32_t sp;          // fields 0..3 of the slice at bit 0, fields 4..7 at bit 16
  if constexpr (Q == 4) {
    sp = d[j];          // field i at bits 4i: and_or(sp >> 4i) pairs fields i and i+4
  } else if constexpr (Q == 2) {
    const uint32_t h = d[j >> 1] >> (16 * (j & 1));              // 8 fields in bits 0..15
    sp = __builtin_amdgcn_perm(0u, h, 0x0c010c00u);               // bytes: f0-3 at 0, f4-7 at 16
  } else {
    // 24-bit word j of the 96-bit block; fields 4..7 move up to bit 16
    const uint32_t w = j == 0 ? d[0]
                     : j == 1 ? __builtin_amdgcn_alignbit(d[1], d[0], 24)
                     : j == 2 ? __builtin_amdgcn_alignbit(d[2], d[1], 16)
                              : d[2] >> 8;
    sp = (w & 0xFFFu) | ((w << 4) & 0x0FFF0000u);
  }
  float f[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t p = and_or(sp >> (Q * i), Q == 4 ? 0x000F000Fu : Q == 3 ? 0x00070007u : 0x00030003u, magic);
    f[i] = __builtin_fmaf(f16_lo(p), s, so);
    f[i + 4] = __builtin_fmaf(f16_hi(p), s, so);
  }
  const uint32_t w0 = pack_bf16x2(f[0], f[1]), w1 = pack_bf16x2(f[2], f[3]);
  const uint32_t w2 = pack_bf16x2(f[4], f[5]), w3 = pack_bf16x2(f[6], f[7]);
  return __builtin_bit_cast(bf16x8, u32x4{w0, w1, w2, w3});
}

// Codes of one 32-weight block (4q bytes) through a buffer descriptor.
template <int Q>
__device__ __forceinline__ void load_block(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t (&d)[Q]) {
  if constexpr (Q == 4) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  } else if constexpr (Q == 3) {
    const u32x3 v = __builtin_amdgcn_raw_buffer_load_b96(r, (int)off, 0, 0);
    d[0] = v.x; d[1] = v.y; d[2] = v.z;
  } else {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
    d[0] = v.x; d[1] = v.y;
  }
}

// Work order.  Workgroups are dealt round-robin to the 8 XCDs (blockIdx % 8), each with
// its own L2; when the work items divide evenly, XCD x takes a contiguous run of them.
// Without a split the items are output tiles with the M tiles of one weight panel
// together (a panel's codes are fetched once per XCD); with a split the K slices of a
// tile come first, then the N tiles of one M tile (an XCD holds one activation panel
// against a run of weight panels, and the slices of a tile meet on one XCD).
__device__ __forceinline__ void work_item(int b, int tiles_m, int tiles_n, int splits, int& tm, int& tn,
                                          int& split) {
  const int items = tiles_m * tiles_n * splits;
  if (items % 8 == 0) b = (b % 8) * (items / 8) + b / 8;
  const bool n_inner = splits > 1;
  const int inner_count = n_inner ? tiles_n : tiles_m;
  split = b % splits;
  const int rest = b / splits;
  const int inner = rest % inner_count, outer = rest / inner_count;
  tm = n_inner ? outer : inner;
  tn = n_inner ? inner : outer;
}

// ---------------------------------------------------------------------------
// Split reduction (host side).  When the output has too few tiles to give every CU a
// workgroup, the K steps of each tile are divided among `splits` workgroups whose fp32
// partial tiles meet in a caller-provided workspace: [counters: one u32 per tile, in the
// fixed counter region][partials: tiles x splits x BM x BN fp32].
// ---------------------------------------------------------------------------
constexpr int kMinStepsPerSplit = 16;

struct Plan {
  int wm;            // wave tiles along M (tile height 128*wm)
  int64_t tiles;
  int splits;
  int64_t workspace; // bytes needed when splits > 1
};

Plan plan_for(int64_t M, int64_t N, int64_t K) {
  Plan p{};
  p.wm = M > 128 ? 2 : 1;
  const int64_t bm = 128 * p.wm;
  p.tiles = ((M + bm - 1) / bm) * ((N + BN - 1) / BN);
  const int64_t steps = (K / 32 + 1) / 2;
  // one workgroup per CU (WM = 2: 128 KB of LDS) or two (WM = 1)
  int64_t s = (p.wm == 2 ? 256 : 512) / p.tiles;
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
  constexpr int BM = C::BM;
  // Four activation stages, each its own LDS object: the compiler then knows that the
  // direct-to-LDS loads filling one stage do not alias the operand reads of another, and
  // does not make those reads wait for them.  The stages are contiguous, so the exchange
  // after the main loop addresses them as one array from the first.
  __shared__ __attribute__((aligned(1024))) uint8_t st0[C::kStageBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st1[C::kStageBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st2[C::kStageBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st3[C::kStageBytes];
  auto stage = [&](auto idx) -> uint8_t* {
    constexpr int i = decltype(idx)::value;
    if constexpr (i == 0) return st0;
    else if constexpr (i == 1) return st1;
    else if constexpr (i == 2) return st2;
    else return st3;
  };
  auto stage_dyn = [&](int i) -> uint8_t* { return i == 0 ? st0 : i == 1 ? st1 : i == 2 ? st2 : st3; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar offsets
  const int grp = wave / C::kGroupWaves;                       // K-group: steps of parity grp
  const int wp = wave % C::kGroupWaves;
  const int wm = wp >> 1, wn = wp & 1;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  int tm, tn, split;
  work_item((int)blockIdx.x, tiles_m, tiles_n, splits, tm, tn, split);
  const int tile_id = tm * tiles_n + tn;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int nblk = K / 32;
  const int total_steps = (nblk + 1) / 2;
  // This workgroup's slice of the reduction: steps [s_begin, s_begin + nsteps), in
  // windows of two (the last window's odd step may lie past the slice: it reads zeros).
  const int per_split = (total_steps + splits - 1) / splits;
  const int s_begin = split * per_split;
  const int nsteps = total_steps - s_begin < per_split ? total_steps - s_begin : per_split;
  const int nwin = (nsteps + 1) / 2;
  const uint32_t row_bytes = (uint32_t)K * Q / 8;
  const uint32_t groups_per_row = (uint32_t)(K / G);
  constexpr bool ZP = META != kMetaNone;
  constexpr int kMetaSize = meta_size<META>();
  const uint8_t* const zp = static_cast<const uint8_t*>(meta);

  // Activation buffer descriptor relative to the tile's first row; rows past M read zeros.
  const uint32_t rows_a = (uint32_t)(M - m0 < BM ? M - m0 : BM);
  const int64_t nw0 = n0 + wn * 64;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(x + m0 * K, rows_a * (uint32_t)K * 2);

  // Activation staging: thread t loads 8 chunks of 16 bytes of stage e = t / (threads/2)
  // of the next window, rows 8 at a time: load i of wavefront v fills rows 8 (8 v' + i) ..
  // +7 (v' = v mod threads/128), lane L writing 16 bytes at 16 L of that 1 KB, i.e. row
  // r_i = 64 v' + 8 i + L/8, swizzled chunk L % 8, so lane L fetches logical chunk
  // (L % 8) ^ ((r_i/2) % 8) = (L % 8) ^ (L/16 + 4 (i % 2)): two chunk columns, one per
  // parity of i.
  constexpr int kStageWaves = C::kWaves / 2;
  const int a_e = wave / kStageWaves;
  const int a_w = wave % kStageWaves;
  const int a_c0 = (lane & 7) ^ (lane >> 4), a_c1 = a_c0 ^ 4;
  const uint32_t a_row = (uint32_t)(64 * a_w + (lane >> 3)) * (uint32_t)K * 2;
  const uint32_t a_b0 = a_row + a_c0 * 16, a_b1 = a_row + a_c1 * 16;
  auto issue_a = [&](int win, auto pair_c) {
    constexpr int pair = decltype(pair_c)::value;
    const uint32_t col = (uint32_t)(s_begin + 2 * win + a_e) * 128u;
    auto fill = [&](uint8_t* st) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            ra, (__attribute__((address_space(3))) void*)(st + a_w * 8192 + i * 1024), 16,
            ((i & 1) ? a_b1 : a_b0) + ((uint32_t)i * 16u * (uint32_t)K + col), 0, 0, 0);
    };
    if (a_e == 0) fill(stage(std::integral_constant<int, 2 * pair>{}));
    else fill(stage(std::integral_constant<int, 2 * pair + 1>{}));
  };
  // Weight stage of a window, filled by direct-to-LDS loads that the workgroup shares
  // (the wavefronts of both M halves read the same rows): codes of the window's four
  // blocks of all BN rows (16q bytes per row: Cq 16-byte chunks), and for each row the
  // dword-aligned 16 bytes of scales (and zero points or minimums) that contain the
  // window's groups.  Rows past N and windows past the slice read zeros.
  // q = 3 rows take four chunks too (48 of the 64 bytes are the window's), so that every
  // lane of every load owns its own 16 bytes of the stage.
  constexpr int Cq = Q == 2 ? 2 : 4;                        // 16-byte code chunks per row
  constexpr int Rq = 64 / Cq;                               // rows per load instruction
  constexpr int kCodeLoads = BN / Rq;                       // 8 or 4
  constexpr int kCodeBytes = BN * Cq * 16;
  static_assert(Rq * Cq == 64 && BN % Rq == 0, "loads tile the stage exactly");
  constexpr int kCodeRounds = (kCodeLoads + C::kWaves - 1) / C::kWaves;   // code loads per wavefront
  static_assert(2 + (ZP ? 2 : 0) <= C::kWaves, "one scale or metadata load per wavefront");
  __shared__ __attribute__((aligned(1024))) uint8_t bc0[kCodeBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t bc1[kCodeBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t bs0[BN * 16];
  __shared__ __attribute__((aligned(1024))) uint8_t bs1[BN * 16];
  __shared__ __attribute__((aligned(1024))) uint8_t bm0[ZP ? BN * 16 : 16];
  __shared__ __attribute__((aligned(1024))) uint8_t bm1[ZP ? BN * 16 : 16];
  auto bstage = [&](auto idx, int which) -> uint8_t* {   // which: 0 codes, 1 scales, 2 metadata
    constexpr int i = decltype(idx)::value;
    if (which == 0) return i == 0 ? bc0 : bc1;
    if (which == 1) return i == 0 ? bs0 : bs1;
    return i == 0 ? bm0 : bm1;
  };
  // The scale and metadata descriptors start at the dword boundary at or below the tile's
  // first entry (`shift` bytes earlier, inside the same allocation), so that every
  // 16-byte piece these loads fetch is dword aligned, and end at the dword boundary at or
  // above the last entry: the range check is per dword, and a dword that straddles the
  // end would read as zero.  The few bytes past the end share the last entry's page.
  const uint32_t rows_wg = (uint32_t)(N - n0 < BN ? N - n0 : BN);
  const __amdgpu_buffer_rsrc_t rcw = make_rsrc(codes + n0 * row_bytes, rows_wg * row_bytes);
  const uint8_t* const s_first = reinterpret_cast<const uint8_t*>(scales + n0 * groups_per_row);
  const uint32_t s_shift = (uint32_t)(reinterpret_cast<uintptr_t>(s_first) & 3u);
  const __amdgpu_buffer_rsrc_t rsw = make_rsrc(s_first - s_shift, (s_shift + rows_wg * groups_per_row * 2 + 3) & ~3u);
  const uint8_t* const m_first = ZP ? zp + n0 * groups_per_row * kMetaSize : zp;
  const uint32_t m_shift = ZP ? (uint32_t)(reinterpret_cast<uintptr_t>(m_first) & 3u) : 0u;
  const __amdgpu_buffer_rsrc_t rzw = make_rsrc(ZP ? m_first - m_shift : zp,
                                               ZP ? (m_shift + rows_wg * groups_per_row * kMetaSize + 3) & ~3u : 0);
  // Code chunk of lane L in load i: row i*Rq + L/Cq, physical chunk L % Cq, which holds
  // logical chunk (L % Cq) ^ ((row/4) % 4) at q = 4 (so that the operand reads of 16
  // consecutive rows hit distinct banks) and L % Cq otherwise.
  auto issue_bstage = [&](int win, auto pair_c) {
    const uint32_t blk0 = 2u * (uint32_t)(s_begin + 2 * win);          // first block of the window
#pragma unroll
    for (int k = 0; k < kCodeRounds; ++k) {
      const int li = wave + k * C::kWaves;                               // load index
      if (li < kCodeLoads) {
        const int row = li * Rq + lane / Cq;
        const int chunk = Q == 4 ? ((lane % Cq) ^ ((row >> 2) & 3)) : lane % Cq;
        const uint32_t off = (uint32_t)row * row_bytes + blk0 * (4 * Q) + (uint32_t)chunk * 16;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rcw, (__attribute__((address_space(3))) void*)(bstage(pair_c, 0) + li * (Rq * Cq * 16)), 16,
            off, 0, 0, 0);
      }
    }
    const uint32_t g0 = blk0 / (G / 32);                                 // first group of the window
    const int r = 64 * (wave & 1) + lane;
    if (wave < 2) {
      const uint32_t off = (s_shift + ((uint32_t)r * groups_per_row + g0) * 2u) & ~3u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsw, (__attribute__((address_space(3))) void*)(bstage(pair_c, 1) + (wave & 1) * 1024), 16,
          off, 0, 0, 0);
    } else if (ZP && wave < 4) {
      const uint32_t off = (m_shift + ((uint32_t)r * groups_per_row + g0) * kMetaSize) & ~3u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rzw, (__attribute__((address_space(3))) void*)(bstage(pair_c, 2) + (wave & 1) * 1024), 16,
          off, 0, 0, 0);
    }
  };

  // Weights: lane l dequantizes block 2*step + h (h = l / 32) of rows l % 32 and
  // 32 + l % 32 of this wavefront's 64, reading codes, scale and metadata from the stage.
  const int h = lane >> 5, lr = lane & 31;
  const int kblk = 2 * grp + h;                  // the lane's block within a window (0..3)

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][c][r] = 0.0f;

  // This K-group's step of window `win`: activation stage at `at`, weight stage `pair`.
  auto compute = [&](const uint8_t* at, int win, auto pair_c) {
    const uint8_t* bc = bstage(pair_c, 0);
    const uint8_t* bs = bstage(pair_c, 1);
    const uint8_t* bm = bstage(pair_c, 2);
    const uint32_t blk = 2u * (uint32_t)(s_begin + 2 * win) + (uint32_t)kblk;
    // a block past the slice or past K weighs zero: scale and metadata forced to 0
    const bool valid = (2 * win + grp < nsteps) & (blk < (uint32_t)nblk);
    const uint32_t g0 = (2u * (uint32_t)(s_begin + 2 * win)) / (G / 32), gi = blk / (G / 32);
    uint32_t cw[2][Q];
    float s[2], so[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int row = wn * 64 + 32 * c + lr;
      if constexpr (Q == 4) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(bc + (row * 4 + (kblk ^ ((row >> 2) & 3))) * 16);
        cw[c][0] = v.x; cw[c][1] = v.y; cw[c][2] = v.z; cw[c][3] = v.w;
      } else if constexpr (Q == 3) {
        const uint32_t* p3 = reinterpret_cast<const uint32_t*>(bc + row * 64 + kblk * 12);
        cw[c][0] = p3[0]; cw[c][1] = p3[1]; cw[c][2] = p3[2];
      } else {
        const u32x2 v = *reinterpret_cast<const u32x2*>(bc + row * 32 + kblk * 8);
        cw[c][0] = v.x; cw[c][1] = v.y;
      }
      const uint32_t rbase = (uint32_t)row * groups_per_row;
      const uint32_t s_in = s_shift + (rbase + gi) * 2u - ((s_shift + (rbase + g0) * 2u) & ~3u);
      const uint32_t sbits = valid ? (uint32_t)*reinterpret_cast<const uint16_t*>(bs + row * 16 + s_in) : 0u;
      uint32_t mbits = 0u;
      if constexpr (ZP) {
        const uint32_t m_in = m_shift + (rbase + gi) * kMetaSize - ((m_shift + (rbase + g0) * kMetaSize) & ~3u);
        const uint32_t raw = META == kMetaMin ? (uint32_t)*reinterpret_cast<const uint16_t*>(bm + row * 16 + m_in)
                                              : (uint32_t)bm[row * 16 + m_in];
        mbits = valid ? raw : 0u;
      }
      s[c] = f16_bits_to_f32(sbits);
      so[c] = dequant_offset<META, Q>(s[c], mbits);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      bf16x8 a[4], b[2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(at + swz(wm * 128 + i * 32 + lr, 4 * h + j));
#pragma unroll
      for (int c = 0; c < 2; ++c) b[c] = dequant_slice<Q>(cw[c], j, s[c], so[c]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 2; ++c)
          acc[i][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[c], acc[i][c], 0, 0, 0);
    }
  };

  // Window t: issue the loads of window t+1 (activations and weight stage, straight into
  // the other half of each ring, last read in window t-1, before the previous barrier),
  // multiply this K-group's step of window t, wait for this thread's loads, barrier:
  // every wavefront's part of window t+1's tiles is then in LDS.
  issue_a(0, std::integral_constant<int, 0>{});
  issue_bstage(0, std::integral_constant<int, 0>{});
  wait_vmcnt<0>();
  __syncthreads();
  auto window = [&](int t, auto par) {
    constexpr int p = decltype(par)::value;
    issue_a(t + 1, std::integral_constant<int, 1 - p>{});
    issue_bstage(t + 1, std::integral_constant<int, 1 - p>{});
    __builtin_amdgcn_sched_barrier(0);       // the loads go out before the arithmetic
    compute(grp == 0 ? stage(std::integral_constant<int, 2 * p>{}) : stage(std::integral_constant<int, 2 * p + 1>{}),
            t, std::integral_constant<int, p>{});
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<0>();
    __syncthreads();
  };
  int t = 0;
  for (; t + 2 <= nwin; t += 2) {
    window(t, std::integral_constant<int, 0>{});
    window(t + 1, std::integral_constant<int, 1>{});
  }
  if (t < nwin) window(t, std::integral_constant<int, 0>{});
  wait_vmcnt<0>();     // the last window's (empty) loads, before LDS is reused
  __syncthreads();

  // The K-groups meet: group g keeps M tiles 2g and 2g+1 of its wave tile and hands the
  // other two to its partner (the same wave position in the other group) through LDS;
  // the activation ring is idle after the last barrier.  Layout: 16 KB per wavefront,
  // lane-contiguous 16-byte pieces (conflict-free).  The kept and given tiles are named
  // with compile-time indices (grp is uniform per wavefront, so the branch is too): a
  // runtime index would move the accumulators to scratch memory.
  f32x16 own[2][2];
  auto exchange = [&](auto keep_c) {
    constexpr int keep = decltype(keep_c)::value, give = 2 - keep;
    constexpr int kPerStage = C::kStageBytes / 16384;     // wavefront areas per stage
    float* xo = reinterpret_cast<float*>(stage_dyn(wave / kPerStage)) + (size_t)(wave % kPerStage) * 4096;
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 v = {acc[give + ii][c][4 * q4], acc[give + ii][c][4 * q4 + 1], acc[give + ii][c][4 * q4 + 2],
                           acc[give + ii][c][4 * q4 + 3]};
          *reinterpret_cast<f32x4*>(xo + ((ii * 2 + c) * 4 + q4) * 256 + lane * 4) = v;
        }
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int c = 0; c < 2; ++c) own[ii][c] = acc[keep + ii][c];
  };
  if (grp == 0) exchange(std::integral_constant<int, 0>{});
  else exchange(std::integral_constant<int, 2>{});
  __syncthreads();
  {
    constexpr int kPerStage = C::kStageBytes / 16384;
    const int partner = (1 - grp) * C::kGroupWaves + wp;
    const float* xi = reinterpret_cast<const float*>(stage_dyn(partner / kPerStage)) + (size_t)(partner % kPerStage) * 4096;
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 v = *reinterpret_cast<const f32x4*>(xi + ((ii * 2 + c) * 4 + q4) * 256 + lane * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) own[ii][c][4 * q4 + e] += v[e];
        }
  }
  const int keep = 2 * grp;     // M tiles keep, keep+1 of the wave tile are this wavefront's

  if (splits > 1) {
    // Split reduction: publish this slice's partial (the 64 accumulators this wavefront
    // owns, in lane order: coalesced), then count arrivals; the last arriving workgroup
    // sums all slices in slice order, writes y and resets the counter so the workspace
    // stays reusable.  Partials are written and read with device-scope (sc1) accesses,
    // which go to memory rather than this XCD's L2, so no device-wide fence is needed:
    // a store's vmcnt is released once memory has acknowledged it.
    float* mine = partials + ((int64_t)tile_id * splits + split) * (BM * BN) + (int64_t)wave * 4096 + lane;
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          __hip_atomic_store(mine + ((ii * 2 + c) * 16 + r) * 64, own[ii][c][r], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    wait_vmcnt<0>();                       // every partial store acknowledged by memory
    unsigned int* arrived = reinterpret_cast<unsigned int*>(st0);
    __syncthreads();                       // the exchange above has finished reading LDS
    if (tid == 0) *arrived = atomicAdd(&counters[tile_id], 1u);
    __syncthreads();
    if (*arrived != (unsigned int)(splits - 1)) return;   // uniform across the workgroup
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) own[ii][c][r] = 0.0f;
    for (int o = 0; o < splits; ++o) {
      const float* part_o = partials + ((int64_t)tile_id * splits + o) * (BM * BN) + (int64_t)wave * 4096 + lane;
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            own[ii][c][r] += __hip_atomic_load(part_o + ((ii * 2 + c) * 16 + r) * 64, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
    }
    if (tid == 0) __hip_atomic_store(&counters[tile_id], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

#pragma unroll
  for (int ii = 0; ii < 2; ++ii)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * 128 + (keep + ii) * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        const int64_t n = nw0 + c * 32 + lr;
        if (m < M && n < N) y[m * N + n] = f32_to_bf16_bits(own[ii][c][r]);
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
  if (p.wm == 2)
    gemm_kernel<Q, G, META, 2><<<grid, Cfg<2>::kThreads, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N,
                                                                   (int)K, splits, y, partials, counters);
  else
    gemm_kernel<Q, G, META, 1><<<grid, Cfg<1>::kThreads, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N,
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
