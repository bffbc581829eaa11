// Prefill GEMM: y[M,N] = x[M,K] * What[N,K]^T on bf16 MFMA.
//
// App. B.3 of the paper: What[n,k] = s[n,b] (u[n,k] - o[n,b]).  Prefill is a dense
// contraction, so it runs on v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
//
// Work split.  A workgroup computes a (128*WM) x 128 output tile (WM = 2 unless
// M <= 128) as two K-groups of 2*WM wavefronts: K-group g takes the 64-deep steps of
// parity g, so two wavefronts share each SIMD without doubling the tile, and their
// accumulators meet in LDS at the end.  Within a K-group a wavefront covers all 128*WM
// rows and 128 / (2*WM) columns: TI x TC MFMA tiles of 32 x 32 (8 x 1 or 4 x 2), 128 fp32
// accumulators per lane.  Only the activations and the packed weights go through LDS;
// each wavefront dequantizes its own weight rows straight into MFMA B operands, so
// dequantized weights never cost LDS bandwidth, and each dequantized operand feeds TI
// MFMAs.  A "window" is one step per K-group: its activation tiles (two stages) and
// its weight stage are read from one half of their LDS rings while the next window's
// are loaded straight into the other half (direct-to-LDS buffer loads, shared by the
// workgroup); one barrier per window.  On gfx950 the matrix cores and the vector ALU of
// a SIMD do not run at the same time (measured: an MFMA stream and a VALU stream take
// the sum of their times, in one wavefront or in two), so the dequantization arithmetic
// adds to the MFMA time.
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
constexpr uint32_t kOutOfRange = 0x80000000u;   // past every buffer a descriptor here covers
constexpr int kStages = 4;               // activation ring: two windows of two steps

template <int WM>
struct Cfg {
  static constexpr int BM = 128 * WM;                   // output rows per workgroup tile
  static constexpr int kGroupWaves = 2 * WM;            // wavefronts per K-group
  static constexpr int kWaves = 2 * kGroupWaves;
  // A wavefront covers all BM rows of the tile and BN / kGroupWaves columns: TI x TC
  // MFMA tiles of 32 x 32, 128 accumulators per lane either way.
  static constexpr int TI = BM / 32;
  static constexpr int TC = BN / (32 * kGroupWaves);
  static_assert(TI * TC == 8, "128 fp32 accumulators per lane");
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
// mantissa of the fp16 constant 1024, two fields per instruction, either where it
// lies (bits 0..q-1 of a half: 0x6400 | u == 1024 + u) or one field higher without a
// shift (bits q..2q-1: 0x6400 | (u << q) == 1024 + 2^q u, still inside the 10-bit
// mantissa).  One v_fma_mix_f32 per weight then forms (1024 + u)*s + so[0], or
// (1024 + 2^q u)*(s 2^-q) + so[1], with so[0] = -(1024 + o)*s and
// so[1] = -(1024 2^-q + o)*s (or m - 1024 s, m - 1024 2^-q s): every product is exact
// in fp32, so the weight is s*(u - o) exactly, rounded to bf16 once.  sc = {s, s 2^-q}.
template <int Q>
__device__ __forceinline__ bf16x8 dequant_slice(const uint32_t (&d)[Q], int j, const float (&sc)[2],
                                                const float (&so)[2]) {
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
  constexpr uint32_t kLow = Q == 4 ? 0x000F000Fu : Q == 3 ? 0x00070007u : 0x00030003u;
  const uint32_t t = sp >> (2 * Q);           // fields 2, 3 (and 6, 7) at the bottom
  const uint32_t p[4] = {and_or(sp, kLow, magic), and_or(sp, kLow << Q, magic), and_or(t, kLow, magic),
                         and_or(t, kLow << Q, magic)};
  float f[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {               // p[i] holds fields i and i + 4
    f[i] = __builtin_fmaf(f16_lo(p[i]), sc[i & 1], so[i & 1]);
    f[i + 4] = __builtin_fmaf(f16_hi(p[i]), sc[i & 1], so[i & 1]);
  }
  const uint32_t w0 = pack_bf16x2(f[0], f[1]), w1 = pack_bf16x2(f[2], f[3]);
  const uint32_t w2 = pack_bf16x2(f[4], f[5]), w3 = pack_bf16x2(f[6], f[7]);
  return __builtin_bit_cast(bf16x8, u32x4{w0, w1, w2, w3});
}

// Constant term so[1] of dequant_slice for the fields OR-ed in one field higher:
// -(1024 2^-q + o)*s (exact: an 11-bit integer by an 11-bit scale) or, for the binary16
// minimum layout, m - 1024 2^-q s (one rounding).
template <int META, int Q>
__device__ __forceinline__ float dequant_offset_high(float s, uint32_t meta_bits) {
  constexpr float kBase = (float)(1024 >> Q);
  if constexpr (META == kMetaMin) {
    return __builtin_fmaf(-kBase, s, f16_bits_to_f32(meta_bits));
  } else {
    const float o = META == kMetaZp ? (float)meta_bits : (float)(1 << (Q - 1));
    return -(kBase + o) * s;
  }
}

// Tile t in the order whole tiles are taken: bands of `bh` M tiles (fewer in the last
// band), each band swept along N with its M tiles together.  An XCD's run of tiles then
// covers about bh activation panels and run/bh weight panels, each fetched into its L2
// once while the workgroups sharing it run side by side; the host picks bh to make
// that sum of panel bytes small.
__device__ __forceinline__ void tile_at(int t, int tiles_m, int tiles_n, int bh, int& tm, int& tn) {
  const int band = t / (bh * tiles_n);
  const int h = tiles_m - bh * band < bh ? tiles_m - bh * band : bh;   // M tiles in this band
  const int rem = t - bh * band * tiles_n;
  tm = bh * band + rem % h;
  tn = rem / h;
}

// Work order.  Workgroups are dealt round-robin to the 8 XCDs (blockIdx % 8), each with
// its own L2; when a run of work items divides evenly, XCD x takes a contiguous part of
// it.  Items are `full` whole output tiles, then the remaining tiles cut into `splits`
// K slices each (all tiles are cut when full = 0, none when splits = 1).  Whole tiles
// (and a cut last round) follow tile_at; when every tile is cut, the K slices of a tile
// come first, then the N tiles of one M tile (an XCD holds one activation panel against
// a run of weight panels).  The slices of a tile are adjacent, so they meet on one XCD.
// `cut` is the tile's index among the cut tiles (its counter and partials), -1 for a
// whole tile.
__device__ __forceinline__ void work_item(int b, int tiles_m, int tiles_n, int full, int splits, int bh,
                                          int& tm, int& tn, int& split, int& cut) {
  if (b < full) {
    if (full % 8 == 0) b = (b % 8) * (full / 8) + b / 8;
    split = 0;
    cut = -1;
    tile_at(b, tiles_m, tiles_n, bh, tm, tn);
    return;
  }
  b -= full;
  const int items = (tiles_m * tiles_n - full) * splits;
  if (items % 8 == 0) b = (b % 8) * (items / 8) + b / 8;
  split = b % splits;
  cut = b / splits;
  if (full == 0) {
    tn = cut % tiles_n;
    tm = cut / tiles_n;
  } else {
    tile_at(full + cut, tiles_m, tiles_n, bh, tm, tn);
  }
}

// ---------------------------------------------------------------------------
// Split reduction (host side).  When the output has too few tiles to give every CU a
// workgroup, or a last round of tiles would leave most CUs idle, the K steps of those
// tiles are divided among `splits` workgroups whose fp32 partial tiles meet in a
// caller-provided workspace: [counters: one u32 per cut tile, in the fixed counter
// region][partials: cut tiles x splits x BM x BN fp32].  Without a workspace every tile
// is computed whole.
// ---------------------------------------------------------------------------
constexpr int kMinStepsPerSplit = 16;

struct Plan {
  int wm;            // wave tiles along M (tile height 128*wm)
  int64_t tiles;
  int64_t full;      // tiles computed whole by one workgroup; the rest are cut into `splits`
  int splits;
  int64_t workspace; // bytes needed when splits > 1
};

// One workgroup per CU (WM = 2: 128 KB of LDS) or two (WM = 1): `slots` run at once.
// Fewer tiles than slots: every tile is cut into K slices to fill them.  More: the tiles
// run in rounds, and a last round less than half full is cut instead, so that its
// slices fill the round and it takes a fraction of a round's time (896 tiles on 256
// CUs: three rounds of whole tiles and one of 256 half tiles rather than a fourth round
// of 128 tiles).
Plan plan_for(int64_t M, int64_t N, int64_t K) {
  Plan p{};
  p.wm = M > 128 ? 2 : 1;
  const int64_t bm = 128 * p.wm;
  p.tiles = ((M + bm - 1) / bm) * ((N + BN - 1) / BN);
  const int64_t steps = (K / 32 + 1) / 2;
  const int64_t slots = p.wm == 2 ? 256 : 512;
  const int64_t last = p.tiles % slots;
  const int64_t cut = p.tiles < slots ? p.tiles : (last != 0 && 2 * last <= slots ? last : 0);
  int64_t s = cut > 0 ? slots / cut : 1;
  s = std::min<int64_t>(s, steps / kMinStepsPerSplit);
  s = std::min<int64_t>(s, 8);
  if (cut > kMaxSplitCounters) s = 1;
  p.splits = (int)std::max<int64_t>(s, 1);
  p.full = p.splits > 1 ? p.tiles - cut : p.tiles;
  p.workspace = p.splits > 1 ? kSplitCounterBytes + cut * p.splits * bm * BN * 4 : 0;
  return p;
}

// Band height of the tile order: an XCD's run of whole tiles (a round's worth at most)
// spans about bh activation panels of BM x K bf16 and run/bh weight panels of BN x K
// codes with their scales and metadata; bh (a power of two up to the M tile count)
// keeps the sum of those bytes smallest.
int band_height(const Plan& p, int64_t M, int q, int group, int meta_bytes) {
  const int64_t bm = 128 * p.wm;
  const int64_t tiles_m = (M + bm - 1) / bm;
  const int64_t run = std::max<int64_t>(1, std::min<int64_t>(p.tiles, p.wm == 2 ? 256 : 512) / 8);
  const double a_panel = (double)bm * 2.0;
  const double w_panel = (double)BN * ((double)q / 8.0 + (2.0 + meta_bytes) / group);
  int bh = 1;
  double best = a_panel + (double)run * w_panel;
  for (int h = 2; h <= tiles_m; h *= 2) {
    const double c = h * a_panel + (double)((run + h - 1) / h) * w_panel;
    if (c < best) { best = c; bh = h; }
  }
  return bh;
}

template <int Q, int G, int META, int WM>
__global__ __launch_bounds__(Cfg<WM>::kThreads) void gemm_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const void* __restrict__ meta, int M, int N, int K, int full, int splits, int bh, uint16_t* __restrict__ y,
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
  const int wp = wave % C::kGroupWaves;                        // column block of the wavefront
  constexpr int TI = C::TI, TC = C::TC;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  int tm, tn, split, cut;
  work_item((int)blockIdx.x, tiles_m, tiles_n, full, splits, bh, tm, tn, split, cut);
  const int parts = cut >= 0 ? splits : 1;     // K slices of this workgroup's tile
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int nblk = K / 32;
  const int total_steps = (nblk + 1) / 2;
  // This workgroup's slice of the reduction: steps [s_begin, s_begin + nsteps), in
  // windows of two (the last window's odd step may lie past the slice: it reads zeros).
  const int per_split = (total_steps + parts - 1) / parts;
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
  const int64_t nw0 = n0 + wp * 32 * TC;

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
  uint32_t a_off[8];                     // per-lane offsets, the same in every window
#pragma unroll
  for (int i = 0; i < 8; ++i) a_off[i] = ((i & 1) ? a_b1 : a_b0) + (uint32_t)i * 16u * (uint32_t)K;
  const int a_bytes = (int)(rows_a * (uint32_t)K * 2);
  auto issue_a = [&](int win, auto pair_c) {
    constexpr int pair = decltype(pair_c)::value;
    // The window's k offset moves the descriptor (scalar arithmetic) rather than every
    // lane's offset; its size shrinks by as much, so the range check is unchanged.
    const int col = (s_begin + 2 * win + a_e) * 128;
    const int rest = a_bytes - col > 0 ? a_bytes - col : 0;
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(x + m0 * K + col / 2, (uint32_t)rest);
    auto fill = [&](uint8_t* st) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rw, (__attribute__((address_space(3))) void*)(st + a_w * 8192 + i * 1024), 16, a_off[i], 0, 0, 0);
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

  f32x16 acc[TI][TC];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int c = 0; c < TC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][c][r] = 0.0f;

  // This K-group's step of window `win`: activation stage at `at`, weight stage `pair`.
  auto compute = [&](const uint8_t* at, int win, auto pair_c, auto&& issue_next) {
    const uint8_t* bc = bstage(pair_c, 0);
    const uint8_t* bs = bstage(pair_c, 1);
    const uint8_t* bm = bstage(pair_c, 2);
    const uint32_t blk = 2u * (uint32_t)(s_begin + 2 * win) + (uint32_t)kblk;
    // a block past the slice or past K weighs zero: scale and metadata forced to 0 (the
    // reads themselves stay inside the row's 16 bytes of the stage, so they are always
    // made and their results selected)
    const bool valid = (2 * win + grp < nsteps) & (blk < (uint32_t)nblk);
    const uint32_t g0 = (2u * (uint32_t)(s_begin + 2 * win)) / (G / 32), gi = blk / (G / 32);
    // The step's LDS reads go out first (codes, scales, metadata, the first slice's
    // activation fragments), then the next window's loads, and only then the arithmetic
    // that waits for those reads: their latency hides behind the load issue.
    uint32_t cw[TC][Q], sraw[TC], mraw[TC];
#pragma unroll
    for (int c = 0; c < TC; ++c) {
      const int row = wp * 32 * TC + 32 * c + lr;
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
      sraw[c] = *reinterpret_cast<const uint16_t*>(bs + row * 16 + s_in);
      mraw[c] = 0u;
      if constexpr (ZP) {
        const uint32_t m_in = m_shift + (rbase + gi) * kMetaSize - ((m_shift + (rbase + g0) * kMetaSize) & ~3u);
        mraw[c] = META == kMetaMin ? (uint32_t)*reinterpret_cast<const uint16_t*>(bm + row * 16 + m_in)
                                   : (uint32_t)bm[row * 16 + m_in];
      }
    }
    // Operand reads run one slice ahead: slice j+1's activation fragments are requested
    // before slice j's weights are dequantized and its MFMAs issued, so the LDS latency
    // hides behind that work.
    bf16x8 a[2][TI];
#pragma unroll
    for (int i = 0; i < TI; ++i) a[0][i] = *reinterpret_cast<const bf16x8*>(at + swz(i * 32 + lr, 4 * h));
    __builtin_amdgcn_sched_barrier(0);
    issue_next();
    __builtin_amdgcn_sched_barrier(0);
    float sc[TC][2], so[TC][2];
#pragma unroll
    for (int c = 0; c < TC; ++c) {
      const uint32_t sbits = valid ? sraw[c] : 0u;
      const uint32_t mbits = valid ? mraw[c] : 0u;
      const float s = f16_bits_to_f32(sbits);
      sc[c][0] = s;
      sc[c][1] = s * (1.0f / (float)(1 << Q));
      so[c][0] = dequant_offset<META, Q>(s, mbits);
      so[c][1] = dequant_offset_high<META, Q>(s, mbits);
    }
    // Scheduling fences keep each group of reads at the head of the previous slice.
    __builtin_amdgcn_sched_barrier(0);
    auto slice = [&](auto jc) {
      constexpr int j = decltype(jc)::value;
      if constexpr (j < 3) {
#pragma unroll
        for (int i = 0; i < TI; ++i)
          a[(j + 1) & 1][i] = *reinterpret_cast<const bf16x8*>(at + swz(i * 32 + lr, 4 * h + j + 1));
        __builtin_amdgcn_sched_barrier(0);
      }
      bf16x8 b[TC];
#pragma unroll
      for (int c = 0; c < TC; ++c) b[c] = dequant_slice<Q>(cw[c], j, sc[c], so[c]);
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int c = 0; c < TC; ++c)
          acc[i][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j & 1][i], b[c], acc[i][c], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    };
    slice(std::integral_constant<int, 0>{});
    slice(std::integral_constant<int, 1>{});
    slice(std::integral_constant<int, 2>{});
    slice(std::integral_constant<int, 3>{});
  };

  // Window t: issue the loads of window t+1 (activations and weight stage, straight into
  // the other half of each ring, last read in window t-1, before the previous barrier),
  // multiply this K-group's step of window t, wait for this thread's loads, barrier:
  // every wavefront's part of window t+1's tiles is then in LDS.  Without metadata,
  // windows 0 and 1 are loaded together at the start, so window 1's loads are in flight
  // from the first moment rather than after window 0 has landed; every wavefront issues
  // window 1's 8 activation loads last, and loads complete in order, so at most 8
  // outstanding means window 0 has landed (the barrier waits for LDS only: window 1
  // stays in flight).  With metadata the extra live state of the peeled first window
  // made the compiler spill around the main loop (measured 1.6 % slower), so those
  // layouts start with window 0 alone.
  constexpr bool kTwoWindowStart = !ZP;
  issue_a(0, std::integral_constant<int, 0>{});
  issue_bstage(0, std::integral_constant<int, 0>{});
  if constexpr (kTwoWindowStart) {
    issue_bstage(1, std::integral_constant<int, 1>{});
    issue_a(1, std::integral_constant<int, 1>{});
    static_assert(C::kALoads == 8, "window 1's trailing activation loads");
    wait_vmcnt<8>();
    lds_barrier();
  } else {
    wait_vmcnt<0>();
    __syncthreads();
  }
  auto window = [&](int t, auto par, auto issue_c) {
    constexpr int p = decltype(par)::value;
    // the next window's loads go out after this step's first LDS reads, before its arithmetic
    compute(grp == 0 ? stage(std::integral_constant<int, 2 * p>{}) : stage(std::integral_constant<int, 2 * p + 1>{}),
            t, std::integral_constant<int, p>{}, [&] {
              if constexpr (decltype(issue_c)::value) {
                issue_a(t + 1, std::integral_constant<int, 1 - p>{});
                issue_bstage(t + 1, std::integral_constant<int, 1 - p>{});
              }
            });
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<0>();
    __syncthreads();
  };
  int t = 0;
  if constexpr (kTwoWindowStart) {
    window(0, std::integral_constant<int, 0>{}, std::false_type{});
    for (t = 1; t + 2 <= nwin; t += 2) {
      window(t, std::integral_constant<int, 1>{}, std::true_type{});
      window(t + 1, std::integral_constant<int, 0>{}, std::true_type{});
    }
    if (t < nwin) window(t, std::integral_constant<int, 1>{}, std::true_type{});
  } else {
    for (; t + 2 <= nwin; t += 2) {
      window(t, std::integral_constant<int, 0>{}, std::true_type{});
      window(t + 1, std::integral_constant<int, 1>{}, std::true_type{});
    }
    if (t < nwin) window(t, std::integral_constant<int, 0>{}, std::true_type{});
  }
  wait_vmcnt<0>();     // the last window's (empty) loads, before LDS is reused
  __syncthreads();

  // The K-groups meet: group g keeps M tiles [g TI/2, (g+1) TI/2) of its wave tile and
  // hands the other half to its partner (the same wave position in the other group)
  // through LDS; the activation ring is idle after the last barrier.  Layout: 16 KB per
  // wavefront, lane-contiguous 16-byte pieces (conflict-free).  The kept and given tiles
  // are named with compile-time indices (grp is uniform per wavefront, so the branch is
  // too): a runtime index would move the accumulators to scratch memory.
  constexpr int TH = TI / 2;
  f32x16 own[TH][TC];
  auto exchange = [&](auto keep_c) {
    constexpr int keep = decltype(keep_c)::value, give = TH - keep;
    constexpr int kPerStage = C::kStageBytes / 16384;     // wavefront areas per stage
    float* xo = reinterpret_cast<float*>(stage_dyn(wave / kPerStage)) + (size_t)(wave % kPerStage) * 4096;
#pragma unroll
    for (int ii = 0; ii < TH; ++ii)
#pragma unroll
      for (int c = 0; c < TC; ++c)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 v = {acc[give + ii][c][4 * q4], acc[give + ii][c][4 * q4 + 1], acc[give + ii][c][4 * q4 + 2],
                           acc[give + ii][c][4 * q4 + 3]};
          *reinterpret_cast<f32x4*>(xo + ((ii * TC + c) * 4 + q4) * 256 + lane * 4) = v;
        }
#pragma unroll
    for (int ii = 0; ii < TH; ++ii)
#pragma unroll
      for (int c = 0; c < TC; ++c) own[ii][c] = acc[keep + ii][c];
  };
  if (grp == 0) exchange(std::integral_constant<int, 0>{});
  else exchange(std::integral_constant<int, TH>{});
  __syncthreads();
  {
    constexpr int kPerStage = C::kStageBytes / 16384;
    const int partner = (1 - grp) * C::kGroupWaves + wp;
    const float* xi = reinterpret_cast<const float*>(stage_dyn(partner / kPerStage)) + (size_t)(partner % kPerStage) * 4096;
#pragma unroll
    for (int ii = 0; ii < TH; ++ii)
#pragma unroll
      for (int c = 0; c < TC; ++c)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 v = *reinterpret_cast<const f32x4*>(xi + ((ii * TC + c) * 4 + q4) * 256 + lane * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) own[ii][c][4 * q4 + e] += v[e];
        }
  }
  const int keep = TH * grp;    // M tiles keep .. keep + TH - 1 of the wave tile are this wavefront's

  if (cut >= 0) {
    // Split reduction: publish this slice's partial (the 64 accumulators this wavefront
    // owns, 16 bytes per lane per store, each store 1 KB contiguous), then count
    // arrivals; the last arriving workgroup sums the slices in slice order (its own from
    // registers, the others loaded), writes y and resets the counter so the workspace
    // stays reusable.  Partials are written and read with device-scope (sc1) accesses,
    // which go to memory rather than this XCD's L2, so no device-wide fence is needed:
    // a store's vmcnt is released once memory has acknowledged it.
    constexpr int kSc1 = 16;                               // buffer aux bits: device-coherent
    const __amdgpu_buffer_rsrc_t rp =
        make_rsrc(partials + (int64_t)cut * splits * (BM * BN), (uint32_t)splits * (BM * BN) * 4u);
    auto part_off = [&](int o, int ii, int c, int q4) {
      return (uint32_t)((o * (BM * BN) + wave * 4096 + ((ii * TC + c) * 4 + q4) * 256 + lane * 4) * 4);
    };
#pragma unroll
    for (int ii = 0; ii < TH; ++ii)
#pragma unroll
      for (int c = 0; c < TC; ++c)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 v = {own[ii][c][4 * q4], own[ii][c][4 * q4 + 1], own[ii][c][4 * q4 + 2], own[ii][c][4 * q4 + 3]};
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rp, (int)part_off(split, ii, c, q4), 0,
                                                 kSc1);
        }
    wait_vmcnt<0>();                       // every partial store acknowledged by memory
    unsigned int* arrived = reinterpret_cast<unsigned int*>(st0);
    __syncthreads();                       // the exchange above has finished reading LDS
    if (tid == 0) *arrived = atomicAdd(&counters[cut], 1u);
    __syncthreads();
    if (*arrived != (unsigned int)(splits - 1)) return;   // uniform across the workgroup
    f32x16 mine[TH][TC];
#pragma unroll
    for (int ii = 0; ii < TH; ++ii)
#pragma unroll
      for (int c = 0; c < TC; ++c) {
        mine[ii][c] = own[ii][c];
#pragma unroll
        for (int r = 0; r < 16; ++r) own[ii][c][r] = 0.0f;
      }
    for (int o = 0; o < splits; ++o) {
      if (o == split) {                    // uniform: this workgroup's own slice
#pragma unroll
        for (int ii = 0; ii < TH; ++ii)
#pragma unroll
          for (int c = 0; c < TC; ++c) own[ii][c] += mine[ii][c];
        continue;
      }
#pragma unroll
      for (int ii = 0; ii < TH; ++ii)
#pragma unroll
        for (int c = 0; c < TC; ++c)
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const f32x4 v = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(rp, (int)part_off(o, ii, c, q4), 0, kSc1));
#pragma unroll
            for (int e = 0; e < 4; ++e) own[ii][c][4 * q4 + e] += v[e];
          }
    }
    if (tid == 0) __hip_atomic_store(&counters[cut], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // y: through a buffer descriptor when y, with M padded to whole tiles, spans under
  // 1 GB (every offset then fits 32 bits, and so does an out-of-range base plus a row
  // offset): a lane's column past N gets an offset past the buffer, a row past M lies
  // past it anyway, so every store is issued and the range check drops those outside y.
  // The stores are non-temporal: this kernel never reads y, and the activation and
  // weight panels other workgroups are reading keep their L2 lines.
  if ((uint64_t)tiles_m * BM * (uint64_t)N * 2u < (1ull << 30)) {
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(y, (uint32_t)M * (uint32_t)N * 2u);
#pragma unroll
    for (int ii = 0; ii < TH; ++ii)
#pragma unroll
      for (int c = 0; c < TC; ++c) {
        const int64_t m = m0 + (keep + ii) * 32 + 4 * h;
        const int64_t n = nw0 + c * 32 + lr;
        const uint32_t base = n < N ? (uint32_t)((m * N + n) * 2) : kOutOfRange;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_bits(own[ii][c][r]), ry,
                                                (int)(base + (uint32_t)(8 * (r >> 2) + (r & 3)) * (uint32_t)N * 2u),
                                                0, kStream);
      }
    return;
  }
#pragma unroll
  for (int ii = 0; ii < TH; ++ii)
#pragma unroll
    for (int c = 0; c < TC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + (keep + ii) * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
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
  const int64_t full = split ? p.full : p.tiles;
  unsigned int* counters = static_cast<unsigned int*>(workspace);
  float* partials = split ? reinterpret_cast<float*>(static_cast<char*>(workspace) + kSplitCounterBytes)
                          : nullptr;
  const dim3 grid((unsigned)(full + (p.tiles - full) * splits));
  const int bh = band_height(p, M, Q, G, meta_size<META>());
  if (p.wm == 2)
    gemm_kernel<Q, G, META, 2><<<grid, Cfg<2>::kThreads, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N,
                                                                   (int)K, (int)full, splits, bh, y, partials, counters);
  else
    gemm_kernel<Q, G, META, 1><<<grid, Cfg<1>::kThreads, 0, stream>>>(x, codes, scales, zp, (int)M, (int)N,
                                                                   (int)K, (int)full, splits, bh, y, partials, counters);
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
