// Sign-rule diagnostics (Sec. 4): for every group of the signed absmax grid, the
// clipped sets of both grid signs (Def. 1, Eq. (6)), the cardinality margin
// m(w) = |C_{-g*}| - |C_{g*}| and the realised error gain
// g(w) = ||w - Q_{-g*}(w)||^2 - ||w - Q_{g*}(w)||^2, which Lemma 1 (Eq. (7)) puts in
// closed form: 2 alpha (sum_{C_{-g*}} (-g* w_i - T) - sum_{C_{g*}} (g* w_i - T)),
// T = M (1 - 2^-q).  Remark 1 and Fig. 1 report these over every weight group of a
// model; the kernel also counts groups by the signs of m and g.
//
// Mapping as in the quantizer: each lane owns 8 consecutive weights, a group is G/8
// consecutive lanes, and a grid-stride loop walks the matrix.  The per-group arithmetic
// (exact integer clipped-set tests and excess sums) is sign_stats in sign_stats.h.
//
// The tally is accumulated beside: each group's leader lane adds one to a 16-bit field
// (one field per (sign m, sign g) cell, two per register), the grid is capped so that
// no field can reach 2^16, and the fields are summed over the wave and the block.  The
// blocks then reduce among themselves without atomics on the caller's buffer: each
// publishes its nine counts with write-through (device-coherent) stores, counts its
// arrival (two levels of counters), and the last block to arrive sums every block's
// counts, writes the tally with plain stores and rearms the counters.  The counts and the
// counter live in a small static device array; every call runs on the null stream, so
// calls on one device never overlap.
#include "mfma_dequant.h"   // wait_vmcnt
#include "sign_stats.h"
#include "ssq_internal.h"

namespace ssq {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 2;              // chunks per lane per loop trip (loads issued together)
constexpr int64_t kMaxTrips = 65535 / kUnroll;  // tally fields are 16 bits wide
constexpr int kMaxBlocks = 2048;        // resident grid: 8 blocks of 4 waves per CU

// Per-block tally counts (cell-major) and the arrival counters of the last-block
// reduction: blocks count into kClasses counters by blockIdx.x mod kClasses, the last of
// each class into one more.  Device-scope atomics on one address serialise at the
// memory side, so a single counter would queue every block of the grid; each counter
// sits on its own 256-byte line.
constexpr int kClasses = 64;
constexpr int kLineWords = 64;
__device__ unsigned int g_block_counts[9 * kMaxBlocks];
__device__ unsigned int g_arrivals[(kClasses + 1) * kLineWords];

// Dwords per chunk of 8 weights: 4 (bf16 pairs) or 8 (binary32).
template <typename In>
constexpr int kWords = 4 * (int)sizeof(In) / 2;

// This lane's 8 weights of chunk `c` of the trip whose first chunk the buffer resource
// starts at, as loaded; a chunk past the end reads as zeros (the resource ends at the
// matrix, so the load is out of its range), and every lane runs the same code.
template <typename In>
__device__ __forceinline__ void load_chunk(__amdgpu_buffer_rsrc_t r, uint32_t c, uint32_t (&d)[kWords<In>]) {
  constexpr uint32_t kBytes = 8 * sizeof(In);
  const int off = (int)(c * kBytes);
#pragma unroll
  for (int h = 0; h < kWords<In> / 4; ++h) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 16 * h, kStream);
    d[4 * h] = v.x; d[4 * h + 1] = v.y; d[4 * h + 2] = v.z; d[4 * h + 3] = v.w;
  }
}

// One group's statistics from its weights as binary32 values (every lane of the
// wavefront calls this: DPP exchanges).
template <int Q, int G>
__device__ __forceinline__ void group_stats_f32(const float (&w)[8], int& m, double& g) {
  constexpr int kLanes = G / 8;
  float mx = w[0], mn = w[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) { mx = fmaxf(mx, w[i]); mn = fminf(mn, w[i]); }
  mx = group_max<kLanes>(mx);
  const float nmn = group_max<kLanes>(-mn);
  sign_stats<Q, G>(w, mx, nmn, m, g);
}

// One group's statistics from this lane's 8 weights as loaded; valid in every lane of
// the group.  bf16 weights take the packed 16-bit arithmetic unless a group of the
// wavefront has a tiny or zero maximum (the choice is uniform over the wavefront: both
// paths exchange values between lanes).
template <typename In, int Q, int G>
__device__ __forceinline__ void group_stats(const uint32_t (&d)[kWords<In>], int& m, double& g) {
  if constexpr (sizeof(In) == 2) {
    bool gamma_neg;
    const uint32_t mb = group_absmax_bf16<G>(d, gamma_neg);
    if (__builtin_amdgcn_ballot_w64(mb < 0x100u) == 0) {
      sign_stats_bf16<Q, G>(d, mb, gamma_neg, m, g);
    } else {
      float w[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) { w[2 * j] = bf16_lo(d[j]); w[2 * j + 1] = bf16_hi(d[j]); }
      group_stats_f32<Q, G>(w, m, g);
    }
  } else {
    float w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = __uint_as_float(d[i]);
    group_stats_f32<Q, G>(w, m, g);
  }
}

template <typename In, int Q, int G>
__global__ __launch_bounds__(kThreads, 8) void diagnostics_kernel(const In* __restrict__ W,
                                                               int64_t total_chunks,
                                                               int16_t* __restrict__ margin,
                                                               float* __restrict__ gain,
                                                               unsigned long long* __restrict__ tally,
                                                               int nblocks) {
  constexpr int kLanes = G / 8;
  const bool leader = threadIdx.x % kLanes == 0;
  uint32_t packed[5] = {0, 0, 0, 0, 0};   // cell k = 3 (sign m + 1) + (sign g + 1): field k % 2 of word k / 2
  const int64_t stride = (int64_t)nblocks * (kThreads * kUnroll);     // nblocks = gridDim.x
  // The statistics of one trip's chunks, and the tally.  total_chunks is a multiple of
  // G/8, so a group's lanes are all valid or all not.
  // Margins and gains go out through buffer stores that every lane issues: a lane other
  // than its group's leader, and a group past the end of the matrix, store out of the
  // resource's range (discarded).  Unconditional stores keep the memory counter exact,
  // so the waits for the next trip's loads do not also wait for these stores.
  // byte offsets of this lane's group within a trip's first part (0x80000000 and above:
  // out of range)
  const uint32_t off_m = leader ? 2u * (threadIdx.x / kLanes) : 0x80000000u;
  const uint32_t off_g = leader ? 4u * (threadIdx.x / kLanes) : 0x80000000u;
  auto consume = [&](int64_t base, uint32_t (&w)[kUnroll][kWords<In>]) {
    const int64_t g0 = base / kLanes;                                       // base is a multiple of G/8
    const int64_t groups_left = (total_chunks - base) / kLanes;             // > 0
    const uint32_t ng = (uint32_t)std::min<int64_t>(groups_left, kThreads * kUnroll / kLanes);
    const __amdgpu_buffer_rsrc_t rm = make_rsrc(margin + g0, ng * 2);
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(gain + g0, ng * 4);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t chunk = base + u * kThreads + threadIdx.x;
      int m;
      double g;
      group_stats<In, Q, G>(w[u], m, g);
      const float gf = (float)g;
      constexpr uint32_t kPart = kThreads / kLanes;                          // groups per trip part
      __builtin_amdgcn_raw_buffer_store_b16((unsigned short)m, rm, (int)(off_m + 2 * u * kPart), 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(gf), rg, (int)(off_g + 4 * u * kPart), 0, 0);
      const int k = ((m > 0) - (m < 0) + 1) * 3 + ((gf > 0.0f) - (gf < 0.0f) + 1);
      const uint32_t inc = (leader && chunk < total_chunks) ? ((k & 1) ? 0x10000u : 1u) : 0u;
#pragma unroll
      for (int j = 0; j < 5; ++j) packed[j] += (k >> 1) == j ? inc : 0u;
    }
  };
  // This lane's chunks of the trip starting at `base` (zeros past the end of the matrix,
  // and for a trip that starts past it: the resource then covers no bytes).
  auto load_trip = [&](int64_t base, uint32_t (&w)[kUnroll][kWords<In>]) {
    const int64_t left = total_chunks - base;
    const uint32_t span = left > 0 ? (uint32_t)std::min<int64_t>(left, kThreads * kUnroll) * (8 * sizeof(In)) : 0u;
    const __amdgpu_buffer_rsrc_t r = make_rsrc(left > 0 ? W + 8 * base : W, span);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t c = u * kThreads + threadIdx.x;
      load_chunk<In>(r, c, w[u]);
    }
  };
  int64_t base = (int64_t)blockIdx.x * (kThreads * kUnroll);
  if constexpr (sizeof(In) == 2) {
    // bf16: the next trip's loads are in flight while this trip's statistics run, so a
    // wavefront waits on memory once rather than once per trip.
    // Two register sets alternate roles (a copy between them would wait for the loads).
    uint32_t a[kUnroll][kWords<In>], b[kUnroll][kWords<In>];
    load_trip(base, a);
    while (base < total_chunks) {
      load_trip(base + stride, b);
      __builtin_amdgcn_sched_barrier(0);
      consume(base, a);
      base += stride;
      if (base >= total_chunks) break;
      load_trip(base + stride, a);
      __builtin_amdgcn_sched_barrier(0);
      consume(base, b);
      base += stride;
    }
  } else {
    for (; base < total_chunks; base += stride) {
      uint32_t w[kUnroll][kWords<In>];
      load_trip(base, w);
      __builtin_amdgcn_sched_barrier(0);      // every load of the trip is in flight before any arithmetic
      consume(base, w);
    }
  }
  if (tally == nullptr) return;                          // uniform over the grid

  __shared__ unsigned int block_counts[9];
  __shared__ bool arrived;
  if (threadIdx.x < 9) block_counts[threadIdx.x] = 0;
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 9; ++k) {
    // a wave's sum of 16-bit fields stays below 2^22: exact in binary32
    const float v = wave_sum((float)((packed[k >> 1] >> (16 * (k & 1))) & 0xFFFFu));
    if ((threadIdx.x & 63) == 63 && v != 0.0f) atomicAdd(&block_counts[k], (unsigned int)v);
  }
  __syncthreads();
  // Publish with write-through stores; vmcnt drains only once memory has acknowledged
  // them, so they are visible device-wide before the arrival is counted.
  if (threadIdx.x < 9)
    __hip_atomic_store(&g_block_counts[threadIdx.x * kMaxBlocks + blockIdx.x], block_counts[threadIdx.x],
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  wait_vmcnt<0>();
  __syncthreads();
  const unsigned int nb = (unsigned int)nblocks;
  if (threadIdx.x == 0) {
    const unsigned int cls = blockIdx.x % kClasses;
    const unsigned int members = (nb - cls + kClasses - 1) / kClasses;   // blocks of this class
    const unsigned int classes = std::min<unsigned int>(nb, kClasses);
    arrived = atomicAdd(&g_arrivals[cls * kLineWords], 1u) == members - 1 &&
              atomicAdd(&g_arrivals[kClasses * kLineWords], 1u) == classes - 1;
  }
  __syncthreads();
  if (!arrived) return;                                  // uniform across the block

  // Last block: sum each cell over the blocks (device-coherent 16-byte loads of four
  // blocks' counts; slots past the grid hold counts of earlier calls and are skipped).
  constexpr int kSc1 = 16;                               // buffer aux bits: device-coherent
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(g_block_counts, sizeof(g_block_counts));
  __shared__ unsigned int wave_counts[kThreads / 64][9];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll 1
  for (int k0 = 0; k0 < 9; k0 += 3) {                  // three cells per round of loads
    uint32_t v[3] = {0, 0, 0};                           // < 2^26 per thread, < 2^32 per wave
#pragma unroll
    for (int i = 0; i < kMaxBlocks / (4 * kThreads); ++i) {
      const unsigned int b0 = (i * kThreads + threadIdx.x) * 4;
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        const u32x4 c =
            __builtin_amdgcn_raw_buffer_load_b128(rc, (int)(((k0 + k) * kMaxBlocks + b0) * 4), 0, kSc1);
        v[k] += (b0 < nb ? c.x : 0u) + (b0 + 1 < nb ? c.y : 0u) + (b0 + 2 < nb ? c.z : 0u) +
                (b0 + 3 < nb ? c.w : 0u);
      }
    }
#pragma unroll
    for (int k = 0; k < 3; ++k) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) v[k] += __shfl_xor(v[k], o, 64);
      if (lane == 0) wave_counts[wave][k0 + k] = v[k];
    }
  }
  __syncthreads();
  if (threadIdx.x < 9) {
    unsigned long long total = 0;
#pragma unroll
    for (int i = 0; i < kThreads / 64; ++i) total += wave_counts[i][threadIdx.x];
    tally[threadIdx.x] = total;
  }
  // Rearm: every block has arrived, so no other block touches the counters now.
  if (threadIdx.x <= kClasses)
    __hip_atomic_store(&g_arrivals[threadIdx.x * kLineWords], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void zero_tally_kernel(unsigned long long* tally) {
  if (threadIdx.x < 9) tally[threadIdx.x] = 0;
}

template <typename In, int Q, int G>
hipError_t diagnose(const In* W, int64_t total_chunks, int16_t* margin, float* gain,
                    unsigned long long* tally) {
  const int64_t per_block = kThreads * kUnroll;
  const int64_t needed = (total_chunks + per_block - 1) / per_block;
  const int64_t blocks = std::min<int64_t>(needed, kMaxBlocks);
  if ((needed + blocks - 1) / blocks > kMaxTrips) return hipErrorInvalidValue;   // past about 2^38 weights
  diagnostics_kernel<In, Q, G><<<dim3((unsigned)blocks), kThreads, 0, nullptr>>>(W, total_chunks, margin,
                                                                                gain, tally, (int)blocks);
  return hipGetLastError();
}

template <typename In>
hipError_t launch_any(const In* W, int64_t rows, int64_t cols, int group, int q, int16_t* margin,
                      float* gain, uint64_t* tally) {
  unsigned long long* t = reinterpret_cast<unsigned long long*>(tally);
  const int64_t total_chunks = rows * cols / 8;
  if (total_chunks == 0) {
    if (t == nullptr) return hipSuccess;
    zero_tally_kernel<<<1, 64, 0, nullptr>>>(t);          // no groups: an all-zero tally
    return hipGetLastError();
  }
  switch (q * 1000 + group) {
    case 2032: return diagnose<In, 2, 32>(W, total_chunks, margin, gain, t);
    case 2064: return diagnose<In, 2, 64>(W, total_chunks, margin, gain, t);
    case 2128: return diagnose<In, 2, 128>(W, total_chunks, margin, gain, t);
    case 3032: return diagnose<In, 3, 32>(W, total_chunks, margin, gain, t);
    case 3064: return diagnose<In, 3, 64>(W, total_chunks, margin, gain, t);
    case 3128: return diagnose<In, 3, 128>(W, total_chunks, margin, gain, t);
    case 4032: return diagnose<In, 4, 32>(W, total_chunks, margin, gain, t);
    case 4064: return diagnose<In, 4, 64>(W, total_chunks, margin, gain, t);
    case 4128: return diagnose<In, 4, 128>(W, total_chunks, margin, gain, t);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_diagnostics_bf16(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                                   int16_t* margin, float* gain, uint64_t* tally) {
  return launch_any<uint16_t>(W, rows, cols, group, q, margin, gain, tally);
}

hipError_t launch_diagnostics_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                                  int16_t* margin, float* gain, uint64_t* tally) {
  return launch_any<float>(W, rows, cols, group, q, margin, gain, tally);
}

}  // namespace ssq
