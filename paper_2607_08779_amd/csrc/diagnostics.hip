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

// This lane's 8 weights of chunk `c` of the trip whose first chunk the buffer resource
// starts at; a chunk past the end reads as zeros (the load is out of the resource's
// range), so every lane runs the same code.
template <typename In>
__device__ __forceinline__ void load_chunk(__amdgpu_buffer_rsrc_t r, uint32_t c, bool valid, float (&w)[8]) {
  constexpr uint32_t kBytes = 8 * sizeof(In);
  const int off = valid ? (int)(c * kBytes) : (int)0x80000000;
  if constexpr (sizeof(In) == 2) {
    const u32x4 d = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kStream);
    w[0] = bf16_lo(d.x); w[1] = bf16_hi(d.x); w[2] = bf16_lo(d.y); w[3] = bf16_hi(d.y);
    w[4] = bf16_lo(d.z); w[5] = bf16_hi(d.z); w[6] = bf16_lo(d.w); w[7] = bf16_hi(d.w);
  } else {
    const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kStream);
    const u32x4 b = __builtin_amdgcn_raw_buffer_load_b128(r, off, 16, kStream);
    w[0] = __uint_as_float(a.x); w[1] = __uint_as_float(a.y); w[2] = __uint_as_float(a.z);
    w[3] = __uint_as_float(a.w); w[4] = __uint_as_float(b.x); w[5] = __uint_as_float(b.y);
    w[6] = __uint_as_float(b.z); w[7] = __uint_as_float(b.w);
  }
}

// One group's statistics from this lane's 8 weights; valid in every lane of the group.
template <int Q, int G>
__device__ __forceinline__ void group_stats(const float (&w)[8], int& m, double& g) {
  constexpr int kLanes = G / 8;
  float mx = w[0], mn = w[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) { mx = fmaxf(mx, w[i]); mn = fminf(mn, w[i]); }
  mx = group_max<kLanes>(mx);
  const float nmn = group_max<kLanes>(-mn);
  sign_stats<Q, G>(w, mx, nmn, m, g);
}

template <typename In, int Q, int G>
__global__ __launch_bounds__(kThreads, 8) void diagnostics_kernel(const In* __restrict__ W,
                                                               int64_t total_chunks,
                                                               int16_t* __restrict__ margin,
                                                               float* __restrict__ gain,
                                                               unsigned long long* __restrict__ tally) {
  constexpr int kLanes = G / 8;
  const bool leader = threadIdx.x % kLanes == 0;
  uint32_t packed[5] = {0, 0, 0, 0, 0};   // cell k = 3 (sign m + 1) + (sign g + 1): field k % 2 of word k / 2
  const int64_t stride = (int64_t)gridDim.x * (kThreads * kUnroll);
  // total_chunks is a multiple of G/8, so a group's lanes are all valid or all not.
  for (int64_t base = (int64_t)blockIdx.x * (kThreads * kUnroll); base < total_chunks; base += stride) {
    const int64_t left = total_chunks - base;             // > 0
    const uint32_t span = (uint32_t)std::min<int64_t>(left, kThreads * kUnroll) * (8 * sizeof(In));
    const __amdgpu_buffer_rsrc_t r = make_rsrc(W + 8 * base, span);
    float w[kUnroll][8];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t c = u * kThreads + threadIdx.x;
      load_chunk<In>(r, c, base + c < total_chunks, w[u]);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t chunk = base + u * kThreads + threadIdx.x;
      int m;
      double g;
      group_stats<Q, G>(w[u], m, g);
      if (leader && chunk < total_chunks) {
        const int64_t group = chunk / kLanes;
        const float gf = (float)g;
        margin[group] = (int16_t)m;
        gain[group] = gf;
        const int k = ((m > 0) - (m < 0) + 1) * 3 + ((gf > 0.0f) - (gf < 0.0f) + 1);
        const uint32_t inc = (k & 1) ? 0x10000u : 1u;
#pragma unroll
        for (int j = 0; j < 5; ++j) packed[j] += (k >> 1) == j ? inc : 0u;
      }
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
  const unsigned int nb = gridDim.x;
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
                                                                                gain, tally);
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
