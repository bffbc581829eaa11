// GGUF array-of-structures export of packed weights (App. B.1, formats table).
//
// The library keeps codes and scales in separate arrays (structure of arrays: a row's
// q-bit indices as one little-endian bit stream, a binary16 scale per group, and for the
// Q*_1 layout a binary16 minimum per group).  llama.cpp stores a weight matrix as
// consecutive 32-weight blocks holding their own scale: per block a binary16 s, for the
// Q*_1 formats a binary16 m, then the block's indices qs:
//   Q4_0 / Q4_0s  s + qs[16]       18 bytes      Q4_1  s + m + qs[16]  20 bytes
//   Q2_0 / Q2_0s  s + qs[8]        10 bytes      Q2_1  s + m + qs[8]   12 bytes
// The signed-symmetric variant is the same layout with a scale that may be negative.
// Index order inside qs (the formats table fixes the sizes, not the order): Q4 byte j
// holds index j in its low nibble and index j + 16 in its high nibble (the nibble split
// that llama.cpp's 4-bit unpack undoes with one shift and one mask); Q2 byte i holds
// indices 4i .. 4i+3 at bits 0, 2, 4, 6 (the order that four shift-and extractions and
// a byte/word interleave restore), which is the library's own bit stream.
//
// One thread per 32-weight block: it loads the block's 4q code bytes, its scale (and
// minimum), reorders the Q4 nibbles and stores the block with 16-bit stores (block
// sizes and offsets are even).  An export runs once per model, off the hot path.
#include "ssq_internal.h"

namespace ssq {
namespace {

constexpr int kExportThreads = 256;

// Index k (0..31) of a q = 4 block held as four dwords.
__device__ __forceinline__ uint32_t nibble(const uint32_t (&d)[4], int k) { return (d[k >> 3] >> (4 * (k & 7))) & 0xFu; }

template <int Q, bool MIN>
__global__ __launch_bounds__(kExportThreads) void export_gguf_kernel(const uint8_t* __restrict__ codes,
                                                                     const uint16_t* __restrict__ scales,
                                                                     const uint16_t* __restrict__ mins,
                                                                     int64_t blocks, int64_t blocks_per_row,
                                                                     int blocks_per_group,
                                                                     uint16_t* __restrict__ out) {
  constexpr int kHalves = (MIN ? 2 : 1) + 2 * Q;     // block size in 16-bit words
  const int64_t blk = (int64_t)blockIdx.x * kExportThreads + threadIdx.x;
  if (blk >= blocks) return;
  const int64_t row = blk / blocks_per_row, b = blk - row * blocks_per_row;
  const int64_t gi = row * (blocks_per_row / blocks_per_group) + b / blocks_per_group;
  uint16_t* const o = out + blk * kHalves;
  o[0] = scales[gi];
  if constexpr (MIN) o[1] = mins[gi];
  constexpr int kQs = MIN ? 2 : 1;                   // first word of qs
  const uint32_t* const src = reinterpret_cast<const uint32_t*>(codes + blk * (4 * Q));
  if constexpr (Q == 2) {
    const uint32_t d0 = src[0], d1 = src[1];         // already in Q2 order
    o[kQs + 0] = (uint16_t)d0; o[kQs + 1] = (uint16_t)(d0 >> 16);
    o[kQs + 2] = (uint16_t)d1; o[kQs + 3] = (uint16_t)(d1 >> 16);
  } else {
    // index k of the block sits at bits 4k of the 128-bit stream d[0..3]
    uint32_t d[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) d[i] = src[i];
#pragma unroll
    for (int w = 0; w < 8; ++w) {                    // qs bytes 2w and 2w + 1
      const uint32_t lo = nibble(d, 2 * w) | (nibble(d, 2 * w + 16) << 4);
      const uint32_t hi = nibble(d, 2 * w + 1) | (nibble(d, 2 * w + 17) << 4);
      o[kQs + w] = (uint16_t)(lo | (hi << 8));
    }
  }
}

template <int Q, bool MIN>
hipError_t export_launch(const uint8_t* codes, const uint16_t* scales, const uint16_t* mins, int64_t rows,
                         int64_t cols, int group, uint8_t* out, hipStream_t stream) {
  const int64_t blocks = rows * (cols / 32);
  const dim3 grid((unsigned)((blocks + kExportThreads - 1) / kExportThreads));
  export_gguf_kernel<Q, MIN><<<grid, kExportThreads, 0, stream>>>(codes, scales, mins, blocks, cols / 32,
                                                                  group / 32, reinterpret_cast<uint16_t*>(out));
  return hipGetLastError();
}

}  // namespace

int64_t gguf_block_bytes(int q, bool with_min) { return (with_min ? 4 : 2) + 4 * q; }

hipError_t launch_export_gguf(const uint8_t* codes, const uint16_t* scales, const uint16_t* mins, int64_t rows,
                              int64_t cols, int group, int q, uint8_t* out, hipStream_t stream) {
  if (q == 4) return mins ? export_launch<4, true>(codes, scales, mins, rows, cols, group, out, stream)
                          : export_launch<4, false>(codes, scales, mins, rows, cols, group, out, stream);
  if (q == 2) return mins ? export_launch<2, true>(codes, scales, mins, rows, cols, group, out, stream)
                          : export_launch<2, false>(codes, scales, mins, rows, cols, group, out, stream);
  return hipErrorInvalidValue;
}

}  // namespace ssq
