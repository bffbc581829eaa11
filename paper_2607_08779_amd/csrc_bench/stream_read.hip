// Measurement-only kernel, not part of the quantization library: a plain streaming
// read of a device buffer, the practical HBM ceiling that bench.py reports next to
// the decode GEMV (same bytes per launch, same number of distinct buffers, same graph
// replay).  Each thread reads four 16-byte items 256 items apart (non-temporal, like
// the GEMV's code loads); each block stores the XOR of what it read as one dword, so
// a launch also writes about as many bytes as the GEMV's output (4 bytes per 16 KB
// read: 8 KB for 33 MB, against the GEMV's 2 bytes per row), and like the GEMV it pays
// for those stores to land before the next launch starts.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kThreads = 256;
constexpr int kItems = 4;

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ p, int64_t n16,
                                                               uint32_t* __restrict__ sink) {
  const int64_t base = (int64_t)blockIdx.x * (kThreads * kItems) + threadIdx.x;
  uint32_t acc = 0;
#pragma unroll
  for (int u = 0; u < kItems; ++u) {
    const int64_t i = base + (int64_t)u * kThreads;
    if (i < n16) {
      const u32x4 v = __builtin_nontemporal_load(p + i);
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
  }
  if (threadIdx.x == 0) sink[blockIdx.x] = acc;
}

}  // namespace

// Reads bytes/16 16-byte items of p (device, 16-byte aligned) on `stream`; sink is a
// device array of at least ssq_bench_stream_read_sink_words(bytes) dwords that the
// kernel writes.  Returns 0 or a hipError_t value.
extern "C" int64_t ssq_bench_stream_read_sink_words(int64_t bytes) {
  return (bytes / 16 + kThreads * kItems - 1) / (kThreads * kItems);
}

extern "C" int ssq_bench_stream_read(const void* p, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  const int64_t n16 = bytes / 16;
  if (n16 <= 0) return 0;
  const int64_t blocks = ssq_bench_stream_read_sink_words(bytes);
  stream_read_kernel<<<dim3((unsigned)blocks), kThreads, 0, stream>>>(static_cast<const u32x4*>(p), n16, sink);
  return (int)hipGetLastError();
}
