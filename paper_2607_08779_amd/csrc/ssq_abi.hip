// C ABI of libssq: argument validation and kernel dispatch (see include/ssq.h).
//
// Every check runs on the host before any HIP call, so an invalid call returns
// without launching anything or touching an output byte.
#include "ssq.h"

#include <mutex>

#include "ssq_internal.h"

namespace ssq {
// Decode GEMV for two tokens (gemv.hip): each unpacked block serves both.
hipError_t launch_gemv2_bf16(const uint16_t* x, const uint8_t* codes, const uint16_t* scales, GroupMeta meta,
                             int64_t N, int64_t K, int group, int q, uint16_t* y, hipStream_t stream);
}  // namespace ssq

namespace {

constexpr int64_t kMaxElems = int64_t(1) << 40;   // rows*cols or N*K
constexpr int64_t kMaxDim = int64_t(1) << 30;     // any single dimension (kernels index in int)
constexpr int64_t kMaxK = int64_t(1) << 22;       // matmul reduction length (32-bit tile offsets)

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
bool valid_q(int q) { return q == 2 || q == 3 || q == 4; }
bool valid_group(int g) { return g == 32 || g == 64 || g == 128; }
int status_of(hipError_t e) { return e == hipSuccess ? SSQ_OK : SSQ_EHIP; }

int check_grid_sizes(int64_t rows, int64_t cols, int group, int q) {
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return SSQ_EINVAL;
  if (!valid_q(q) || !valid_group(group)) return SSQ_EINVAL;
  if (cols % group != 0) return SSQ_EINVAL;
  if (rows * cols > kMaxElems) return SSQ_EINVAL;
  return SSQ_OK;
}

int check_quantize(const void* W, int64_t rows, int64_t cols, int group, int q, int mode,
                   const uint8_t* codes, const uint16_t* scales, const uint8_t* zp) {
  if (check_grid_sizes(rows, cols, group, q) != SSQ_OK) return SSQ_EINVAL;
  if (mode != SSQ_SIGNED_SYM && mode != SSQ_UNSIGNED_SYM && mode != SSQ_ASYM) return SSQ_EINVAL;
  if ((mode == SSQ_ASYM) != (zp != nullptr)) return SSQ_EINVAL;
  if (rows == 0 || cols == 0) return SSQ_OK;
  if (W == nullptr || codes == nullptr || scales == nullptr) return SSQ_EINVAL;
  if (!aligned(W, 16) || !aligned(codes, 16) || !aligned(scales, 2)) return SSQ_EALIGN;
  return SSQ_OK;
}

int check_matmul_sizes(int64_t M, int64_t N, int64_t K, int group, int q) {
  if (M < 0 || N < 0 || K <= 0 || M > kMaxDim || N > kMaxDim || K > kMaxK) return SSQ_EINVAL;
  if (!valid_q(q) || !valid_group(group) || K % group != 0) return SSQ_EINVAL;
  if (N * K > kMaxElems || M * K > kMaxElems || M * N > kMaxElems) return SSQ_EINVAL;
  return SSQ_OK;
}

int check_matmul(const void* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                 int64_t N, int64_t K, int group, int q, const void* y) {
  if (check_matmul_sizes(M, N, K, group, q) != SSQ_OK) return SSQ_EINVAL;
  if (M == 0 || N == 0) return SSQ_OK;
  if (x == nullptr || codes == nullptr || scales == nullptr || y == nullptr) return SSQ_EINVAL;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(y, 16) || !aligned(scales, 2))
    return SSQ_EALIGN;
  return SSQ_OK;
}

int check_diagnostics(const void* W, int64_t rows, int64_t cols, int group, int q,
                      const int16_t* margin, const float* gain, const uint64_t* tally) {
  if (check_grid_sizes(rows, cols, group, q) != SSQ_OK) return SSQ_EINVAL;
  if (rows == 0 || cols == 0) return aligned(tally, 8) ? SSQ_OK : SSQ_EALIGN;   // tally only
  if (W == nullptr || margin == nullptr || gain == nullptr) return SSQ_EINVAL;
  if (!aligned(W, 16) || !aligned(margin, 2) || !aligned(gain, 4) || !aligned(tally, 8)) return SSQ_EALIGN;
  return SSQ_OK;
}

ssq::GroupMeta zero_points(const uint8_t* zp) { return {zp, zp ? ssq::kMetaZp : ssq::kMetaNone}; }
ssq::GroupMeta minimums(const uint16_t* mins) { return {mins, ssq::kMetaMin}; }

// bf16 matmul kernel choice by token count: streaming GEMV (M = 1, 2), skinny-M MFMA
// kernel (batched decode), tiled MFMA GEMM with an optional split reduction (prefill).
int dispatch_bf16(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                  ssq::GroupMeta meta, int64_t N, int64_t K, int group, int q, uint16_t* y,
                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (M == 1) return status_of(ssq::launch_gemv_bf16(x, codes, scales, meta, N, K, group, q, y, stream));
  if (M == 2) return status_of(ssq::launch_gemv2_bf16(x, codes, scales, meta, N, K, group, q, y, stream));
  if (M <= ssq::kSkinnyMaxM)
    return status_of(ssq::launch_skinny_bf16(x, M, codes, scales, meta, N, K, group, q, y, workspace,
                                             workspace_bytes, stream));
  return status_of(ssq::launch_gemm_bf16(x, M, codes, scales, meta, N, K, group, q, y, workspace,
                                         workspace_bytes, stream));
}

// ---------------------------------------------------------------------------
// Static split-reduction scratch of ssq_matmul_noalloc, for callers that cannot
// allocate.  Every GPU the library runs on holds its own copy of the array until the
// process ends; the host name `scratch` is only a handle, so its device address is
// looked up once per device (hipGetSymbolAddress) and only that address is passed on.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::once_flag g_scratch_once[kMaxScratchDevices];
void* g_scratch_ptr[kMaxScratchDevices];
hipError_t g_scratch_err[kMaxScratchDevices];

__global__ void zero_words(uint32_t* p, int n) {
  const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (i < n) p[i] = 0u;
}

// Device address of the current device's scratch (null on error, with *err set).  The
// first call on a device also clears the arrival counters at the front of the array
// with a fill kernel on `stream` (a kernel, not a memset, so that a first call under
// graph capture records nothing else); the split kernels return the counters to zero
// at the end of every call, so later calls find them cleared.
void* scratch_for_current_device(hipStream_t stream, hipError_t* err) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) {
    *err = e != hipSuccess ? e : hipErrorInvalidDevice;
    return nullptr;
  }
  std::call_once(g_scratch_once[dev], [&] {
    void* p = nullptr;
    hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r == hipSuccess) {
      constexpr int kWords = (int)(ssq::kSplitCounterBytes / 4);
      zero_words<<<kWords / 256, 256, 0, stream>>>(static_cast<uint32_t*>(p), kWords);
      r = hipGetLastError();
    }
    g_scratch_err[dev] = r;
    if (r == hipSuccess) g_scratch_ptr[dev] = p;
  });
  *err = g_scratch_err[dev];
  return g_scratch_ptr[dev];
}

int check_act_q8(const void* x, int64_t M, int64_t K, const void* q, const uint16_t* d) {
  if (M < 0 || K < 0 || M > kMaxDim || K > kMaxDim || K % 32 != 0 || M * K > kMaxElems) return SSQ_EINVAL;
  if (M == 0 || K == 0) return SSQ_OK;
  if (x == nullptr || q == nullptr || d == nullptr) return SSQ_EINVAL;
  if (!aligned(x, 16) || !aligned(q, 16) || !aligned(d, 2)) return SSQ_EALIGN;
  return SSQ_OK;
}

int check_matmul_q8(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                    const uint16_t* scales, int64_t N, int64_t K, int group, int q, const uint16_t* y) {
  const int st = check_matmul(qx, M, codes, scales, N, K, group, q, y);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  if (dx == nullptr) return SSQ_EINVAL;
  return aligned(dx, 2) ? SSQ_OK : SSQ_EALIGN;
}

// Shared checks of the binary16-minimum entry points: a minimum per group, 2-byte aligned.
int check_mins(const uint16_t* mins, bool needed) {
  if (!needed) return SSQ_OK;
  if (mins == nullptr) return SSQ_EINVAL;
  return aligned(mins, 2) ? SSQ_OK : SSQ_EALIGN;
}

}  // namespace

extern "C" {

int ssq_quantize(const uint16_t* W, int64_t rows, int64_t cols, int group, int q, int mode,
                 uint8_t* codes, uint16_t* scales, uint8_t* zp) {
  const int st = check_quantize(W, rows, cols, group, q, mode, codes, scales, zp);
  if (st != SSQ_OK || rows == 0 || cols == 0) return st;
  return status_of(ssq::launch_quantize_bf16(W, rows, cols, group, q, mode, codes, scales, zp, nullptr));
}

int ssq_quantize_min(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                     uint8_t* codes, uint16_t* scales, uint16_t* mins) {
  int st = check_quantize(W, rows, cols, group, q, SSQ_SIGNED_SYM, codes, scales, nullptr);
  if (st == SSQ_OK) st = check_mins(mins, rows > 0 && cols > 0);
  if (st != SSQ_OK || rows == 0 || cols == 0) return st;
  return status_of(ssq::launch_quantize_bf16(W, rows, cols, group, q, ssq::kModeAsymMin, codes, scales,
                                             mins, nullptr));
}

int ssq_quantize_min_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                         uint8_t* codes, uint16_t* scales, uint16_t* mins) {
  int st = check_quantize(W, rows, cols, group, q, SSQ_SIGNED_SYM, codes, scales, nullptr);
  if (st == SSQ_OK) st = check_mins(mins, rows > 0 && cols > 0);
  if (st != SSQ_OK || rows == 0 || cols == 0) return st;
  return status_of(ssq::launch_quantize_f32(W, rows, cols, group, q, ssq::kModeAsymMin, codes, scales,
                                            mins, nullptr));
}

int ssq_quantize_f32(const float* W, int64_t rows, int64_t cols, int group, int q, int mode,
                     uint8_t* codes, uint16_t* scales, uint8_t* zp) {
  const int st = check_quantize(W, rows, cols, group, q, mode, codes, scales, zp);
  if (st != SSQ_OK || rows == 0 || cols == 0) return st;
  return status_of(ssq::launch_quantize_f32(W, rows, cols, group, q, mode, codes, scales, zp, nullptr));
}

int ssq_matmul(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
               const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
               hipStream_t stream) {
  const int st = check_matmul(x, M, codes, scales, N, K, group, q, y);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  return dispatch_bf16(x, M, codes, scales, zero_points(zp), N, K, group, q, y, nullptr, 0, stream);
}

int ssq_matmul_min(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                   const uint16_t* mins, int64_t N, int64_t K, int group, int q, uint16_t* y,
                   hipStream_t stream) {
  int st = check_matmul(x, M, codes, scales, N, K, group, q, y);
  if (st == SSQ_OK) st = check_mins(mins, M > 0 && N > 0);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  return dispatch_bf16(x, M, codes, scales, minimums(mins), N, K, group, q, y, nullptr, 0, stream);
}

size_t ssq_matmul_workspace_size(int64_t M, int64_t N, int64_t K, int group, int q) {
  if (check_matmul_sizes(M, N, K, group, q) != SSQ_OK || M <= 2 || N == 0) return 0;   // GEMV: no split
  return M <= ssq::kSkinnyMaxM ? ssq::skinny_workspace_bytes(M, N, K, q) : ssq::gemm_workspace_bytes(M, N, K);
}

int ssq_matmul_ws(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                  const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  const int st = check_matmul(x, M, codes, scales, N, K, group, q, y);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  if (workspace != nullptr && !aligned(workspace, 256)) return SSQ_EALIGN;
  return dispatch_bf16(x, M, codes, scales, zero_points(zp), N, K, group, q, y, workspace, workspace_bytes,
                       stream);
}

int ssq_matmul_noalloc(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                       const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
                       hipStream_t stream) {
  const int st = check_matmul(x, M, codes, scales, N, K, group, q, y);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  const size_t need = ssq_matmul_workspace_size(M, N, K, group, q);
  if (need > kScratchBytes) return SSQ_ESCRATCH;
  void* ws = nullptr;
  if (need > 0) {
    hipError_t e = hipSuccess;
    ws = scratch_for_current_device(stream, &e);
    if (ws == nullptr) return SSQ_EHIP;
  }
  return dispatch_bf16(x, M, codes, scales, zero_points(zp), N, K, group, q, y, ws, need, stream);
}

int ssq_matmul_min_ws(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                      const uint16_t* mins, int64_t N, int64_t K, int group, int q, uint16_t* y,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = check_matmul(x, M, codes, scales, N, K, group, q, y);
  if (st == SSQ_OK) st = check_mins(mins, M > 0 && N > 0);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  if (workspace != nullptr && !aligned(workspace, 256)) return SSQ_EALIGN;
  return dispatch_bf16(x, M, codes, scales, minimums(mins), N, K, group, q, y, workspace, workspace_bytes,
                       stream);
}

int ssq_matmul_f32(const float* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                   const uint8_t* zp, int64_t N, int64_t K, int group, int q, float* y,
                   hipStream_t stream) {
  const int st = check_matmul(x, M, codes, scales, N, K, group, q, y);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  return status_of(ssq::launch_matmul_f32(x, M, codes, scales, zero_points(zp), N, K, group, q, y, stream));
}

int ssq_matmul_min_f32(const float* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                       const uint16_t* mins, int64_t N, int64_t K, int group, int q, float* y,
                       hipStream_t stream) {
  int st = check_matmul(x, M, codes, scales, N, K, group, q, y);
  if (st == SSQ_OK) st = check_mins(mins, M > 0 && N > 0);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  return status_of(ssq::launch_matmul_f32(x, M, codes, scales, minimums(mins), N, K, group, q, y, stream));
}

int ssq_sign_diagnostics(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                         int16_t* margin, float* gain, uint64_t* tally) {
  const int st = check_diagnostics(W, rows, cols, group, q, margin, gain, tally);
  if (st != SSQ_OK || ((rows == 0 || cols == 0) && tally == nullptr)) return st;
  return status_of(ssq::launch_diagnostics_bf16(W, rows, cols, group, q, margin, gain, tally));
}

int ssq_sign_diagnostics_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                             int16_t* margin, float* gain, uint64_t* tally) {
  const int st = check_diagnostics(W, rows, cols, group, q, margin, gain, tally);
  if (st != SSQ_OK || ((rows == 0 || cols == 0) && tally == nullptr)) return st;
  return status_of(ssq::launch_diagnostics_f32(W, rows, cols, group, q, margin, gain, tally));
}

int ssq_quantize_diag(const uint16_t* W, int64_t rows, int64_t cols, int group, int q, uint8_t* codes,
                      uint16_t* scales, int16_t* margin, float* gain) {
  int st = check_quantize(W, rows, cols, group, q, SSQ_SIGNED_SYM, codes, scales, nullptr);
  if (st == SSQ_OK && rows > 0 && cols > 0)
    st = margin == nullptr || gain == nullptr ? SSQ_EINVAL : !aligned(margin, 2) || !aligned(gain, 4) ? SSQ_EALIGN : SSQ_OK;
  if (st != SSQ_OK || rows == 0 || cols == 0) return st;
  return status_of(ssq::launch_quantize_diag_bf16(W, rows, cols, group, q, codes, scales, margin, gain, nullptr));
}

int ssq_quantize_diag_f32(const float* W, int64_t rows, int64_t cols, int group, int q, uint8_t* codes,
                          uint16_t* scales, int16_t* margin, float* gain) {
  int st = check_quantize(W, rows, cols, group, q, SSQ_SIGNED_SYM, codes, scales, nullptr);
  if (st == SSQ_OK && rows > 0 && cols > 0)
    st = margin == nullptr || gain == nullptr ? SSQ_EINVAL : !aligned(margin, 2) || !aligned(gain, 4) ? SSQ_EALIGN : SSQ_OK;
  if (st != SSQ_OK || rows == 0 || cols == 0) return st;
  return status_of(ssq::launch_quantize_diag_f32(W, rows, cols, group, q, codes, scales, margin, gain, nullptr));
}

int ssq_quantize_act_q8(const uint16_t* x, int64_t M, int64_t K, int8_t* q, uint16_t* d,
                        hipStream_t stream) {
  const int st = check_act_q8(x, M, K, q, d);
  if (st != SSQ_OK || M == 0 || K == 0) return st;
  return status_of(ssq::launch_quantize_act_q8(x, M, K, q, d, stream));
}

int ssq_matmul_q8(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                  const uint16_t* scales, const uint8_t* zp, int64_t N, int64_t K, int group, int q,
                  uint16_t* y, hipStream_t stream) {
  const int st = check_matmul_q8(qx, dx, M, codes, scales, N, K, group, q, y);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  return status_of(ssq::launch_matmul_q8(qx, dx, M, codes, scales, zero_points(zp), N, K, group, q, y, stream));
}

int ssq_matmul_q8_min(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                      const uint16_t* scales, const uint16_t* mins, int64_t N, int64_t K, int group, int q,
                      uint16_t* y, hipStream_t stream) {
  int st = check_matmul_q8(qx, dx, M, codes, scales, N, K, group, q, y);
  if (st == SSQ_OK) st = check_mins(mins, M > 0 && N > 0);
  if (st != SSQ_OK || M == 0 || N == 0) return st;
  return status_of(ssq::launch_matmul_q8(qx, dx, M, codes, scales, minimums(mins), N, K, group, q, y, stream));
}

int64_t ssq_gguf_block_bytes(int q, int with_min) {
  return q == 2 || q == 4 ? ssq::gguf_block_bytes(q, with_min != 0) : 0;
}

int ssq_export_gguf(const uint8_t* codes, const uint16_t* scales, const uint16_t* mins, int64_t rows,
                    int64_t cols, int group, int q, uint8_t* blocks, hipStream_t stream) {
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim || rows * cols > kMaxElems) return SSQ_EINVAL;
  if ((q != 2 && q != 4) || !valid_group(group) || cols % group != 0) return SSQ_EINVAL;
  if (rows == 0 || cols == 0) return SSQ_OK;
  if (codes == nullptr || scales == nullptr || blocks == nullptr) return SSQ_EINVAL;
  if (!aligned(codes, 16) || !aligned(scales, 2) || !aligned(blocks, 2) || (mins != nullptr && !aligned(mins, 2)))
    return SSQ_EALIGN;
  return status_of(ssq::launch_export_gguf(codes, scales, mins, rows, cols, group, q, blocks, stream));
}

const char* ssq_strerror(int status) {
  switch (status) {
    case SSQ_OK: return "success";
    case SSQ_EINVAL: return "invalid argument (size, q, group, mode, zero-point/mode mismatch or missing minimums)";
    case SSQ_EALIGN: return "misaligned pointer (W, x, y, codes need 16 bytes; scales, mins 2; workspace 256)";
    case SSQ_EHIP: return "HIP runtime error at kernel launch";
    case SSQ_ESCRATCH: return "the split reduction needs more than ssq_matmul_noalloc's 64 MiB static scratch "
                              "(use ssq_matmul_ws with a workspace)";
    default: return "unknown status";
  }
}

}  // extern "C"
