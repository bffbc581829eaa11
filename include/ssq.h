/*
 * ssq.h -- C ABI of libssq: group-wise signed symmetric few-bit weight
 * quantization and the weight-only dequantizing matmul, on AMD Instinct
 * MI355X (gfx950).
 *
 * Method: Colbert, Dash et al., "Signed Symmetric Quantization for Few-Bit
 * Integers".  Argument names follow the paper's notation: q (bit width),
 * group (g, the number of consecutive weights sharing one scale), scales (s),
 * zp (z, the zero point), mins (m, the group minimum of the Q*_1 layout).
 *
 * Storage format (shared by every entry point)
 * ---------------------------------------------
 *   W      [rows, cols]            row-major weights, groups of `group`
 *                                  consecutive entries along cols (the
 *                                  reduction index K of the matmul).
 *   codes  [rows, cols*q/8] u8     row-major; field k of a row occupies bits
 *                                  [k*q, k*q+q) of the row's little-endian bit
 *                                  stream (q=4: byte j = u[2j] | u[2j+1]<<4).
 *   scales [rows, cols/group] u16  IEEE binary16 bit patterns, one signed scale
 *                                  per group (App. B.1: the Q*_0 formats store
 *                                  s = gamma*alpha, which may be negative).
 *   zp     [rows, cols/group] u8   integer zero point, asymmetric mode only.
 *   mins   [rows, cols/group] u16  IEEE binary16 group minimum m, the *_min
 *                                  entry points only (App. B.1: the Q*_1 blocks
 *                                  store an fp16 scale and an fp16 minimum).
 *
 *   Symmetric modes store the offset-binary index u = c + 2^(q-1) of the code
 *   c in A_q = {-2^(q-1), ..., 2^(q-1)-1}; the weight is s*(u - 2^(q-1)).
 *   The asymmetric mode stores u in {0, ..., 2^q-1}; the weight is s*(u - z).
 *   The minimum layout stores u in {0, ..., 2^q-1}; the weight is s*u + m.
 *
 * Conventions
 *   - Every pointer is a device pointer owned by the caller.  The library
 *     allocates nothing, frees nothing and keeps no pointer after returning;
 *     scratch memory, where a path can use it, is a caller-provided workspace.
 *     The one exception is a static device array (about 90 KB per GPU, held
 *     until the process ends) in which ssq_sign_diagnostics meets its blocks
 *     to form the tally.
 *   - W, x, y and codes must be 16-byte aligned; scales and mins 2-byte aligned.
 *   - bf16 and fp16 tensors are passed as their uint16_t bit patterns.
 *   - Inputs must be finite; NaN/Inf inputs give unspecified codes.
 *   - Arguments are validated on the host before any launch.  On an error
 *     return nothing is launched and no output byte is written.
 *   - Calls are asynchronous; device faults surface at the caller's next
 *     synchronisation.  Calls never abort, exit or print.
 *   - Sizes of zero (rows or cols for quantize, M or N for matmul) are valid
 *     and do nothing.
 */
#ifndef SSQ_H
#define SSQ_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Quantization grid (Sec. 3). */
typedef enum {
  SSQ_SIGNED_SYM = 0,   /* signed absmax grid, sign rule of Eq. (5)            */
  SSQ_UNSIGNED_SYM = 1, /* absmax grid with s > 0, Eq. (3)                     */
  SSQ_ASYM = 2          /* min-max grid, Eq. (2), with a u8 zero point         */
} ssq_mode;

typedef enum {
  SSQ_OK = 0,
  SSQ_EINVAL = -1,      /* bad size, q, group, mode or zp/mode combination     */
  SSQ_EALIGN = -2,      /* a pointer violates the alignment rule above         */
  SSQ_EHIP = -3,        /* the HIP runtime reported an error at launch         */
  SSQ_ESCRATCH = -4     /* ssq_matmul_noalloc: split scratch above its maximum  */
} ssq_status;

/*
 * ssq_quantize -- quantize bf16 weights W[rows, cols] group by group.
 *
 * Per group of `group` consecutive weights w (Sec. 3; Eq. (1)-(5)):
 *   SSQ_SIGNED_SYM:   M = max|w|, alpha = M / 2^(q-1), gamma = -1 if the
 *                     largest-magnitude entry is positive and unique in
 *                     magnitude among opposite signs (max w > -min w), else +1;
 *                     s = gamma*alpha; c = clip(rne(fl32(w/s)), A_q).
 *   SSQ_UNSIGNED_SYM: the same with gamma = +1 (Eq. (3)).
 *   SSQ_ASYM:         min' = min(min w, 0), max' = max(max w, 0),
 *                     s = fl32(fl32(max' - min') / (2^q - 1)),
 *                     z = clip(rne(fl32(-min'/s)), 0, 2^q-1),
 *                     u = clip(rne(fl32(w/s)) + z, 0, 2^q-1).
 * Arithmetic is IEEE binary32 with round-half-to-even; the stored scale is
 * binary16(s) rounded half to even.  A group whose scale would be zero (all
 * entries zero) stores scale +0 and code 0 (index 2^(q-1), or 0 for ASYM).
 *
 *   W      device, bf16 bits [rows, cols] row-major, read only
 *   rows   >= 0, number of weight rows (output channels N)
 *   cols   >= 0, multiple of group (reduction length K)
 *   group  32, 64 or 128
 *   q      2, 3 or 4
 *   mode   ssq_mode
 *   codes  device, u8 [rows, cols*q/8], written
 *   scales device, u16 [rows, cols/group], written
 *   zp     device, u8 [rows, cols/group], written; must be non-NULL iff
 *          mode == SSQ_ASYM
 * Enqueued on the null stream.  Returns SSQ_OK or a negative ssq_status.
 */
int ssq_quantize(const uint16_t* W, int64_t rows, int64_t cols, int group, int q, int mode,
                 uint8_t* codes, uint16_t* scales, uint8_t* zp);

/* ssq_quantize for binary32 weights W[rows, cols]; otherwise identical. */
int ssq_quantize_f32(const float* W, int64_t rows, int64_t cols, int group, int q, int mode,
                     uint8_t* codes, uint16_t* scales, uint8_t* zp);

/*
 * ssq_matmul -- y[M, N] = x[M, K] * What[N, K]^T, where What is the
 * dequantized weight (App. B.3):
 *   What[n, k] = fp32(scales[n, b]) * (u[n, k] - o[n, b]),   b = k / group,
 *   o = 2^(q-1) when zp == NULL (symmetric formats, signed or not: the sign
 *   lives in the scale, so both run the same kernel), o = zp[n, b] otherwise.
 * Products accumulate in fp32; y is rounded to bf16 (half to even).
 * M = 1 and M = 2 run a streaming GEMV (two tokens share each unpacked block);
 * 3 <= M <= 32 (batched decode) shares each weight among the tokens through bf16
 * MFMA: for q = 2 or 4, M <= 16 and K a multiple of 512 (with a workspace, or
 * K <= 2048) the weights enter exactly (the code as 128 + u, the scale and offset
 * applied per 32-weight block in fp32), otherwise each weight is dequantized once
 * and rounded to bf16; larger M runs a tiled kernel that dequantizes weight tiles
 * into LDS and multiplies them with bf16 MFMA.
 *
 *   x      device, bf16 bits [M, K] row-major, read only
 *   M      >= 0, number of activation rows (tokens)
 *   codes  device, u8 [N, K*q/8] as written by ssq_quantize
 *   scales device, u16 [N, K/group]
 *   zp     device, u8 [N, K/group] for the asymmetric format, else NULL
 *   N      >= 0, number of weight rows (outputs)
 *   K      > 0, multiple of group, at most 2^22
 *   group  32, 64 or 128;  q  2, 3 or 4
 *   y      device, bf16 bits [M, N] row-major, written
 *   stream HIP stream the kernels are enqueued on (NULL: null stream)
 */
int ssq_matmul(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
               const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
               hipStream_t stream);

/*
 * ssq_matmul_workspace_size -- bytes of workspace that let ssq_matmul_ws split
 * the reduction of an M x N x K product across workgroups (App. B.3 sums over
 * blocks of K, so disjoint block ranges can be reduced separately and added).
 * Returns 0 when splitting would not help (M <= 2: the streaming GEMV, or enough
 * output tiles already) or the arguments are invalid.  3 <= M <= 32 sizes the
 * batched-decode kernel's split, larger M the tiled kernel's.
 */
size_t ssq_matmul_workspace_size(int64_t M, int64_t N, int64_t K, int group, int q);

/*
 * ssq_matmul_ws -- ssq_matmul with a caller-provided device workspace.  With a
 * workspace of at least ssq_matmul_workspace_size() bytes the GEMM splits its
 * reduction; with a smaller one, or NULL, it behaves exactly like ssq_matmul.
 *   workspace       device, 256-byte aligned, zero-filled by the caller before
 *                   its first use; every call leaves it reusable (the arrival
 *                   counters it holds return to zero).  Two calls that may run
 *                   concurrently must not share a workspace.
 *   workspace_bytes size of the workspace in bytes
 * Other arguments, results and errors as ssq_matmul (plus SSQ_EALIGN for a
 * misaligned workspace).  The split adds fp32 partials in a fixed order, so
 * results are reproducible, but y can differ from ssq_matmul's in the last
 * bf16 bit (a different summation order).
 */
int ssq_matmul_ws(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                  const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
                  void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * ssq_matmul_noalloc -- ssq_matmul_ws without a caller workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The split reduction uses a static device array
 * of the library instead: 64 MiB per GPU the library runs on, held until the process
 * ends.  The call itself allocates nothing (no hipMalloc, hipFree or allocating
 * library routine).
 *   x, M, codes, scales, zp, N, K, group, q, y, stream   as ssq_matmul; the current
 *                   device must be the device of `stream`
 * Results equal ssq_matmul_ws's with a workspace of ssq_matmul_workspace_size()
 * bytes, bit for bit.  Returns SSQ_ESCRATCH, launching nothing, when that size
 * exceeds 64 MiB; otherwise as ssq_matmul_ws.  Every call on one GPU shares that
 * GPU's array and leaves its arrival counters at zero; calls that may overlap on
 * one GPU (other streams, other threads) race and must not be issued.  The first
 * call on a device also enqueues a small kernel on `stream` that clears the counters.
 */
int ssq_matmul_noalloc(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                       const uint8_t* zp, int64_t N, int64_t K, int group, int q, uint16_t* y,
                       hipStream_t stream);

/* ssq_matmul with binary32 x[M, K] and y[M, N] (fp32 accumulation and output). */
int ssq_matmul_f32(const float* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                   const uint8_t* zp, int64_t N, int64_t K, int group, int q, float* y,
                   hipStream_t stream);

/*
 * The min-max grid in the layout of App. B.1's Q4_1 / Q2_1 rows: an fp16 scale and
 * an fp16 minimum per group (20 bytes per 32 weights at q=4, 12 at q=2), the
 * weight reading back as s*u + m.
 *
 * ssq_quantize_min -- per group of `group` consecutive weights w (Eq. (2) on the
 * group's own range, Eq. (1) with the real zero point z = -min/s):
 *   s = fl32(fl32(max w - min w) / (2^q - 1)),
 *   u = clip(rne(fl32(fl32(w - min w) / s)), 0, 2^q-1),
 *   scales = binary16(s), mins = binary16(min w) (both half to even; a minimum
 *   that is or rounds to a zero is stored as +0).
 * A constant group stores s = 0, codes 0 and its value as the minimum.
 *   W, rows, cols, group, q, codes, scales   as ssq_quantize
 *   mins   device, u16 [rows, cols/group], written; 2-byte aligned, non-NULL
 * Enqueued on the null stream.  Returns SSQ_OK or a negative ssq_status.
 */
int ssq_quantize_min(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                     uint8_t* codes, uint16_t* scales, uint16_t* mins);

/* ssq_quantize_min for binary32 weights W[rows, cols]; otherwise identical. */
int ssq_quantize_min_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                         uint8_t* codes, uint16_t* scales, uint16_t* mins);

/*
 * ssq_matmul_min, ssq_matmul_min_ws, ssq_matmul_min_f32 -- ssq_matmul,
 * ssq_matmul_ws and ssq_matmul_f32 for weights in the minimum layout:
 *   What[n, k] = fp32(scales[n, b]) * u[n, k] + fp32(mins[n, b]),   b = k / group,
 * so each block adds m * sum_{k in b} x[k] to the symmetric product (App. B.3).
 *   mins   device, u16 [N, K/group] binary16 minimums, 2-byte aligned, non-NULL
 * Every other argument, the kernels chosen by M, the workspace rules and the
 * errors are those of the corresponding entry point above.
 */
int ssq_matmul_min(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                   const uint16_t* mins, int64_t N, int64_t K, int group, int q, uint16_t* y,
                   hipStream_t stream);
int ssq_matmul_min_ws(const uint16_t* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                      const uint16_t* mins, int64_t N, int64_t K, int group, int q, uint16_t* y,
                      void* workspace, size_t workspace_bytes, hipStream_t stream);
int ssq_matmul_min_f32(const float* x, int64_t M, const uint8_t* codes, const uint16_t* scales,
                       const uint16_t* mins, int64_t N, int64_t K, int group, int q, float* y,
                       hipStream_t stream);

/*
 * ssq_sign_diagnostics -- the statistics of Sec. 4 Remark 1 (Fig. 1) for every
 * group of the signed absmax grid: with gamma* the sign rule of Eq. (5) (ties
 * +1), alpha = M / 2^(q-1), T = M (1 - 2^-q) and the clipped sets of Def. 1,
 * C_gamma = {i : gamma w_i > T} (Eq. (6)):
 *   margin[g] = |C_{-gamma*}| - |C_{gamma*}|            (the cardinality margin m(w))
 *   gain[g]   = ||w - Q_{-gamma*}(w)||^2 - ||w - Q_{gamma*}(w)||^2
 *             = 2 alpha (sum_{C_{-gamma*}} (-gamma* w_i - T) - sum_{C_{gamma*}} (gamma* w_i - T))
 *                                                       (the realised gain g(w), Lemma 1)
 * Margin is exact; the gain's terms and sums are exact (integer multiples of a
 * power of two) and only the final product rounds, to binary64 and then to the
 * stored binary32 (an exact zero gain may be stored as +0 or -0).  m >= 0 is
 * Corollary 1's condition for gamma* minimising the worst-case bound; g > 0 means
 * gamma* also lowers the realised l2 error.
 *
 *   W      device, bf16 bits [rows, cols] row-major, read only (16-byte aligned)
 *   rows, cols, group, q   as ssq_quantize
 *   margin device, int16 [rows, cols/group], written (2-byte aligned)
 *   gain   device, float [rows, cols/group], written (4-byte aligned)
 *   tally  device, uint64 [9] or NULL: counts of groups by the signs of the stored
 *          margin and gain, tally[(sign(m) + 1) * 3 + (sign(g) + 1)]; overwritten,
 *          all zero when rows or cols is 0 (8-byte aligned)
 * Weights must be finite.  Enqueued on the null stream, so calls on one device run
 * one after another: the tally's per-block counts and arrival counter live in a
 * static device array that consecutive calls reuse.  Returns SSQ_OK or a negative
 * ssq_status (SSQ_EINVAL also past about 2^38 weights).
 */
int ssq_sign_diagnostics(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                         int16_t* margin, float* gain, uint64_t* tally);

/* ssq_sign_diagnostics for binary32 weights W[rows, cols]; otherwise identical. */
int ssq_sign_diagnostics_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                             int16_t* margin, float* gain, uint64_t* tally);

/*
 * ssq_quantize_diag -- ssq_quantize with mode SSQ_SIGNED_SYM fused with the
 * sign-rule margin and gain of ssq_sign_diagnostics (Sec. 4 Remark 1): one pass over
 * W writes the same codes and scales as ssq_quantize and the same margin and gain as
 * ssq_sign_diagnostics (no tally: count the outputs, or call ssq_sign_diagnostics).
 *
 *   W, rows, cols, group, q, codes, scales   as ssq_quantize (signed symmetric)
 *   margin device, int16 [rows, cols/group], written (2-byte aligned)
 *   gain   device, float [rows, cols/group], written (4-byte aligned)
 * Enqueued on the null stream.  Returns SSQ_OK or a negative ssq_status.
 */
int ssq_quantize_diag(const uint16_t* W, int64_t rows, int64_t cols, int group, int q,
                      uint8_t* codes, uint16_t* scales, int16_t* margin, float* gain);

/* ssq_quantize_diag for binary32 weights W[rows, cols]; otherwise identical. */
int ssq_quantize_diag_f32(const float* W, int64_t rows, int64_t cols, int group, int q,
                          uint8_t* codes, uint16_t* scales, int16_t* margin, float* gain);

/*
 * ssq_quantize_act_q8 -- dynamic Q8_0 activation quantization (Sec. 5.2, App. C):
 * per token and block of 32 activations the narrow-range symmetric grid
 * {-127, ..., 127}, d = amax / 127 (binary32), q = clip(rne(x / d), -127, 127)
 * computed from that d (Eq. (1) with z = 0), stored scale binary16(d); an all-zero
 * block stores d = +0 and codes 0.
 *
 *   x      device, bf16 bits [M, K] row-major, read only (16-byte aligned)
 *   M, K   tokens and activations per token; K a multiple of 32
 *   q      device, int8 [M, K], written (16-byte aligned)
 *   d      device, binary16 bits [M, K/32], written (2-byte aligned)
 *   stream HIP stream the kernel is enqueued on (0 = null stream)
 * Returns SSQ_OK or a negative ssq_status.
 */
int ssq_quantize_act_q8(const uint16_t* x, int64_t M, int64_t K, int8_t* q, uint16_t* d,
                        hipStream_t stream);

/*
 * ssq_matmul_q8 -- y[M, N] = X W^T with Q8_0 activations and packed weights, by
 * App. B.3's split into the integer GEMM term and the row-sum correction: for each
 * block b of 32 activations inside weight group g,
 *   I = sum_{j in b} qx[m, j] u[n, j],  R = sum_{j in b} qx[m, j]     (exact integers)
 *   y[m, n] += d[m, b] s[n, g] (I - o[n, g] R)
 * with o = 2^(q-1) (zp == NULL: the symmetric formats) or the zero point zp[n, g].
 * Exact integer block terms (4-way byte dot products at M = 1; int8 MFMA, v_mfma_i32_16x16x32_i8,
 * for 2 <= M, where up to 32 tokens share one read of the weights and K <= 32768; longer
 * rows take the M = 1 kernel per token); fp32 accumulation; y rounded to bf16 once.
 *
 *   qx, dx codes and scales from ssq_quantize_act_q8 ([M, K] int8, 16-byte aligned;
 *          [M, K/32] binary16, 2-byte aligned)
 *   codes, scales, zp, N, K, group, q, y   as ssq_matmul
 * Returns SSQ_OK or a negative ssq_status.
 */
int ssq_matmul_q8(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                  const uint16_t* scales, const uint8_t* zp, int64_t N, int64_t K, int group, int q,
                  uint16_t* y, hipStream_t stream);

/* ssq_matmul_q8 for the binary16-minimum layout: y[m, n] += d[m, b] (s[n, g] I +
 * mins[n, g] R); mins as ssq_matmul_min (required when M, N > 0). */
int ssq_matmul_q8_min(const int8_t* qx, const uint16_t* dx, int64_t M, const uint8_t* codes,
                      const uint16_t* scales, const uint16_t* mins, int64_t N, int64_t K, int group,
                      int q, uint16_t* y, hipStream_t stream);

/*
 * ssq_export_gguf -- the packed weights as llama.cpp GGUF blocks (App. B.1, formats
 * table; App. B.2 notes that quantized models can be exported to that runtime).  Per 32
 * weights of a row, one array-of-structures block: binary16 s, then (mins != NULL) a
 * binary16 m, then the block's indices qs:
 *   q = 4: Q4_0 / Q4_0s 18 bytes {s, qs[16]};  with mins Q4_1 20 bytes {s, m, qs[16]}
 *   q = 2: Q2_0 / Q2_0s 10 bytes {s, qs[8]};   with mins Q2_1 12 bytes {s, m, qs[8]}
 * The signed-symmetric variant (Q*_0s) is the Q*_0 layout with a scale that may be
 * negative.  qs order: q = 4 byte j = index j | index (j+16) << 4 (j < 16); q = 2
 * byte i = indices 4i..4i+3 at bits 0, 2, 4, 6.  A weight reads back as s*(u - 2^(q-1))
 * (Q*_0) or s*u + m (Q*_1), as in this library.  With group 64 or 128 every 32-weight
 * block repeats its group's s (and m).  Blocks are row-major: row r's blocks first.
 *
 *   codes, scales, mins  device, as ssq_quantize (SSQ_SIGNED_SYM or SSQ_UNSIGNED_SYM)
 *                        or ssq_quantize_min wrote them; mins NULL for the symmetric
 *                        formats.  The zero-point layout (SSQ_ASYM) has no GGUF form.
 *   rows, cols, group, q q in {2, 4} (GGUF has no 3-bit block in the table)
 *   blocks               device, written: rows * cols/32 * ssq_gguf_block_bytes(q, mins
 *                        != NULL) bytes (2-byte aligned; codes 16, scales and mins 2)
 *   stream               HIP stream
 * Returns SSQ_OK, SSQ_EINVAL (q = 3, bad sizes, missing pointer) or SSQ_EALIGN.
 */
int ssq_export_gguf(const uint8_t* codes, const uint16_t* scales, const uint16_t* mins, int64_t rows,
                    int64_t cols, int group, int q, uint8_t* blocks, hipStream_t stream);

/* Bytes of one GGUF block of ssq_export_gguf: 18, 20 (q = 4), 10, 12 (q = 2) without and
 * with a minimum; 0 for any other q. */
int64_t ssq_gguf_block_bytes(int q, int with_min);

/* Static description of a status code; never NULL. */
const char* ssq_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* SSQ_H */
