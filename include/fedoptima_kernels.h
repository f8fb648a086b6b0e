/*
 * fedoptima_kernels.h -- kernel-level entry points of libfedoptima (testing,
 * tuning and benchmarking of the matrix-core kernels in isolation).
 *
 * Each call enqueues one pass of the bf16 MFMA GEMM that the server steps use
 * (the forward, input-gradient and weight-gradient products of Alg. 4's
 * training iteration) on `hip_stream` and returns at once.  All pointers are
 * device memory; bf16 operands are uint16 bit patterns; outputs are fp32.
 * Arguments are checked on the host (FO_EINVAL before any launch).
 */
#ifndef FEDOPTIMA_KERNELS_H
#define FEDOPTIMA_KERNELS_H

#include "fedoptima.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Operand layouts for fo_gemm_bf16. */
enum { FO_LAYOUT_ROW_K = 0,   /* element (r, k) at P[r * ld + k]  (k contiguous)  */
       FO_LAYOUT_K_ROW = 1 }; /* element (r, k) at P[k * ld + r]  (r contiguous)  */

/* C[m][n] = sum_k A(m, k) B(n, k), C row-major with leading dimension ldc.
 * With A_lo and B_lo (the bf16 low parts of A and B, x = hi + lo) the product
 * is the compensated sum A.B + A.B_lo + A_lo.B (A_lo may be NULL for an exactly
 * bf16 A; B_lo NULL means a plain product).  splits > 1 divides K over that many
 * workgroup slices whose fp32 partials (workspace: splits * M * N floats) are
 * summed afterwards.  M, N, K >= 1. */
FO_API fo_status fo_gemm_bf16(int32_t M, int32_t N, int32_t K, int32_t a_layout, const uint16_t* A,
                              const uint16_t* A_lo, int64_t lda, int32_t b_layout, const uint16_t* B,
                              const uint16_t* B_lo, int64_t ldb, float* C, int64_t ldc, int32_t splits,
                              float* workspace, void* hip_stream);

/* fo_gemm_bf16 for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same product with the same kernels and results, and no workspace argument.
 * Split-K partials go to a 16 MiB array that the library's code object holds
 * on every GPU it is loaded on, from load until the process ends; so
 * splits * M * N must not exceed 4,194,304 floats (FO_EINVAL otherwise,
 * nothing launched).  splits == 1 uses no scratch.  The call allocates
 * nothing: its first call on a device looks up that device's copy of the
 * array (hip_stream must belong to the current device, else FO_EINVAL).
 * Every slice writes all of its partials before they are summed, so nothing
 * needs clearing between calls; but all calls on one GPU share the one array,
 * so calls whose split-K work overlaps in time on one GPU (on different
 * streams, or from different threads) race, and must be ordered by the
 * caller.  Other arguments and errors as fo_gemm_bf16. */
FO_API fo_status fo_gemm_bf16_noalloc(int32_t M, int32_t N, int32_t K, int32_t a_layout, const uint16_t* A,
                                      const uint16_t* A_lo, int64_t lda, int32_t b_layout, const uint16_t* B,
                                      const uint16_t* B_lo, int64_t ldb, float* C, int64_t ldc, int32_t splits,
                                      void* hip_stream);

/* One pass of a 2-D convolution (cross-correlation) in NHWC layout as an
 * implicit GEMM; weights are [Co][k][k][Ci].
 *   pass 0 (forward):          out[Bn][Ho][Wo][Co] = conv(x, w)           x = in [Bn][H][W][Ci]
 *   pass 1 (input gradient):   out[Bn][H][W][Ci]  = conv^T(dy, w)         dy = in [Bn][Ho][Wo][Co]
 *   pass 2 (weight gradient):  out[Co][k][k][Ci]  = sum over pixels dy (x) x   (in = dy, in2 = x)
 * Ho = (H + 2 pad - k) / stride + 1 (same for W).  For pass 0, in_lo / w_lo give
 * compensated products as in fo_gemm_bf16.  Requires Ci % 64 == 0 (pass 0),
 * Co % 64 == 0 (pass 1) and Ci % 8 == 0.  splits / workspace as above (workspace
 * floats: splits * rows * cols of the pass's output matrix). */
FO_API fo_status fo_conv2d_bf16(int32_t pass, int32_t Bn, int32_t H, int32_t W, int32_t Ci, int32_t Co, int32_t k,
                                int32_t stride, int32_t pad, const uint16_t* in, const uint16_t* in_lo,
                                const uint16_t* in2, const uint16_t* w, const uint16_t* w_lo, float* out,
                                int32_t splits, float* workspace, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* FEDOPTIMA_KERNELS_H */
