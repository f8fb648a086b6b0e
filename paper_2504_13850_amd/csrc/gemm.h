// bf16 MFMA GEMM / implicit-GEMM convolution for gfx950.
//
//   C[m][n] = sum_k A(m,k) * B(n,k)        fp32 accumulation
//
// A and B are read through "loaders" that describe where element (row, k)
// lives, so one kernel serves linear layers (forward, input gradient, weight
// gradient) and NHWC convolutions as implicit GEMMs (forward, input gradient,
// weight gradient) without materialising im2col matrices.
#pragma once

#include "common.h"

namespace fo {

enum OperandMode : int {
    OP_RK = 0,        // element (r,k) at P[r*ld + k]     (k contiguous)
    OP_KR = 1,        // element (r,k) at P[k*ld + r]     (r contiguous)
    OP_CONV_FWD = 2,  // A of a conv forward:  r = output pixel, k = (ky,kx,ci); P = input NHWC
    OP_CONV_DX = 3,   // A of a conv dgrad:    r = input pixel,  k = (ky,kx,co); P = dY NHWC
    OP_CONV_DXW = 4,  // B of a conv dgrad:    r = ci,           k = (ky,kx,co); P = W [co][ky][kx][ci]
    OP_CONV_DWX = 5,  // B of a conv wgrad:    r = (ky,kx,ci),   k = output pixel; P = input NHWC
};

struct ConvGeom {
    int Bn = 0, H = 0, W = 0, Ci = 0;  // input  [Bn][H][W][Ci]
    int Ho = 0, Wo = 0, Co = 0;        // output [Bn][Ho][Wo][Co]
    int kh = 1, kw = 1, stride = 1, pad = 0;
};

enum Act : int { ACT_NONE = 0, ACT_RELU = 1, ACT_GELU = 2 };

struct GemmDesc {
    int M = 0, N = 0, K = 0;
    int amode = OP_RK, bmode = OP_RK;
    const bf16_t* A = nullptr;
    int64_t lda = 0;
    const bf16_t* B = nullptr;
    int64_t ldb = 0;
    // Compensated (split-bf16) products: with A2 / B2 the low parts of A / B
    // (x = hi + lo, hi = bf16(x), lo = bf16(x - hi)), nseg = 3 accumulates
    // A.B + A.B2 + A2.B over three K segments: the result carries about 16
    // bits of operand precision instead of 8 (the lo.lo term is below it).
    // nseg = 2 keeps the first two segments (for an A that is exactly bf16).
    const bf16_t* A2 = nullptr;
    const bf16_t* B2 = nullptr;
    int nseg = 1;
    ConvGeom g;
    // epilogue, applied in this order: + bias[n], + resid[m][n] (fp32),
    // act (GELU also stores its derivative at the input, GELU'(x), to `dact_out`
    // when set), * [mask[m][n] > 0], * dact[m][n] (a stored activation
    // derivative); then stores to Cf (fp32) and/or Cb (bf16).
    const float* bias = nullptr;
    const float* resid = nullptr;
    int64_t ldr = 0;
    int act = ACT_NONE;
    bf16_t* dact_out = nullptr;
    const bf16_t* mask = nullptr;
    const bf16_t* dact = nullptr;
    int64_t ldm = 0;  // leading dimension of dact_out / mask / dact
    float* Cf = nullptr;
    int64_t ldcf = 0;
    bf16_t* Cb = nullptr;   // bf16(v)
    bf16_t* Cb2 = nullptr;  // bf16(v - bf16(v)), the low part (same leading dimension)
    int64_t ldcb = 0;
    // Fused SGD (Alg. 4's update) on a weight gradient stored in the weight's
    // own layout (Cf, leading dimension ldcf): after the store, theta[m][n]
    // becomes fma(-sgd_lr, v, theta[m][n]) and its bf16 high and low parts go to
    // sgd_hi / sgd_lo (same indexing).  Needs Cf.
    float* sgd_theta = nullptr;
    bf16_t* sgd_hi = nullptr;
    bf16_t* sgd_lo = nullptr;
    float sgd_lr = 0.f;
    // Column sums of the stored value: colpart[m / 128][n] = sum of v over the
    // valid rows of that 128-row tile (no split-K); launch_colsum_finish with
    // rows_per_part 128 completes them.
    float* colpart = nullptr;
    // split-K: z-slices write fp32 partials to ws[z][M][N]; a second pass sums
    // them and runs the epilogue.
    int splits = 1;
    float* ws = nullptr;
    // Optional device-side bounds (packed variable-length batches): the
    // effective M (or K) is min(M, *Mdev) (or min(K, *Kdev)); the grid is
    // sized by the static M, and tiles past the effective bound do nothing.
    const int* Mdev = nullptr;
    const int* Kdev = nullptr;
    int* prof_snap = nullptr;  // set by the launcher when profiling: receives (M, K) effective
    int vec_epi = 0;           // set by the launcher: the epilogue may move four columns per access
    // With split-K: leave the partials in ws and skip the reduction pass; the
    // consumer sums them (see SplitRows).  A launch that runs unsplit (one
    // active slice) still applies its epilogue and writes Cf.
    bool defer_reduce = false;
};

// Split-K slices a launch with a device-side row bound M_eff uses: as many as
// keep two workgroups per CU busy over the active 128 x 128 tiles, each slice
// at least four 64-long K tiles (ktot: the reduction length including the
// compensated segments).  With a static row count every launched slice is used.
__device__ __forceinline__ int gemm_active_splits(int splits, int M_eff, int N, int ktot) {
    if (splits <= 1) return splits;
    const int tiles = ((M_eff + 127) / 128) * ((N + 127) / 128);
    int s = min(splits, max(1, 512 / max(tiles, 1)));
    while (s > 1 && ktot < 4 * 64 * s) --s;
    return s;
}

// A product's rows as a consumer reads them when the producing GEMM deferred
// its split-K reduction: row r = x[r] if the launch ran unsplit, else
// (sum of ws[z][r] over the active slices, in the reduction pass's order)
// + bias + resid[r].  N columns, leading dimension N everywhere.
struct SplitRows {
    const float* x = nullptr;
    const float* ws = nullptr;    // [splits][M][N] (NULL: x only)
    const float* bias = nullptr;  // [N] or NULL
    const float* resid = nullptr; // [M][N] or NULL
    int M = 0, N = 0, splits = 1, ktot = 0;
    __device__ int active(int M_eff) const { return ws ? gemm_active_splits(splits, M_eff, N, ktot) : 1; }
};

// Enqueues the GEMM (and its split-K reduction) on stream s.
fo_status gemm(const GemmDesc& d, hipStream_t s);

// Enqueues n <= kGemmGroupMax independent products.  When all of them are
// unsplit products of aligned k-major operands (weight gradients) they run as
// one launch over the concatenation of their output tiles, each tile over its
// whole K (no split-K partials, no reduction pass); otherwise one launch each.
// max_wg > 0 caps the workgroups of the grouped launch (rounded down to a
// multiple of 8); they then walk the tiles in rounds, leaving workgroup slots
// to work on other streams.
constexpr int kGemmGroupMax = 4;
fo_status gemm_group(const GemmDesc* d, int n, hipStream_t s, int max_wg = 0);

// Deferred split-K sums of several products with a plain epilogue (no bias,
// activation or mask: a weight gradient): job i adds slices 0 .. S_i - 1 of
// ws_i ([S_i][M_i][N_i], as a launch with defer_reduce left them) into
// C_i[m][n] = C_i[m ldc_i + n], in splitk_reduce's order.  One launch for up to
// kSplitJobsMax products.
constexpr int kSplitJobsMax = 48;
struct SplitJob {
    const float* ws = nullptr;
    float* C = nullptr;
    int64_t ldc = 0;
    int S = 1, M = 0, N = 0;
};
struct SplitJobs {
    SplitJob j[kSplitJobsMax];
    int n = 0;
};
fo_status launch_splitk_sum_multi(const SplitJobs& jobs, hipStream_t s);

// Bytes of split-K workspace a descriptor needs (0 if splits == 1).
inline size_t gemm_ws_bytes(int M, int N, int splits) {
    return splits > 1 ? sizeof(float) * (size_t)M * N * splits : 0;
}

}  // namespace fo
