// Host-side launchers of the HIP kernels (each defined in a k_*.hip file).
#pragma once

#include <algorithm>

#include "common.h"

namespace fo {

// ------------------------------------------------------------------ k_update.hip
constexpr int kAggMaxFused = 64;
struct AggTable {
    int count;
    const float* local[kAggMaxFused];
    float w[kAggMaxFused];
};
fo_status launch_agg_lerp(float* g, const float* l, int64_t n, float w, hipStream_t s);
// One activation batch (bytes, a multiple of 16; 16-byte aligned device
// pointers), its labels and (if len_src) lengths into a pool slot: one launch.
fo_status launch_pool_put(const void* x_src, void* x_dst, int64_t bytes, const int32_t* lab_src, int32_t* lab_dst,
                          const int32_t* len_src, int32_t* len_dst, int batch, hipStream_t s);
// Several admitted batches (same slot size) in one launch.
constexpr int kPutMaxBatches = 32;
struct PutTable {
    const uint4* xs[kPutMaxBatches];
    uint4* xd[kPutMaxBatches];
    const int32_t* ls[kPutMaxBatches];
    int32_t* ld[kPutMaxBatches];
    const int32_t* ns[kPutMaxBatches];
    int32_t* nd[kPutMaxBatches];
    int count;
};
fo_status launch_pool_put_gather(const PutTable& t, int64_t bytes, int batch, hipStream_t s);
fo_status launch_agg_lerp_multi(float* g, const AggTable& tab, int64_t n, hipStream_t s);
// theta -= lr * g (momentum v <- mu v + g first when v is set); refreshes the
// bf16 high/low shadows of theta when w16/w16lo are set.
fo_status launch_sgd(float* p, const float* g, float* v, bf16_t* w16, bf16_t* w16lo, int64_t n, float lr, float mu,
                     hipStream_t s);
// The same update on the ranges [chunks[2i], chunks[2i] + chunks[2i + 1]) (device
// array, one block per range).
fo_status launch_sgd_chunks(float* p, const float* g, bf16_t* w16, bf16_t* w16lo, const int64_t* chunks,
                            int nchunks, float lr, hipStream_t s);
// y = bf16(x), ylo = bf16(x - y) (ylo may be NULL)
fo_status launch_cast_bf16(const float* x, bf16_t* y, bf16_t* ylo, int64_t n, hipStream_t s);

// ------------------------------------------------------------------ k_attn.hip
// qkv / qkvlo [T][3d] bf16 high and low parts of the projection, cu int32[B+1]
// packed-row offsets (sequences <= 128 tokens, head width 64); out / outlo [T][d]
// bf16 high and low parts of the output; lse fp32 [B][H][128] (natural log);
// dout the bf16 output gradient, dqkv bf16 [T][3d].  The backward reads the
// high parts only.
// order (device, optional): the sequences in the order their workgroups are
// launched, e.g. longest first so that short ones fill in behind long ones.
fo_status launch_attn_fwd(const bf16_t* qkv, const bf16_t* qkvlo, const int* cu, bf16_t* out, bf16_t* outlo,
                          float* lse, int B, int H, int d, hipStream_t s, const int* order = nullptr);
fo_status launch_attn_bwd(const bf16_t* qkv, const int* cu, const bf16_t* out, const bf16_t* dout,
                          const float* lse, bf16_t* dqkv, int B, int H, int d, hipStream_t s,
                          const int* order = nullptr);
// The same attention for the first token of each sequence only (the last
// encoder layer, read at token 0 alone): out / outlo and lse are compact
// ([B][d], [B][H]); the backward writes every row of dqkv (the query part of
// rows past the first is zero).
fo_status launch_attn_cls_fwd(const bf16_t* qkv, const bf16_t* qkvlo, const int* cu, bf16_t* out, bf16_t* outlo,
                              float* lse, int B, int H, int d, hipStream_t s);
fo_status launch_attn_cls_bwd(const bf16_t* qkv, const bf16_t* qkvlo, const int* cu, const bf16_t* out,
                              const bf16_t* outlo, const bf16_t* dout, const float* lse, bf16_t* dqkv, int B, int H,
                              int d, hipStream_t s);

// ------------------------------------------------------------------ k_common.hip
// mean cross-entropy of logits z [B][C] and dz = (softmax - onehot)/B into
// loss[0]; loss[1] receives the number of labels outside [0, C) (each clamped
// to the nearest class so that every access stays in bounds)
// (labels: in->labels, device int32[B])
fo_status launch_xent(const float* z, const StepIn* in, float* dz, float* loss, int B, int C, hipStream_t s);
// out[c] = sum over rows r < min(rows, *rows_dev) of X[r*ld + c]; ws holds colsum_ws_floats(rows, N)
size_t colsum_ws_floats(int rows, int N);
fo_status launch_colsum(const float* X, int64_t ld, int rows, const int* rows_dev, int N, float* out, float* ws,
                        hipStream_t s);
fo_status launch_colsum(const bf16_t* X, int64_t ld, int rows, const int* rows_dev, int N, float* out, float* ws,
                        hipStream_t s);
// Destination of a column-sum finish: column c goes to p[c / seg][c % seg] (up to three outputs).
struct ColOut {
    float* p[3] = {nullptr, nullptr, nullptr};
    int seg = 0;
};
// Adds partial rows part[p][N] over p < ceil(min(rows, *rows_dev) / rows_per_part), in order.
fo_status launch_colsum_finish(const float* part, int rows, const int* rows_dev, int rows_per_part, int N,
                               const ColOut& out, hipStream_t s);
// Several finishing passes in one launch: job i adds the partial rows of part_i
// (as launch_colsum_finish) into out_i; at most kColJobsMax jobs.
constexpr int kColJobsMax = 16;
struct ColJob {
    const float* part = nullptr;
    int rows = 0, rows_per_part = 1, N = 0;
    const int* rows_dev = nullptr;
    ColOut out;
};
struct ColJobs {
    ColJob j[kColJobsMax];
    int n = 0;
};
fo_status launch_colsum_finish_multi(const ColJobs& jobs, hipStream_t s);
// Several first passes of launch_colsum (fp32 matrices) in one launch: job i
// writes the partial rows of X_i [rows_i][N_i] (leading dimension ld_i) to
// part_i, with colsum_partial's arithmetic; at most kColJobsMax jobs.
struct ColPartJob {
    const float* X = nullptr;
    int64_t ld = 0;
    int rows = 0, N = 0;
    float* part = nullptr;
};
struct ColPartJobs {
    ColPartJob j[kColJobsMax];
    int n = 0;
};
fo_status launch_colsum_partial_multi(const ColPartJobs& jobs, hipStream_t s);
// A pass over several fp32 matrices: adds each X_i's column sums to out_i,
// as launch_colsum would, in two launches whatever the count (part_i holds
// colsum_ws_floats(rows_i, N_i) floats each, distinct).
struct ColSums {
    ColPartJobs parts;
    ColJobs fin;
    void add(const float* X, int64_t ld, int rows, int N, float* part, float* out);
};
fo_status launch_colsums(const ColSums& c, hipStream_t s);
// The first pass of launch_colsum alone: ws receives the partial rows (CS_ROWS
// rows each) that launch_colsum_finish (rows_per_part = colsum_rows_per_part())
// completes.
fo_status launch_colsum_partial(const bf16_t* X, int64_t ld, int rows, const int* rows_dev, int N, float* ws,
                                hipStream_t s);
int colsum_rows_per_part();
fo_status launch_fill(float* p, int64_t n, float v, hipStream_t s);
// y = x w^T + bias (tanh when tanh_act) for x [B][I], w [O][I], I <= 768
fo_status launch_small_linear_fwd(const float* x, const float* w, const float* bias, float* y, int B, int I, int O,
                                  bool tanh_act, hipStream_t s);
// gw = dy^T x, gb = colsum dy, dx = (dy W) * (1 - xin_tanh^2 if given); dx may be NULL.
// ws holds small_linear_ws_floats(B, I, O) floats when dx is set.
size_t small_linear_ws_floats(int B, int I, int O);
fo_status launch_small_linear_bwd(const float* dy, const float* x, const float* w, const float* xin_tanh, float* gw,
                                  float* gb, float* dx, int B, int I, int O, float* ws, hipStream_t s);

// ------------------------------------------------------------------ k_gemm_f32.hip
// C[m][n] = epi(sum_k A(m, k) B(n, k)) in fp32, A(m, k) at A[m am + k ak], B(n, k)
// at B[n bn + k bk], C row m at C + m ldc; epi adds bias[n] and add[m ldadd + n],
// applies ReLU, and zeroes entries whose mask[m ldmask + n] is not positive
// (each optional).  S > 1 splits K into S slices whose sums go to part
// ([S][M][N], part_floats available; fewer slices if it is smaller) and are
// added in order by a second launch.  inA / inB / inAdd take that operand from
// the step's batch record instead.
struct GemmF32 {
    const float* A;
    int64_t am, ak;
    const float* B;
    int64_t bn, bk;
    float* C;
    int64_t ldc;
    int M, N, K, S;
    const float* bias;
    const float* add;
    int64_t ldadd;
    const float* mask;
    int64_t ldmask;
    int relu;
    float* part;
    const StepIn* inA;
    const StepIn* inB;
    const StepIn* inAdd;
    // S > 1: leave the slices in part for the caller to sum (no epilogue
    // operands then), instead of the second launch
    int defer;
    // with S == 1: let the launcher split K when the product has few output
    // tiles and a long K (its slices then summed by the second launch).  Used
    // by the VGG-5 and MobileNetV3 server parts (their classifier and SE
    // products run on 2 to 20 tiles over K up to 1280)
    int auto_split;
};
fo_status launch_gemm_f32(GemmF32 g, float* part, size_t part_floats, hipStream_t s);

}  // namespace fo
