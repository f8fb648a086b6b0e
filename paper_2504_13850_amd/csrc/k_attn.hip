// Masked multi-head self-attention over packed variable-length sequences,
// forward and backward, one workgroup per (sequence, head).
//
// Tokens of sequence b occupy rows cu[b] .. cu[b]+len_b-1 of the packed
// activations; keys at positions >= len_b do not exist in the packed layout,
// which is exactly the -inf key mask of the padded formulation.  The fused
// projection qkv is [T][3*d] with the query, key and value of head h in
// columns h*dh, d + h*dh and 2d + h*dh.
//
// This version keeps two [len][64] fp32 operands of one (sequence, head) in
// LDS and gives each query (or key) row its own thread; softmax uses the
// running-maximum form and the backward pass recomputes the probabilities
// from the saved log-sum-exp.
#include "kernels.h"
#include "prof.h"

namespace fo {
namespace {

constexpr int DH = 64;      // head width
constexpr int LMAX = 128;   // longest sequence

__global__ void __launch_bounds__(LMAX) attn_fwd_kernel(const float* __restrict__ qkv, const int* __restrict__ cu,
                                                        bf16_t* __restrict__ out, bf16_t* __restrict__ outlo,
                                                        float* __restrict__ lse, int H, int d, float scale,
                                                        int* __restrict__ snap, int nb) {
    if (snap && blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nb; i += blockDim.x) snap[i] = cu[i];
    __shared__ float Ks[LMAX][DH];
    __shared__ float Vs[LMAX][DH];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int ld = 3 * d;
    for (int idx = threadIdx.x; idx < len * DH; idx += blockDim.x) {
        int j = idx / DH, c = idx % DH;
        const float* row = qkv + (int64_t)(base + j) * ld;
        Ks[j][c] = (row[d + h * DH + c]);
        Vs[j][c] = (row[2 * d + h * DH + c]);
    }
    __syncthreads();
    const int i = threadIdx.x;
    if (i >= len) return;
    float q[DH], o[DH];
    const float* qrow = qkv + (int64_t)(base + i) * ld + h * DH;
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        q[c] = (qrow[c]) * scale;
        o[c] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    for (int j = 0; j < len; ++j) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < DH; ++c) s = fmaf(q[c], Ks[j][c], s);
        float mn = fmaxf(m, s);
        float corr = expf(m - mn), p = expf(s - mn);
        l = l * corr + p;
#pragma unroll
        for (int c = 0; c < DH; ++c) o[c] = fmaf(p, Vs[j][c], o[c] * corr);
        m = mn;
    }
    float inv = 1.f / l;
    bf16_t* orow = out + (int64_t)(base + i) * d + h * DH;
    bf16_t* lrow = outlo + (int64_t)(base + i) * d + h * DH;
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        const float v = o[c] * inv;
        const bf16_t hi = f2bf(v);
        orow[c] = hi;
        lrow[c] = f2bf(v - bf2f(hi));
    }
    lse[((int64_t)b * H + h) * LMAX + i] = m + logf(l);
}

// Backward.  With P = softmax(S), S = scale * Q K^T:
//   D_i = sum_c dO_ic O_ic;  dS_ij = P_ij (dO_i . V_j - D_i)
//   dQ_i = scale * sum_j dS_ij K_j;  dK_j = scale * sum_i dS_ij Q_i;  dV_j = sum_i P_ij dO_i
// Three kernels: D per query row, dQ (thread per query, K and V in LDS) and
// dK/dV (thread per key, Q and dO in LDS); probabilities are recomputed from
// the saved log-sum-exp.  Every LDS row is read by all threads at once
// (broadcast), so rows are unpadded.
__global__ void __launch_bounds__(LMAX) attn_bwd_rowdot(const int* __restrict__ cu, const bf16_t* __restrict__ out,
                                                        const bf16_t* __restrict__ dout, float* __restrict__ D,
                                                        int H, int d, int* __restrict__ snap, int nb) {
    if (snap && blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nb; i += blockDim.x) snap[i] = cu[i];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int i = threadIdx.x;
    if (i >= len) return;
    const bf16_t* orow = out + (int64_t)(base + i) * d + h * DH;
    const bf16_t* drow = dout + (int64_t)(base + i) * d + h * DH;
    float acc = 0.f;
    for (int c = 0; c < DH; ++c) acc = fmaf(bf2f(drow[c]), bf2f(orow[c]), acc);
    D[((int64_t)b * H + h) * LMAX + i] = acc;
}

__global__ void __launch_bounds__(LMAX) attn_bwd_dq(const float* __restrict__ qkv, const int* __restrict__ cu,
                                                    const bf16_t* __restrict__ dout, const float* __restrict__ lse,
                                                    const float* __restrict__ D, bf16_t* __restrict__ dqkv, int H,
                                                    int d, float scale) {
    __shared__ float Ks[LMAX][DH];
    __shared__ float Vs[LMAX][DH];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int ld = 3 * d;
    for (int idx = threadIdx.x; idx < len * DH; idx += blockDim.x) {
        int j = idx / DH, c = idx % DH;
        const float* row = qkv + (int64_t)(base + j) * ld;
        Ks[j][c] = (row[d + h * DH + c]);
        Vs[j][c] = (row[2 * d + h * DH + c]);
    }
    __syncthreads();
    const int i = threadIdx.x;
    if (i >= len) return;
    float q[DH], g[DH], dq[DH];
    const float* qrow = qkv + (int64_t)(base + i) * ld + h * DH;
    const bf16_t* grow = dout + (int64_t)(base + i) * d + h * DH;
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        q[c] = (qrow[c]) * scale;
        g[c] = bf2f(grow[c]);
        dq[c] = 0.f;
    }
    const int64_t r = ((int64_t)b * H + h) * LMAX + i;
    const float Di = D[r], Li = lse[r];
    for (int j = 0; j < len; ++j) {
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int c = 0; c < DH; ++c) {
            s = fmaf(q[c], Ks[j][c], s);
            dp = fmaf(g[c], Vs[j][c], dp);
        }
        float ds = expf(s - Li) * (dp - Di);
#pragma unroll
        for (int c = 0; c < DH; ++c) dq[c] = fmaf(ds, Ks[j][c], dq[c]);
    }
    bf16_t* row = dqkv + (int64_t)(base + i) * ld + h * DH;
#pragma unroll
    for (int c = 0; c < DH; ++c) row[c] = f2bf(dq[c] * scale);
}

__global__ void __launch_bounds__(LMAX) attn_bwd_dkdv(const float* __restrict__ qkv, const int* __restrict__ cu,
                                                      const bf16_t* __restrict__ dout, const float* __restrict__ lse,
                                                      const float* __restrict__ D, bf16_t* __restrict__ dqkv, int H,
                                                      int d, float scale) {
    __shared__ float Qs[LMAX][DH];
    __shared__ float Gs[LMAX][DH];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int ld = 3 * d;
    for (int idx = threadIdx.x; idx < len * DH; idx += blockDim.x) {
        int i = idx / DH, c = idx % DH;
        Qs[i][c] = qkv[(int64_t)(base + i) * ld + h * DH + c] * scale;
        Gs[i][c] = bf2f(dout[(int64_t)(base + i) * d + h * DH + c]);
    }
    __syncthreads();
    const int j = threadIdx.x;
    if (j >= len) return;
    float k[DH], v[DH], dk[DH], dv[DH];
    const float* row = qkv + (int64_t)(base + j) * ld;
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        k[c] = (row[d + h * DH + c]);
        v[c] = (row[2 * d + h * DH + c]);
        dk[c] = dv[c] = 0.f;
    }
    const int64_t r0 = ((int64_t)b * H + h) * LMAX;
    for (int i = 0; i < len; ++i) {
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int c = 0; c < DH; ++c) {
            s = fmaf(Qs[i][c], k[c], s);
            dp = fmaf(Gs[i][c], v[c], dp);
        }
        float p = expf(s - lse[r0 + i]);
        float ds = p * (dp - D[r0 + i]);
#pragma unroll
        for (int c = 0; c < DH; ++c) {
            dv[c] = fmaf(p, Gs[i][c], dv[c]);
            dk[c] = fmaf(ds, Qs[i][c], dk[c]);  // Qs already carries the scale
        }
    }
    bf16_t* out = dqkv + (int64_t)(base + j) * ld;
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        out[d + h * DH + c] = f2bf(dk[c]);
        out[2 * d + h * DH + c] = f2bf(dv[c]);
    }
}

}  // namespace

fo_status launch_attn_fwd(const float* qkv, const int* cu, bf16_t* out, bf16_t* outlo, float* lse, int B, int H,
                          int d, hipStream_t s) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    ProfInfo pi;
    pi.kind = PROF_ATTN_FWD; pi.cu = cu; pi.B = B; pi.d = d;
    const int h = prof_begin(s, "attn_fwd_kernel", pi);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipLaunchKernelGGL(attn_fwd_kernel, dim3(B * H), dim3(LMAX), 0, s, qkv, cu, out, outlo, lse, H, d,
                       1.f / sqrtf((float)DH), snap, B);
    prof_end(h, s);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_attn_bwd(const float* qkv, const int* cu, const bf16_t* out, const bf16_t* dout,
                          const float* lse, float* Dws, bf16_t* dqkv, int B, int H, int d, hipStream_t s) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    const float scale = 1.f / sqrtf((float)DH);
    ProfInfo pi;
    pi.kind = PROF_ATTN_BWD; pi.cu = cu; pi.B = B; pi.d = d;
    const int h = prof_begin(s, "attn_bwd (3 kernels)", pi);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipLaunchKernelGGL(attn_bwd_rowdot, dim3(B * H), dim3(LMAX), 0, s, cu, out, dout, Dws, H, d, snap, B);
    hipLaunchKernelGGL(attn_bwd_dq, dim3(B * H), dim3(LMAX), 0, s, qkv, cu, dout, lse, Dws, dqkv, H, d, scale);
    hipLaunchKernelGGL(attn_bwd_dkdv, dim3(B * H), dim3(LMAX), 0, s, qkv, cu, dout, lse, Dws, dqkv, H, d, scale);
    prof_end(h, s);
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
