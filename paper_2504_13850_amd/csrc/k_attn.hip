// Masked multi-head self-attention over packed variable-length sequences,
// forward and backward, one workgroup per (sequence, head).
//
// Tokens of sequence b occupy rows cu[b] .. cu[b]+len_b-1 of the packed
// activations; keys at positions >= len_b do not exist in the packed layout,
// which is exactly the -inf key mask of the padded formulation.  The fused
// projection qkv is [T][3*d] with the query, key and value of head h in
// columns h*dh, d + h*dh and 2d + h*dh.
//
// Both passes run on the matrix cores (v_mfma_f32_32x32x16_bf16) with the
// whole (sequence, head) resident in LDS: sequences are at most 128 tokens.
#include "kernels.h"
#include "prof.h"

namespace fo {
namespace {

constexpr int DH = 64;      // head width
constexpr int LMAX = 128;   // longest sequence

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Eight fp32 values -> their bf16 (high, low) parts as MFMA operands.
__device__ __forceinline__ void split8(const float* v, bf16x8_t& hi, bf16x8_t& lo) {
    u32x4_t h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const bf16_t h0 = f2bf(v[2 * e]), h1 = f2bf(v[2 * e + 1]);
        const bf16_t l0 = f2bf(v[2 * e] - bf2f(h0)), l1 = f2bf(v[2 * e + 1] - bf2f(h1));
        h[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        l[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
    }
    hi = __builtin_bit_cast(bf16x8_t, h);
    lo = __builtin_bit_cast(bf16x8_t, l);
}

__device__ __forceinline__ void load8f(const float* p, bool ok, float scale, float* v) {
    if (ok) {
        const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
        v[0] = a.x * scale; v[1] = a.y * scale; v[2] = a.z * scale; v[3] = a.w * scale;
        v[4] = b.x * scale; v[5] = b.y * scale; v[6] = b.z * scale; v[7] = b.w * scale;
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
    }
}

__device__ __forceinline__ f32x16 mfma3(const bf16x8_t& ah, const bf16x8_t& al, const bf16x8_t& bh,
                                        const bf16x8_t& bl, f32x16 c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, c, 0, 0, 0);
}

__device__ __forceinline__ float half_max(float v) {  // over the 32 lanes of a half-wave
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ float half_sum(float v) {
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) v += __shfl_xor(v, o);
    return v;
}

constexpr int PADJ = LMAX + 8;  // LDS row stride (bf16) of the key dimension

// Forward on the matrix cores.  Workgroup = (sequence, head), wave w owns
// query rows 32w..32w+31.  S = Q K^T and O = P V are compensated products
// (bf16 high/low parts of both operands, three MFMAs each) so that the
// attention keeps about 16 bits of operand precision.  The v_mfma 32x32x16
// operand layouts: lane l supplies row (l mod 32) and k = 8*(l div 32) + 0..7
// of A, column (l mod 32) and the same k of B; the accumulator holds
// C[8*(r div 4) + 4*(l div 32) + (r mod 4)][l mod 32] in register r.
__global__ void __launch_bounds__(256) attn_fwd_mfma(const float* __restrict__ qkv, const int* __restrict__ cu,
                                                     bf16_t* __restrict__ out, bf16_t* __restrict__ outlo,
                                                     float* __restrict__ lse, int H, int d, float scale,
                                                     int* __restrict__ snap, int nb) {
    __shared__ __attribute__((aligned(16))) bf16_t Vt[2][DH][PADJ];      // V^T (high, low), zero past len
    __shared__ __attribute__((aligned(16))) bf16_t Ps[4][2][32][PADJ];   // per-wave P (high, low)
    if (snap && blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nb; i += blockDim.x) snap[i] = cu[i];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int ld = 3 * d;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    for (int idx = tid; idx < LMAX * DH; idx += blockDim.x) {
        const int j = idx / DH, c = idx % DH;
        const float v = j < len ? qkv[(int64_t)(base + j) * ld + 2 * d + h * DH + c] : 0.f;
        const bf16_t hi = f2bf(v);
        Vt[0][c][j] = hi;
        Vt[1][c][j] = f2bf(v - bf2f(hi));
    }
    __syncthreads();
    const int i0 = 32 * w;
    const bool active = i0 < len;
    const int nj = (len + 31) >> 5;
    const int lr = lane & 31, lh = lane >> 5;
    f32x16 S[4];
    float rmax[16], rsum[16];
    if (active) {
        bf16x8_t qh[4], ql[4];
        const int qi = i0 + lr;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            float v[8];
            load8f(qkv + (int64_t)(base + qi) * ld + h * DH + 16 * kk + 8 * lh, qi < len, scale, v);
            split8(v, qh[kk], ql[kk]);
        }
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) S[jt][r] = 0.f;
            if (jt < nj) {
                const int kj = 32 * jt + lr;
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    float v[8];
                    bf16x8_t kh, kl;
                    load8f(qkv + (int64_t)(base + kj) * ld + d + h * DH + 16 * kk + 8 * lh, kj < len, 1.f, v);
                    split8(v, kh, kl);
                    S[jt] = mfma3(qh[kk], ql[kk], kh, kl, S[jt]);
                }
            }
        }
        // masked softmax over keys, rows spread as in the accumulator layout
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float m = -INFINITY;
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
                if (jt < nj && 32 * jt + lr < len) m = fmaxf(m, S[jt][r]);
            m = half_max(m);
            float sum = 0.f;
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) {
                const float p = (jt < nj && 32 * jt + lr < len) ? expf(S[jt][r] - m) : 0.f;
                S[jt][r] = p;
                sum += p;
            }
            sum = half_sum(sum);
            rmax[r] = m;
            rsum[r] = sum;
            const float inv = 1.f / sum;
            const int il = 8 * (r >> 2) + 4 * lh + (r & 3);
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) {
                if (jt < nj) {
                    const float p = S[jt][r] * inv;
                    const bf16_t ph = f2bf(p);
                    Ps[w][0][il][32 * jt + lr] = ph;
                    Ps[w][1][il][32 * jt + lr] = f2bf(p - bf2f(ph));
                }
            }
        }
    }
    __syncthreads();
    if (!active) return;
    f32x16 O[2];
#pragma unroll
    for (int dt = 0; dt < 2; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) O[dt][r] = 0.f;
    for (int jk = 0; jk < 2 * nj; ++jk) {
        const int jc = 16 * jk + 8 * lh;
        const bf16x8_t ph = *reinterpret_cast<const bf16x8_t*>(&Ps[w][0][lr][jc]);
        const bf16x8_t pl = *reinterpret_cast<const bf16x8_t*>(&Ps[w][1][lr][jc]);
#pragma unroll
        for (int dt = 0; dt < 2; ++dt) {
            const bf16x8_t vh = *reinterpret_cast<const bf16x8_t*>(&Vt[0][32 * dt + lr][jc]);
            const bf16x8_t vl = *reinterpret_cast<const bf16x8_t*>(&Vt[1][32 * dt + lr][jc]);
            O[dt] = mfma3(ph, pl, vh, vl, O[dt]);
        }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int i = i0 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (i < len) {
#pragma unroll
            for (int dt = 0; dt < 2; ++dt) {
                const float v = O[dt][r];
                const bf16_t hi = f2bf(v);
                const int64_t o = (int64_t)(base + i) * d + h * DH + 32 * dt + lr;
                out[o] = hi;
                outlo[o] = f2bf(v - bf2f(hi));
            }
            if (lr == 0) lse[((int64_t)b * H + h) * LMAX + i] = rmax[r] + logf(rsum[r]);
        }
    }
}

// Backward.  With P = softmax(S), S = scale * Q K^T:
//   D_i = sum_c dO_ic O_ic;  dS_ij = P_ij (dO_i . V_j - D_i)
//   dQ_i = scale * sum_j dS_ij K_j;  dK_j = scale * sum_i dS_ij Q_i;  dV_j = sum_i P_ij dO_i
// D comes from its own small kernel (thread per query row); the probabilities
// are recomputed from the forward's log-sum-exp.
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

// Backward on the matrix cores (plain bf16 products: the backward feeds
// gradients only).  Workgroup = (sequence, head); wave w owns query rows and
// key rows 32w..32w+31.  Phase 1: each wave recomputes P = exp(S - lse) for
// its query rows, dP = dO V^T, and dS = P (dP - D), and leaves P^T, dS^T and dS
// in LDS.  Phase 2: dQ = scale dS K for its query rows, dK = dS^T (scale Q) and
// dV = P^T dO for its key rows, from LDS-staged K^T, (scale Q)^T and dO^T.
__global__ void __launch_bounds__(256) attn_bwd_mfma(const float* __restrict__ qkv, const int* __restrict__ cu,
                                                     const bf16_t* __restrict__ dout, const float* __restrict__ lse,
                                                     const float* __restrict__ Dv, bf16_t* __restrict__ dqkv, int H,
                                                     int d, float scale) {
    __shared__ __attribute__((aligned(16))) bf16_t Kt[DH][PADJ];
    __shared__ __attribute__((aligned(16))) bf16_t Qt[DH][PADJ];
    __shared__ __attribute__((aligned(16))) bf16_t Gt[DH][PADJ];
    __shared__ __attribute__((aligned(16))) bf16_t Pt[LMAX][PADJ];
    __shared__ __attribute__((aligned(16))) bf16_t Dst[LMAX][PADJ];
    __shared__ __attribute__((aligned(16))) bf16_t Dsr[LMAX][PADJ];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int ld = 3 * d;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int lr = lane & 31, lh = lane >> 5;
    for (int idx = tid; idx < LMAX * DH; idx += blockDim.x) {
        const int j = idx / DH, c = idx % DH;
        const bool ok = j < len;
        const float* row = qkv + (int64_t)(base + j) * ld + h * DH + c;
        Qt[c][j] = f2bf(ok ? row[0] * scale : 0.f);
        Kt[c][j] = f2bf(ok ? row[d] : 0.f);
        Gt[c][j] = ok ? dout[(int64_t)(base + j) * d + h * DH + c] : (bf16_t)0;
    }
    const int i0 = 32 * w;
    const bool active = i0 < len;
    const int nj = (len + 31) >> 5;
    const int64_t rb = ((int64_t)b * H + h) * LMAX;
    if (active) {
        bf16x8_t qa[4], ga[4];
        const int qi = i0 + lr;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            float v[8];
            bf16x8_t lo;
            load8f(qkv + (int64_t)(base + qi) * ld + h * DH + 16 * kk + 8 * lh, qi < len, scale, v);
            split8(v, qa[kk], lo);
            u32x4_t gv = {0u, 0u, 0u, 0u};
            if (qi < len)
                gv = *reinterpret_cast<const u32x4_t*>(dout + (int64_t)(base + qi) * d + h * DH + 16 * kk + 8 * lh);
            ga[kk] = __builtin_bit_cast(bf16x8_t, gv);
        }
        float Lr[16], Dr[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = i0 + 8 * (r >> 2) + 4 * lh + (r & 3);
            Lr[r] = i < len ? lse[rb + i] : 0.f;
            Dr[r] = i < len ? Dv[rb + i] : 0.f;
        }
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            if (jt >= nj) continue;
            f32x16 S, G;
#pragma unroll
            for (int r = 0; r < 16; ++r) S[r] = G[r] = 0.f;
            const int kj = 32 * jt + lr;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                float v[8];
                bf16x8_t kb, vb, lo;
                const float* krow = qkv + (int64_t)(base + kj) * ld + h * DH + 16 * kk + 8 * lh;
                load8f(krow + d, kj < len, 1.f, v);
                split8(v, kb, lo);
                load8f(krow + 2 * d, kj < len, 1.f, v);
                split8(v, vb, lo);
                S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[kk], kb, S, 0, 0, 0);
                G = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ga[kk], vb, G, 0, 0, 0);
            }
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                uint32_t pw[2], sw[2];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int r = 4 * rr + q;
                    const int i = i0 + 8 * rr + 4 * lh + q;
                    const bool ok = i < len && kj < len;
                    const float p = ok ? expf(S[r] - Lr[r]) : 0.f;
                    const float ds = ok ? p * (G[r] - Dr[r]) : 0.f;
                    const bf16_t pb = f2bf(p), sb = f2bf(ds);
                    Dsr[i][kj] = sb;
                    if (q & 1) {
                        pw[q >> 1] |= (uint32_t)pb << 16;
                        sw[q >> 1] |= (uint32_t)sb << 16;
                    } else {
                        pw[q >> 1] = pb;
                        sw[q >> 1] = sb;
                    }
                }
                const int ib = i0 + 8 * rr + 4 * lh;
                *reinterpret_cast<uint2*>(&Pt[kj][ib]) = make_uint2(pw[0], pw[1]);
                *reinterpret_cast<uint2*>(&Dst[kj][ib]) = make_uint2(sw[0], sw[1]);
            }
        }
    }
    __syncthreads();
    if (!active) return;
    f32x16 dq[2], dk[2], dv[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) dq[t][r] = dk[t][r] = dv[t][r] = 0.f;
    for (int k16 = 0; k16 < 2 * nj; ++k16) {
        const int kc = 16 * k16 + 8 * lh;
        const bf16x8_t a_ds = *reinterpret_cast<const bf16x8_t*>(&Dsr[i0 + lr][kc]);  // dS rows (query block)
        const bf16x8_t a_dst = *reinterpret_cast<const bf16x8_t*>(&Dst[i0 + lr][kc]); // dS^T rows (key block)
        const bf16x8_t a_pt = *reinterpret_cast<const bf16x8_t*>(&Pt[i0 + lr][kc]);   // P^T rows (key block)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const bf16x8_t bk = *reinterpret_cast<const bf16x8_t*>(&Kt[32 * t + lr][kc]);
            const bf16x8_t bq = *reinterpret_cast<const bf16x8_t*>(&Qt[32 * t + lr][kc]);
            const bf16x8_t bg = *reinterpret_cast<const bf16x8_t*>(&Gt[32 * t + lr][kc]);
            dq[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_ds, bk, dq[t], 0, 0, 0);
            dk[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_dst, bq, dk[t], 0, 0, 0);
            dv[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_pt, bg, dv[t], 0, 0, 0);
        }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int i = i0 + 8 * (r >> 2) + 4 * lh + (r & 3);  // query row for dq, key row for dk / dv
        if (i >= len) continue;
        bf16_t* row = dqkv + (int64_t)(base + i) * ld + h * DH;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int c = 32 * t + lr;
            row[c] = f2bf(dq[t][r] * scale);
            row[d + c] = f2bf(dk[t][r]);
            row[2 * d + c] = f2bf(dv[t][r]);
        }
    }
}

}  // namespace

fo_status launch_attn_fwd(const float* qkv, const int* cu, bf16_t* out, bf16_t* outlo, float* lse, int B, int H,
                          int d, hipStream_t s) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    ProfInfo pi;
    pi.kind = PROF_ATTN_FWD; pi.cu = cu; pi.B = B; pi.d = d;
    const int h = prof_begin(s, "attn_fwd_mfma", pi);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipLaunchKernelGGL(attn_fwd_mfma, dim3(B * H), dim3(256), 0, s, qkv, cu, out, outlo, lse, H, d,
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
    const int h = prof_begin(s, "attn_bwd (rowdot + mfma)", pi);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipLaunchKernelGGL(attn_bwd_rowdot, dim3(B * H), dim3(LMAX), 0, s, cu, out, dout, Dws, H, d, snap, B);
    hipLaunchKernelGGL(attn_bwd_mfma, dim3(B * H), dim3(256), 0, s, qkv, cu, dout, lse, Dws, dqkv, H, d, scale);
    prof_end(h, s);
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
