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
#include <hip/hip_ext.h>

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
        h[e] = f2bf2(v[2 * e], v[2 * e + 1]);
        l[e] = f2bf2(v[2 * e] - bf2f((bf16_t)(h[e] & 0xFFFFu)), v[2 * e + 1] - bf2f((bf16_t)(h[e] >> 16)));
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

constexpr int PADJ = LMAX + 8;  // LDS row stride (bf16) of arrays indexed [.][key or query]
constexpr int PADK = DH + 8;    // LDS row stride (bf16) of row-major [token][head column] arrays

// Transposed orientation.  Both passes compute S^T = K Q^T: a wave owns 32
// queries, which sit on the accumulator columns, so every lane holds one
// query and 16 keys per 32x32 tile (key j = 32 jt + 8 (r div 4) + 4 (l div
// 32) + r mod 4 in register r).  Row statistics over keys then reduce within
// the lane plus one exchange between the half-waves, and a tile of P^T (or
// dS^T) already is the B operand of a product that sums over keys, provided
// the A operand takes its k index through the same permutation: for k block
// kb of tile jt, lane half h supplies keys 32 jt + 16 kb + {4h..4h+3} and
// 32 jt + 16 kb + 8 + {4h..4h+3} (registers 8 kb .. 8 kb + 7).

// Eight bf16 of an LDS row at key offsets {j, .., j+3, j+8, .., j+11}.
__device__ __forceinline__ bf16x8_t ld_perm(const bf16_t* row, int j) {
    const uint2 a = *reinterpret_cast<const uint2*>(row + j);
    const uint2 c = *reinterpret_cast<const uint2*>(row + j + 8);
    const u32x4_t v = {a.x, a.y, c.x, c.y};
    return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ uint2 pack4(bf16_t a, bf16_t b, bf16_t c, bf16_t e) {
    return make_uint2((uint32_t)a | ((uint32_t)b << 16), (uint32_t)c | ((uint32_t)e << 16));
}

// Forward.  Workgroup = (sequence, head), wave w owns queries 32w..32w+31.
// S^T = K Q^T and O^T = V^T P^T are compensated products (bf16 high/low parts
// of both operands, three MFMAs each), so the attention keeps about 16 bits
// of operand precision.  K (row-major) and V^T are staged in LDS once, with
// every global load of the workgroup issued before the first LDS store.
__global__ void __launch_bounds__(256, 2) attn_fwd_mfma(const float* __restrict__ qkv, const int* __restrict__ cu,
                                                        bf16_t* __restrict__ out, bf16_t* __restrict__ outlo,
                                                        float* __restrict__ lse, int H, int d, float scale,
                                                        int* __restrict__ snap, int nb) {
    __shared__ __attribute__((aligned(16))) bf16_t Ks[2][LMAX][PADK];  // K (high, low), zero past len
    __shared__ __attribute__((aligned(16))) bf16_t Vt[2][DH][PADJ];    // V^T (high, low), zero past len
    if (snap && blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nb; i += blockDim.x) snap[i] = cu[i];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int ld = 3 * d;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int lr = lane & 31, lh = lane >> 5;
    const int i0 = 32 * w, qi = i0 + lr;
    const bool active = i0 < len;
    float qv[4][8];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
        load8f(qkv + (int64_t)(base + qi) * ld + h * DH + 16 * kk + 8 * lh, qi < len, scale, qv[kk]);
    {
        // thread: head columns c4..c4+3 of tokens j = tid/16 + 16u
        const int c4 = (tid & 15) * 4;
        float4 kv[8], vv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = (tid >> 4) + 16 * u;
            const float* row = qkv + (int64_t)(base + j) * ld + d + h * DH + c4;
            kv[u] = vv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (j < len) {
                kv[u] = *reinterpret_cast<const float4*>(row);
                vv[u] = *reinterpret_cast<const float4*>(row + d);
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = (tid >> 4) + 16 * u;
            const float ke[4] = {kv[u].x, kv[u].y, kv[u].z, kv[u].w};
            const float ve[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
            bf16_t kh[4], kl[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                kh[q] = f2bf(ke[q]);
                kl[q] = f2bf(ke[q] - bf2f(kh[q]));
                const bf16_t vh = f2bf(ve[q]);
                Vt[0][c4 + q][j] = vh;
                Vt[1][c4 + q][j] = f2bf(ve[q] - bf2f(vh));
            }
            *reinterpret_cast<uint2*>(&Ks[0][j][c4]) = pack4(kh[0], kh[1], kh[2], kh[3]);
            *reinterpret_cast<uint2*>(&Ks[1][j][c4]) = pack4(kl[0], kl[1], kl[2], kl[3]);
        }
    }
    __syncthreads();
    if (!active) return;  // no barrier follows
    const int nj = (len + 31) >> 5;
    bf16x8_t qh[4], ql[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) split8(qv[kk], qh[kk], ql[kk]);
    f32x16 S[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) S[jt][r] = 0.f;
        if (jt < nj) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const bf16x8_t kh = *reinterpret_cast<const bf16x8_t*>(&Ks[0][32 * jt + lr][16 * kk + 8 * lh]);
                const bf16x8_t kl = *reinterpret_cast<const bf16x8_t*>(&Ks[1][32 * jt + lr][16 * kk + 8 * lh]);
                S[jt] = mfma3(kh, kl, qh[kk], ql[kk], S[jt]);
            }
        }
    }
    // softmax over the keys of this lane's query
    float m = -INFINITY;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int j = 32 * jt + 8 * (r >> 2) + 4 * lh + (r & 3);
            if (jt < nj && j < len) m = fmaxf(m, S[jt][r]);
        }
    m = fmaxf(m, __shfl_xor(m, 32));
    float sum = 0.f;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int j = 32 * jt + 8 * (r >> 2) + 4 * lh + (r & 3);
            const float p = (jt < nj && j < len) ? expf(S[jt][r] - m) : 0.f;
            S[jt][r] = p;
            sum += p;
        }
    sum += __shfl_xor(sum, 32);
    const float inv = 1.f / sum;
    // O^T = V^T P^T
    f32x16 O[2];
#pragma unroll
    for (int dt = 0; dt < 2; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) O[dt][r] = 0.f;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
        if (jt >= nj) break;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            float pv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) pv[e] = S[jt][8 * kb + e] * inv;
            bf16x8_t ph, pl;
            split8(pv, ph, pl);
            const int jb = 32 * jt + 16 * kb + 4 * lh;
#pragma unroll
            for (int dt = 0; dt < 2; ++dt) {
                const bf16x8_t vh = ld_perm(&Vt[0][32 * dt + lr][0], jb);
                const bf16x8_t vl = ld_perm(&Vt[1][32 * dt + lr][0], jb);
                O[dt] = mfma3(vh, vl, ph, pl, O[dt]);
            }
        }
    }
    if (qi < len) {
        // O^T accumulator: head column c = 32 dt + 8 q + 4 lh + (r mod 4), query qi
        const int64_t o = (int64_t)(base + qi) * d + h * DH;
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                bf16_t hi[4], lo[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float v = O[dt][4 * q + e];
                    hi[e] = f2bf(v);
                    lo[e] = f2bf(v - bf2f(hi[e]));
                }
                const int c = 32 * dt + 8 * q + 4 * lh;
                *reinterpret_cast<uint2*>(out + o + c) = pack4(hi[0], hi[1], hi[2], hi[3]);
                *reinterpret_cast<uint2*>(outlo + o + c) = pack4(lo[0], lo[1], lo[2], lo[3]);
            }
        if (lh == 0) lse[((int64_t)b * H + h) * LMAX + qi] = m + logf(sum);
    }
}

// Backward (plain bf16 products: the backward feeds gradients only).  With
// P = softmax(S), S = scale Q K^T and D_i = sum_c dO_ic O_ic:
//   dS_ij = P_ij (dO_i . V_j - D_i)
//   dQ_i = scale sum_j dS_ij K_j;  dK_j = scale sum_i dS_ij Q_i;  dV_j = sum_i P_ij dO_i
// Phase 1, wave w on queries 32w..: S^T = K (scale Q)^T and dP^T = V dO^T from
// row-major K, V in LDS; P^T = exp(S^T - lse) from the forward's log-sum-exp,
// dS^T; both go to LDS for phase 2, and dQ^T = K^T dS^T takes dS^T straight from
// the registers.  Phase 2, wave w on keys 32w..: dK = dS^T (scale Q) and
// dV = P^T dO.
__global__ void __launch_bounds__(256) attn_bwd_mfma(const float* __restrict__ qkv, const int* __restrict__ cu,
                                                     const bf16_t* __restrict__ out, const bf16_t* __restrict__ dout,
                                                     const float* __restrict__ lse, bf16_t* __restrict__ dqkv, int H,
                                                     int d, float scale, int* __restrict__ snap, int nb) {
    __shared__ __attribute__((aligned(16))) bf16_t Kr[LMAX][PADK];   // K
    __shared__ __attribute__((aligned(16))) bf16_t Vr[LMAX][PADK];   // V
    __shared__ __attribute__((aligned(16))) bf16_t Kt[DH][PADJ];     // K^T
    __shared__ __attribute__((aligned(16))) bf16_t Qt[DH][PADJ];     // (scale Q)^T
    __shared__ __attribute__((aligned(16))) bf16_t Gt[DH][PADJ];     // dO^T
    __shared__ __attribute__((aligned(16))) bf16_t Pt[LMAX][PADJ];   // P^T
    __shared__ __attribute__((aligned(16))) bf16_t Dst[LMAX][PADJ];  // dS^T
    if (snap && blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nb; i += blockDim.x) snap[i] = cu[i];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int ld = 3 * d;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int lr = lane & 31, lh = lane >> 5;
    const int i0 = 32 * w, qi = i0 + lr;
    const bool active = i0 < len;
    const int nj = (len + 31) >> 5;
    const int64_t rb = ((int64_t)b * H + h) * LMAX;
    // this lane's query: scale Q, dO and O at head columns 16 kk + 8 lh + 0..7
    float qv[4][8];
    u32x4_t gv[4], ov[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int c = h * DH + 16 * kk + 8 * lh;
        load8f(qkv + (int64_t)(base + qi) * ld + c, qi < len, scale, qv[kk]);
        gv[kk] = ov[kk] = u32x4_t{0u, 0u, 0u, 0u};
        if (qi < len) {
            gv[kk] = *reinterpret_cast<const u32x4_t*>(dout + (int64_t)(base + qi) * d + c);
            ov[kk] = *reinterpret_cast<const u32x4_t*>(out + (int64_t)(base + qi) * d + c);
        }
    }
    const float lq = qi < len ? lse[rb + qi] : 0.f;
    {
        const int c4 = (tid & 15) * 4;
        float4 qs[8], ks[8], vs[8];
        uint2 gs[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = (tid >> 4) + 16 * u;
            const bool ok = j < len;
            const float* row = qkv + (int64_t)(base + j) * ld + h * DH + c4;
            qs[u] = ks[u] = vs[u] = make_float4(0.f, 0.f, 0.f, 0.f);
            gs[u] = make_uint2(0, 0);
            if (ok) {
                qs[u] = *reinterpret_cast<const float4*>(row);
                ks[u] = *reinterpret_cast<const float4*>(row + d);
                vs[u] = *reinterpret_cast<const float4*>(row + 2 * d);
                gs[u] = *reinterpret_cast<const uint2*>(dout + (int64_t)(base + j) * d + h * DH + c4);
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = (tid >> 4) + 16 * u;
            const float qe[4] = {qs[u].x, qs[u].y, qs[u].z, qs[u].w};
            const float ke[4] = {ks[u].x, ks[u].y, ks[u].z, ks[u].w};
            const float ve[4] = {vs[u].x, vs[u].y, vs[u].z, vs[u].w};
            bf16_t kb[4], vb[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                kb[q] = f2bf(ke[q]);
                vb[q] = f2bf(ve[q]);
                Kt[c4 + q][j] = kb[q];
                Qt[c4 + q][j] = f2bf(qe[q] * scale);
            }
            Gt[c4 + 0][j] = (bf16_t)(gs[u].x & 0xFFFFu);
            Gt[c4 + 1][j] = (bf16_t)(gs[u].x >> 16);
            Gt[c4 + 2][j] = (bf16_t)(gs[u].y & 0xFFFFu);
            Gt[c4 + 3][j] = (bf16_t)(gs[u].y >> 16);
            *reinterpret_cast<uint2*>(&Kr[j][c4]) = pack4(kb[0], kb[1], kb[2], kb[3]);
            *reinterpret_cast<uint2*>(&Vr[j][c4]) = pack4(vb[0], vb[1], vb[2], vb[3]);
        }
    }
    __syncthreads();
    f32x16 dq[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) dq[t][r] = 0.f;
    if (active) {
        bf16x8_t qa[4], ga[4];
        float dsum = 0.f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            bf16x8_t lo;
            split8(qv[kk], qa[kk], lo);
            ga[kk] = __builtin_bit_cast(bf16x8_t, gv[kk]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t g2 = gv[kk][e], o2 = ov[kk][e];
                dsum = fmaf(bf2f((bf16_t)(g2 & 0xFFFFu)), bf2f((bf16_t)(o2 & 0xFFFFu)), dsum);
                dsum = fmaf(bf2f((bf16_t)(g2 >> 16)), bf2f((bf16_t)(o2 >> 16)), dsum);
            }
        }
        const float Dq = dsum + __shfl_xor(dsum, 32);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            if (jt >= nj) break;
            f32x16 S, G;
#pragma unroll
            for (int r = 0; r < 16; ++r) S[r] = G[r] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const bf16x8_t kb = *reinterpret_cast<const bf16x8_t*>(&Kr[32 * jt + lr][16 * kk + 8 * lh]);
                const bf16x8_t vb = *reinterpret_cast<const bf16x8_t*>(&Vr[32 * jt + lr][16 * kk + 8 * lh]);
                S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb, qa[kk], S, 0, 0, 0);
                G = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vb, ga[kk], G, 0, 0, 0);
            }
            float dsv[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = 32 * jt + 8 * (r >> 2) + 4 * lh + (r & 3);
                const bool ok = qi < len && j < len;
                const float p = ok ? expf(S[r] - lq) : 0.f;
                const float ds = ok ? p * (G[r] - Dq) : 0.f;
                dsv[r] = ds;
                Pt[j][qi] = f2bf(p);
                Dst[j][qi] = f2bf(ds);
            }
            // dQ^T += K^T dS^T over this tile's keys
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                u32x4_t sv;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    sv[e] = (uint32_t)f2bf(dsv[8 * kb + 2 * e]) | ((uint32_t)f2bf(dsv[8 * kb + 2 * e + 1]) << 16);
                const bf16x8_t bs = __builtin_bit_cast(bf16x8_t, sv);
                const int jb = 32 * jt + 16 * kb + 4 * lh;
#pragma unroll
                for (int t = 0; t < 2; ++t)
                    dq[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_perm(&Kt[32 * t + lr][0], jb), bs, dq[t], 0,
                                                                    0, 0);
            }
        }
    }
    __syncthreads();
    if (!active) return;  // no barrier follows
    if (qi < len) {
        // dQ^T accumulator: head column c = 32 t + 8 q + 4 lh + (r mod 4), query qi
        bf16_t* row = dqkv + (int64_t)(base + qi) * ld + h * DH;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                bf16_t o[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = f2bf(dq[t][4 * q + e] * scale);
                *reinterpret_cast<uint2*>(row + 32 * t + 8 * q + 4 * lh) = pack4(o[0], o[1], o[2], o[3]);
            }
    }
    f32x16 dk[2], dv[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) dk[t][r] = dv[t][r] = 0.f;
    const int j0 = 32 * w;
    for (int k16 = 0; k16 < 2 * nj; ++k16) {
        const int kc = 16 * k16 + 8 * lh;
        const bf16x8_t a_ds = *reinterpret_cast<const bf16x8_t*>(&Dst[j0 + lr][kc]);
        const bf16x8_t a_p = *reinterpret_cast<const bf16x8_t*>(&Pt[j0 + lr][kc]);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const bf16x8_t bq = *reinterpret_cast<const bf16x8_t*>(&Qt[32 * t + lr][kc]);
            const bf16x8_t bg = *reinterpret_cast<const bf16x8_t*>(&Gt[32 * t + lr][kc]);
            dk[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_ds, bq, dk[t], 0, 0, 0);
            dv[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_p, bg, dv[t], 0, 0, 0);
        }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int j = j0 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (j >= len) continue;
        bf16_t* row = dqkv + (int64_t)(base + j) * ld + h * DH;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int c = 32 * t + lr;
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
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("attn_fwd_mfma", pi, &ea, &eb);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipExtLaunchKernelGGL(attn_fwd_mfma, dim3(B * H), dim3(256), 0, s, ea, eb, 0, qkv, cu, out, outlo, lse, H, d,
                          1.f / sqrtf((float)DH), snap, B);
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_attn_bwd(const float* qkv, const int* cu, const bf16_t* out, const bf16_t* dout,
                          const float* lse, bf16_t* dqkv, int B, int H, int d, hipStream_t s) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    const float scale = 1.f / sqrtf((float)DH);
    ProfInfo pi;
    pi.kind = PROF_ATTN_BWD; pi.cu = cu; pi.B = B; pi.d = d;
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("attn_bwd_mfma", pi, &ea, &eb);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipExtLaunchKernelGGL(attn_bwd_mfma, dim3(B * H), dim3(256), 0, s, ea, eb, 0, qkv, cu, out, dout, lse, dqkv, H, d,
                          scale, snap, B);
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
