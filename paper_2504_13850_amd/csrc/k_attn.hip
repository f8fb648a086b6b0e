// Masked multi-head self-attention over packed variable-length sequences,
// forward and backward, one workgroup per (sequence, head).
//
// Tokens of sequence b occupy rows cu[b] .. cu[b]+len_b-1 of the packed
// activations; keys at positions >= len_b do not exist in the packed layout,
// which is exactly the -inf key mask of the padded formulation.  The fused
// projection qkv is [T][3*d] (bf16 high parts; qkvlo the low parts) with the
// query, key and value of head h in columns h*dh, d + h*dh and 2d + h*dh.
//
// Both passes run on the matrix cores (v_mfma_f32_32x32x16_bf16) with the
// whole (sequence, head) resident in LDS: sequences are at most 128 tokens.
// q, k and v come in as bf16 (high, low) pairs written by the projection.
#include <hip/hip_ext.h>

#include "kernels.h"
#include "prof.h"

namespace fo {
namespace {

constexpr int DH = 64;      // head width
constexpr int LMAX = 128;   // longest sequence
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

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

__device__ __forceinline__ f32x16 mfma(const bf16x8_t& a, const bf16x8_t& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma3(const bf16x8_t& ah, const bf16x8_t& al, const bf16x8_t& bh,
                                        const bf16x8_t& bl, f32x16 c) {
    c = mfma(ah, bh, c);
    c = mfma(ah, bl, c);
    return mfma(al, bh, c);
}

__device__ __forceinline__ uint2 pack4f(float a, float b, float c, float e) {
    return make_uint2(f2bf2(a, b), f2bf2(c, e));
}

// LDS tiles, unpadded, with their 16-byte chunks XOR-swizzled per row:
//  - [row][64] (128-byte rows): chunk c of row r at c xor g8(r), g8 mapping
//    m = (r / 2) mod 8 to 4 (m mod 2) + m / 2.  The 16 rows of a 128-bit operand
//    read (one chunk each) land in 16 distinct chunk slots of a 256-byte bank
//    row, and the four consecutive rows of half a wave's transpose read land in
//    four distinct 64-byte bank groups (rows 4a, 4a+1 and 4a+2, 4a+3 differ in
//    the top bit of g8).
//  - [row][128] (256-byte rows): chunk c of row r at c xor (4 (r mod 4) + (r / 4)
//    mod 4): four consecutive rows of a transpose read fall in distinct 64-byte
//    groups, and the 8-byte stores of 32 consecutive rows (one chunk each) fill
//    16 chunk slots twice.
__device__ __forceinline__ int idx64(int row, int col) {
    const int m = (row >> 1) & 7;
    return row * 64 + ((((col >> 3) ^ (((m & 1) << 2) | (m >> 1))) << 3) | (col & 7));
}
__device__ __forceinline__ int idx128(int row, int col) {
    return row * 128 + ((((col >> 3) ^ (((row & 3) << 2) | ((row >> 2) & 3))) << 3) | (col & 7));
}

// An MFMA operand fragment (lane l: operand row l % 32, eight k values) from a
// tile whose rows are k and whose columns are the operand rows, through two
// LDS transpose reads (ds_read_b64_tr_b16: within each group of 16 lanes, lane
// i receives element i mod 4 of the 8 bytes addressed by lane 4 j + i / 4, for
// j = 0..3).  Lane (g = l / 16, s = l % 16) addresses tile row kr(g) + s / 4 at
// columns col0 + 16 (g mod 2) + 4 (s mod 4); kr is 8 h + 4 r for the plain k
// order (k = 8 h + e, h = l / 32) and 4 h + 8 r for the attention key order
// (keys 4h..4h+3 and 8+4h..8+4h+3 of a 16-key block), r = 0, 1 the two reads.
template <bool WIDE>
__device__ __forceinline__ bf16x8_t frag_tr(const bf16_t* T, int row0, int col0, bool keyorder, int lane) {
    const int g = lane >> 4, s = lane & 15, h = lane >> 5;
    const int col = col0 + 16 * (g & 1) + 4 * (s & 3);
    s16x4_t v[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const int row = row0 + (keyorder ? 4 * h + 8 * r : 8 * h + 4 * r) + (s >> 2);
        const int i = WIDE ? idx128(row, col) : idx64(row, col);
        v[r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(T + i));
    }
    const s16x8_t o = {v[0][0], v[0][1], v[0][2], v[0][3], v[1][0], v[1][1], v[1][2], v[1][3]};
    return __builtin_bit_cast(bf16x8_t, o);
}
// A fragment whose lane rows are tile rows row0 + l % 32 (k = 8 (l / 32) + e along a row).
__device__ __forceinline__ bf16x8_t frag_row(const bf16_t* T, int row0, int col0, int lane) {
    return *reinterpret_cast<const bf16x8_t*>(&T[idx64(row0 + (lane & 31), col0 + 8 * (lane >> 5))]);
}

// Rows 0..127 of a head's 64 columns from a packed [T][ld] bf16 matrix into a
// [row][64] tile (zeros past len): 16-byte loads, all issued before the stores.
__device__ __forceinline__ void stage64(bf16_t* T, const bf16_t* src, int64_t ld, int base, int len, int tid) {
    const int c = (tid & 7) * 8;
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int row = (tid >> 3) + 32 * u;
        v[u] = row < len ? *reinterpret_cast<const uint4*>(src + (int64_t)(base + row) * ld + c) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) *reinterpret_cast<uint4*>(&T[idx64((tid >> 3) + 32 * u, c)]) = v[u];
}

__device__ __forceinline__ bf16x8_t ld8(const bf16_t* p, bool ok) {
    return ok ? *reinterpret_cast<const bf16x8_t*>(p) : __builtin_bit_cast(bf16x8_t, u32x4_t{0u, 0u, 0u, 0u});
}

// Transposed orientation.  Both passes compute S^T = K Q^T: a wave owns 32
// queries, which sit on the accumulator columns, so every lane holds one
// query and 16 keys per 32x32 tile (key j = 32 jt + 8 (r div 4) + 4 (l div
// 32) + r mod 4 in register r).  Row statistics over keys then reduce within
// the lane plus one exchange between the half-waves, and a tile of P^T (or
// dS^T) already is the B operand of a product that sums over keys, provided
// the A operand takes its k index in the same key order (see frag_tr).

// Forward.  Workgroup = (sequence, head), wave w owns queries 32w..32w+31.
// q, k, v arrive as bf16 (high, low) pairs from the projection's epilogue.
// S^T = K Q^T and O^T = V^T P^T are compensated products (three MFMAs each),
// so the attention keeps about 16 bits of operand precision.  The softmax
// runs in base 2 with the scale and log2(e) folded into one multiply.
__global__ void __launch_bounds__(256, 2) attn_fwd_mfma(const bf16_t* __restrict__ qkv, const bf16_t* __restrict__ qkvlo,
                                                        const int* __restrict__ cu, bf16_t* __restrict__ out,
                                                        bf16_t* __restrict__ outlo, float* __restrict__ lse, int H,
                                                        int d, float scale, int* __restrict__ snap, int nb,
                                                        const int* __restrict__ order) {
    __shared__ __attribute__((aligned(16))) bf16_t Kh[LMAX * DH], Kl[LMAX * DH], Vh[LMAX * DH], Vl[LMAX * DH];
    if (snap && blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nb; i += blockDim.x) snap[i] = cu[i];
    const int b = order ? order[blockIdx.x / H] : blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int64_t ld = 3 * d;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int lr = lane & 31, lh = lane >> 5;
    const int i0 = 32 * w, qi = i0 + lr;
    // this lane's query, head columns 16 kk + 8 lh .. + 7 (high and low parts)
    bf16x8_t qh[4], ql[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int64_t o = (int64_t)(base + qi) * ld + h * DH + 16 * kk + 8 * lh;
        qh[kk] = ld8(qkv + o, qi < len);
        ql[kk] = ld8(qkvlo + o, qi < len);
    }
    stage64(Kh, qkv + d + h * DH, ld, base, len, tid);
    stage64(Kl, qkvlo + d + h * DH, ld, base, len, tid);
    stage64(Vh, qkv + 2 * d + h * DH, ld, base, len, tid);
    stage64(Vl, qkvlo + 2 * d + h * DH, ld, base, len, tid);
    __syncthreads();
    if (i0 >= len) return;  // no barrier follows
    const int nj = (len + 31) >> 5;
    f32x16 S[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) S[jt][r] = 0.f;
        if (jt < nj) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                S[jt] = mfma3(frag_row(Kh, 32 * jt, 16 * kk, lane), frag_row(Kl, 32 * jt, 16 * kk, lane), qh[kk],
                              ql[kk], S[jt]);
        }
    }
    // softmax over the keys of this lane's query, base 2: x = S scale log2(e)
    const float c2 = scale * kLog2e;
    float m = -INFINITY;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int j = 32 * jt + 8 * (r >> 2) + 4 * lh + (r & 3);
            S[jt][r] = j < len ? S[jt][r] * c2 : -INFINITY;
            m = fmaxf(m, S[jt][r]);
        }
    m = fmaxf(m, __shfl_xor(m, 32));
    float sum = 0.f;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float p = __builtin_amdgcn_exp2f(S[jt][r] - m);  // masked keys: exp2(-inf) = 0
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
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
                O[dt] = mfma3(frag_tr<false>(Vh, 32 * jt + 16 * kb, 32 * dt, true, lane),
                              frag_tr<false>(Vl, 32 * jt + 16 * kb, 32 * dt, true, lane), ph, pl, O[dt]);
        }
    }
    if (qi < len) {
        // O^T accumulator: head column c = 32 dt + 8 q + 4 lh + (r mod 4), query qi
        const int64_t o = (int64_t)(base + qi) * d + h * DH;
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                f32x4 v = {O[dt][4 * q], O[dt][4 * q + 1], O[dt][4 * q + 2], O[dt][4 * q + 3]};
                const uint2 hi = pack4f(v[0], v[1], v[2], v[3]);
                const f32x4 lo = v - f32x4{bf2f((bf16_t)(hi.x & 0xFFFFu)), bf2f((bf16_t)(hi.x >> 16)),
                                           bf2f((bf16_t)(hi.y & 0xFFFFu)), bf2f((bf16_t)(hi.y >> 16))};
                const int c = 32 * dt + 8 * q + 4 * lh;
                *reinterpret_cast<uint2*>(out + o + c) = hi;
                *reinterpret_cast<uint2*>(outlo + o + c) = pack4f(lo[0], lo[1], lo[2], lo[3]);
            }
        if (lh == 0) lse[((int64_t)b * H + h) * LMAX + qi] = (m + __log2f(sum)) * kLn2;
    }
}

// Backward (plain bf16 products of the high parts: the backward feeds
// gradients only).  With P = softmax(S), S = scale Q K^T and D_i = sum_c dO_ic O_ic:
//   dS_ij = P_ij (dO_i . V_j - D_i)
//   dQ_i = scale sum_j dS_ij K_j;  dK_j = scale sum_i dS_ij Q_i;  dV_j = sum_i P_ij dO_i
// Two workgroups per (sequence, head), each recomputing P (from the forward's
// log-sum-exp) and dS for the rows it owns:
//  - the query workgroup, wave w on queries 32w..: K and V in LDS, the lane's
//    Q and dO row in registers; S^T = K Q^T and dP^T = V dO^T, then
//    dQ^T = K^T dS^T with dS^T straight from the registers;
//  - the key workgroup, wave w on keys 32w..: Q and dO in LDS with each
//    query's lse and D, the lane's K and V row in registers; per tile of 32
//    queries S = Q K^T and dP = dO V^T, then dK^T += Q^T dS and dV^T += dO^T P,
//    dS and P again straight from the registers (the query index of a tile
//    taken in the attention key order on both operands).
// Neither stores P or dS: a workgroup holds 33 KB of LDS, so all 2 B H of them
// are resident at once.
// D_i of the lane's row: dO and O over head columns 16 kk + 8 half + 0..7, the
// two halves summed by the caller (one exchange), in the same order on both
// workgroups so that they agree bit for bit.
__device__ __forceinline__ float dsum_half(const bf16_t* dout, const bf16_t* out, int64_t o, bool ok) {
    float acc = 0.f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const u32x4_t g = __builtin_bit_cast(u32x4_t, ld8(dout + o + 16 * kk, ok));
        const u32x4_t v = __builtin_bit_cast(u32x4_t, ld8(out + o + 16 * kk, ok));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc = fmaf(bf2f((bf16_t)(g[e] & 0xFFFFu)), bf2f((bf16_t)(v[e] & 0xFFFFu)), acc);
            acc = fmaf(bf2f((bf16_t)(g[e] >> 16)), bf2f((bf16_t)(v[e] >> 16)), acc);
        }
    }
    return acc;
}
__device__ __forceinline__ bf16x8_t pack8(const float* v) {
    u32x4_t u;
#pragma unroll
    for (int e = 0; e < 4; ++e) u[e] = f2bf2(v[2 * e], v[2 * e + 1]);
    return __builtin_bit_cast(bf16x8_t, u);
}
// A [64][32] transposed accumulator pair (rows = head columns 32 t + 8 q + 4 lh
// + r mod 4, column = the lane's row) times s, as bf16, into a token row.
__device__ __forceinline__ void store_rowT(bf16_t* row, const f32x16* acc, float s, int lh) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<uint2*>(row + 32 * t + 8 * q + 4 * lh) =
                pack4f(acc[t][4 * q] * s, acc[t][4 * q + 1] * s, acc[t][4 * q + 2] * s, acc[t][4 * q + 3] * s);
}

__global__ void __launch_bounds__(256, 2) attn_bwd_mfma(const bf16_t* __restrict__ qkv, const int* __restrict__ cu,
                                                        const bf16_t* __restrict__ out, const bf16_t* __restrict__ dout,
                                                        const float* __restrict__ lse, bf16_t* __restrict__ dqkv, int H,
                                                        int d, float scale, int* __restrict__ snap, int nb,
                                                        const int* __restrict__ order) {
    __builtin_amdgcn_s_setprio(2);  // on the input-gradient chain: its waves win issue arbitration
    __shared__ __attribute__((aligned(16))) bf16_t T0[LMAX * DH], T1[LMAX * DH];
    __shared__ __attribute__((aligned(16))) float rowL[LMAX], rowD[LMAX];
    if (snap && blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nb; i += blockDim.x) snap[i] = cu[i];
    const int pair = blockIdx.x >> 1;
    const bool keys = blockIdx.x & 1;
    const int b = order ? order[pair / H] : pair / H, h = pair % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int64_t ld = 3 * d;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int lr = lane & 31, lh = lane >> 5;
    const int r0 = 32 * w, ri = r0 + lr;  // the lane's query (query workgroup) or key (key workgroup)
    const int n32 = (len + 31) >> 5;
    const int64_t rb = ((int64_t)b * H + h) * LMAX;
    const float c2 = scale * kLog2e;
    const int hc = h * DH + 8 * lh;  // first head column of the lane's operand rows
    f32x16 acc0[2], acc1[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc0[t][r] = acc1[t][r] = 0.f;
    if (!keys) {
        bf16x8_t qa[4], ga[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            qa[kk] = ld8(qkv + (int64_t)(base + ri) * ld + hc + 16 * kk, ri < len);
            ga[kk] = ld8(dout + (int64_t)(base + ri) * d + hc + 16 * kk, ri < len);
        }
        const float lq = ri < len ? lse[rb + ri] * kLog2e : 0.f;
        float Dv = dsum_half(dout, out, (int64_t)(base + ri) * d + hc, ri < len);
        stage64(T0, qkv + d + h * DH, ld, base, len, tid);
        stage64(T1, qkv + 2 * d + h * DH, ld, base, len, tid);
        __syncthreads();
        if (r0 >= len) return;  // no barrier follows
        Dv += __shfl_xor(Dv, 32);
        for (int jt = 0; jt < n32; ++jt) {
            f32x16 S, G;
#pragma unroll
            for (int r = 0; r < 16; ++r) S[r] = G[r] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                S = mfma(frag_row(T0, 32 * jt, 16 * kk, lane), qa[kk], S);
                G = mfma(frag_row(T1, 32 * jt, 16 * kk, lane), ga[kk], G);
            }
            float dsv[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = 32 * jt + 8 * (r >> 2) + 4 * lh + (r & 3);
                const float p = ri < len && j < len ? __builtin_amdgcn_exp2f(fmaf(S[r], c2, -lq)) : 0.f;
                dsv[r] = p * (G[r] - Dv);
            }
            // dQ^T += K^T dS^T over this tile's keys (dS^T in the attention key order)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const bf16x8_t bs = pack8(dsv + 8 * kb);
#pragma unroll
                for (int t = 0; t < 2; ++t)
                    acc0[t] = mfma(frag_tr<false>(T0, 32 * jt + 16 * kb, 32 * t, true, lane), bs, acc0[t]);
            }
        }
        if (ri < len) store_rowT(dqkv + (int64_t)(base + ri) * ld + h * DH, acc0, scale, lh);
        return;
    }
    // key workgroup: per-query base-2 lse and D, then Q and dO tiles
    {
        const int i = tid >> 1, half = tid & 1;
        float Dv = dsum_half(dout, out, (int64_t)(base + i) * d + h * DH + 8 * half, i < len);
        Dv += __shfl_xor(Dv, 1);
        if (!half) {
            rowL[i] = i < len ? lse[rb + i] * kLog2e : 0.f;
            rowD[i] = Dv;
        }
    }
    bf16x8_t ka[4], va[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        ka[kk] = ld8(qkv + (int64_t)(base + ri) * ld + d + hc + 16 * kk, ri < len);
        va[kk] = ld8(qkv + (int64_t)(base + ri) * ld + 2 * d + hc + 16 * kk, ri < len);
    }
    stage64(T0, qkv + h * DH, ld, base, len, tid);
    stage64(T1, dout + h * DH, d, base, len, tid);
    __syncthreads();
    if (r0 >= len) return;  // no barrier follows
    for (int it = 0; it < n32; ++it) {
        f32x16 S, G;
#pragma unroll
        for (int r = 0; r < 16; ++r) S[r] = G[r] = 0.f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            S = mfma(frag_row(T0, 32 * it, 16 * kk, lane), ka[kk], S);
            G = mfma(frag_row(T1, 32 * it, 16 * kk, lane), va[kk], G);
        }
        // S, G: the lane's key ri, queries i = 32 it + 8 q + 4 lh + (r mod 4)
        float pv[16], dsv[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i0 = 32 * it + 8 * q + 4 * lh;
            const f32x4 L4 = *reinterpret_cast<const f32x4*>(&rowL[i0]);
            const f32x4 D4 = *reinterpret_cast<const f32x4*>(&rowD[i0]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 4 * q + e;
                const float p = ri < len && i0 + e < len ? __builtin_amdgcn_exp2f(fmaf(S[r], c2, -L4[e])) : 0.f;
                pv[r] = p;
                dsv[r] = p * (G[r] - D4[e]);
            }
        }
        // dV^T += dO^T P and dK^T += Q^T dS over this tile's queries
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const bf16x8_t bp = pack8(pv + 8 * kb), bs = pack8(dsv + 8 * kb);
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                acc1[t] = mfma(frag_tr<false>(T1, 32 * it + 16 * kb, 32 * t, true, lane), bp, acc1[t]);
                acc0[t] = mfma(frag_tr<false>(T0, 32 * it + 16 * kb, 32 * t, true, lane), bs, acc0[t]);
            }
        }
    }
    if (ri < len) {
        bf16_t* row = dqkv + (int64_t)(base + ri) * ld + h * DH;
        store_rowT(row + d, acc0, scale, lh);
        store_rowT(row + 2 * d, acc1, 1.f, lh);
    }
}

// Attention of the first token only (the CLS query of each sequence), for
// the last encoder layer, whose output is read at token 0 alone.  One
// workgroup per (sequence, head), thread j on key j, in fp32 from the bf16
// (high, low) parts of q, k and v.  Forward: out row b (compact, [B][d],
// high and low parts) and lse[b H + h] = log sum_j exp(s_j), s_j = scale q.k_j.
__device__ __forceinline__ float ldhl(const bf16_t* hi, const bf16_t* lo, int64_t o) {
    return bf2f(hi[o]) + bf2f(lo[o]);
}
__device__ __forceinline__ float block_reduce2(float v, float* red, bool is_max) {
    // two waves of 64
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float u = __shfl_xor(v, off);
        v = is_max ? fmaxf(v, u) : v + u;
    }
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    const float r = is_max ? fmaxf(red[0], red[1]) : red[0] + red[1];
    __syncthreads();
    return r;
}

// Eight consecutive values from the (high, low) parts at element offset o (16-byte aligned).
__device__ __forceinline__ void ld8hl(const bf16_t* hi, const bf16_t* lo, int64_t o, float* v) {
    const uint4 h = *reinterpret_cast<const uint4*>(hi + o), l = *reinterpret_cast<const uint4*>(lo + o);
    const uint32_t hw[4] = {h.x, h.y, h.z, h.w}, lw[4] = {l.x, l.y, l.z, l.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[2 * e] = bf2f((bf16_t)(hw[e] & 0xFFFFu)) + bf2f((bf16_t)(lw[e] & 0xFFFFu));
        v[2 * e + 1] = bf2f((bf16_t)(hw[e] >> 16)) + bf2f((bf16_t)(lw[e] >> 16));
    }
}
// q . row over the head's 64 columns (row offset o), q in LDS
__device__ __forceinline__ float dot64(const float* q, const bf16_t* hi, const bf16_t* lo, int64_t o) {
    float acc = 0.f, v[8];
#pragma unroll
    for (int c8 = 0; c8 < DH; c8 += 8) {
        ld8hl(hi, lo, o + c8, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(q[c8 + e], v[e], acc);
    }
    return acc;
}
// sum_j w_j row_j[c] for the 64 columns of a head: thread t takes the eight
// columns 8 (t % 8) .. and the keys j = t / 8 (mod 16); the sixteen partial sums
// of a column meet in LDS (part, 16 x 64) and thread c < 64 returns column c.
__device__ __forceinline__ float wsum64(const float* w, int len, const bf16_t* hi, const bf16_t* lo, int64_t o0,
                                        int64_t ld, float (*part)[DH]) {
    const int t = threadIdx.x, c8 = (t & 7) * 8, g = t >> 3;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, v[8];
    for (int j = g; j < len; j += 16) {
        ld8hl(hi, lo, o0 + (int64_t)j * ld + c8, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(w[j], v[e], acc[e]);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) part[g][c8 + e] = acc[e];
    __syncthreads();
    float r = 0.f;
    if (t < DH) {
#pragma unroll
        for (int k = 0; k < 16; ++k) r += part[k][t];
    }
    return r;
}

__global__ void __launch_bounds__(128) attn_cls_fwd(const bf16_t* __restrict__ qkv, const bf16_t* __restrict__ qkvlo,
                                                     const int* __restrict__ cu, bf16_t* __restrict__ out,
                                                     bf16_t* __restrict__ outlo, float* __restrict__ lse, int H, int d,
                                                     float scale) {
    __shared__ float qs[DH], p[LMAX], part[16][DH], red[2];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int64_t ld = 3 * d;
    const int t = threadIdx.x;
    if (t < DH) qs[t] = ldhl(qkv, qkvlo, (int64_t)base * ld + h * DH + t);
    __syncthreads();
    const float sc = t < len ? scale * dot64(qs, qkv, qkvlo, (int64_t)(base + t) * ld + d + h * DH) : -INFINITY;
    const float m = block_reduce2(sc, red, true);
    const float e = t < len ? expf(sc - m) : 0.f;
    const float sum = block_reduce2(e, red, false);
    p[t] = e / sum;
    if (t == 0) lse[(int64_t)b * H + h] = m + logf(sum);
    __syncthreads();
    const float v = wsum64(p, len, qkv, qkvlo, (int64_t)base * ld + 2 * d + h * DH, ld, part);
    if (t < DH) {
        const bf16_t hi = f2bf(v);
        const int64_t o = (int64_t)b * d + h * DH + t;
        out[o] = hi;
        outlo[o] = f2bf(v - bf2f(hi));
    }
}

// Backward of attn_cls_fwd, given dO of the first token (compact rows, bf16)
// and the forward's O (compact, high and low parts) and lse:
//   p_j = exp(s_j - lse), D = dO . O, ds_j = p_j (dO . v_j - D)
//   dq = scale sum_j ds_j k_j (row 0 of the sequence), dk_j = scale ds_j q,
//   dv_j = p_j dO; the query part of every other row is zero.  Writes every
// row of the sequence in dqkv (bf16, [T][3d]).
__global__ void __launch_bounds__(128) attn_cls_bwd(const bf16_t* __restrict__ qkv, const bf16_t* __restrict__ qkvlo,
                                                     const int* __restrict__ cu, const bf16_t* __restrict__ out,
                                                     const bf16_t* __restrict__ outlo, const bf16_t* __restrict__ dout,
                                                     const float* __restrict__ lse, bf16_t* __restrict__ dqkv, int H,
                                                     int d, float scale) {
    __shared__ float qs[DH], dos[DH], p[LMAX], ds[LMAX], part[16][DH], red[2];
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int base = cu[b], len = cu[b + 1] - cu[b];
    const int64_t ld = 3 * d;
    const int t = threadIdx.x;
    float dprod = 0.f;
    if (t < DH) {
        qs[t] = ldhl(qkv, qkvlo, (int64_t)base * ld + h * DH + t);
        const int64_t o = (int64_t)b * d + h * DH + t;
        dos[t] = bf2f(dout[o]);
        dprod = dos[t] * ldhl(out, outlo, o);
    }
    const float Dv = block_reduce2(dprod, red, false);  // (also orders the stores of qs, dos)
    const float L = lse[(int64_t)b * H + h];
    float pj = 0.f, dsj = 0.f;
    if (t < len) {
        const int64_t o = (int64_t)(base + t) * ld + h * DH;
        pj = expf(scale * dot64(qs, qkv, qkvlo, o + d) - L);
        dsj = pj * (dot64(dos, qkv, qkvlo, o + 2 * d) - Dv);
    }
    p[t] = pj;
    ds[t] = dsj;
    __syncthreads();
    // rows: eight threads per row, 8 columns each, for the q (zero past row 0), k and v parts
    for (int idx = t; idx < len * 8; idx += blockDim.x) {
        const int j = idx >> 3, c8 = (idx & 7) * 8;
        bf16_t* row = dqkv + (int64_t)(base + j) * ld + h * DH + c8;
        uint32_t kw[4], vw[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            kw[e] = f2bf2(scale * ds[j] * qs[c8 + 2 * e], scale * ds[j] * qs[c8 + 2 * e + 1]);
            vw[e] = f2bf2(p[j] * dos[c8 + 2 * e], p[j] * dos[c8 + 2 * e + 1]);
        }
        if (j > 0) *reinterpret_cast<uint4*>(row) = make_uint4(0, 0, 0, 0);
        *reinterpret_cast<uint4*>(row + d) = make_uint4(kw[0], kw[1], kw[2], kw[3]);
        *reinterpret_cast<uint4*>(row + 2 * d) = make_uint4(vw[0], vw[1], vw[2], vw[3]);
    }
    // dq (row 0)
    const float dq = wsum64(ds, len, qkv, qkvlo, (int64_t)base * ld + d + h * DH, ld, part);
    if (t < DH) dqkv[(int64_t)base * ld + h * DH + t] = f2bf(scale * dq);
}

}  // namespace

fo_status launch_attn_fwd(const bf16_t* qkv, const bf16_t* qkvlo, const int* cu, bf16_t* out, bf16_t* outlo,
                          float* lse, int B, int H, int d, hipStream_t s, const int* order) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    ProfInfo pi;
    pi.kind = PROF_ATTN_FWD; pi.cu = cu; pi.B = B; pi.d = d;
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("attn_fwd_mfma", pi, &ea, &eb);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipExtLaunchKernelGGL(attn_fwd_mfma, dim3(B * H), dim3(256), 0, s, ea, eb, 0, qkv, qkvlo, cu, out, outlo, lse, H,
                          d, 1.f / sqrtf((float)DH), snap, B, order);
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_attn_bwd(const bf16_t* qkv, const int* cu, const bf16_t* out, const bf16_t* dout,
                          const float* lse, bf16_t* dqkv, int B, int H, int d, hipStream_t s, const int* order) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    const float scale = 1.f / sqrtf((float)DH);
    ProfInfo pi;
    pi.kind = PROF_ATTN_BWD; pi.cu = cu; pi.B = B; pi.d = d;
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("attn_bwd_mfma", pi, &ea, &eb);
    int* snap = B + 1 <= kProfSnapInts ? prof_snap(h) : nullptr;
    hipExtLaunchKernelGGL(attn_bwd_mfma, dim3(2 * B * H), dim3(256), 0, s, ea, eb, 0, qkv, cu, out, dout, lse, dqkv, H, d,
                          scale, snap, B, order);
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_attn_cls_fwd(const bf16_t* qkv, const bf16_t* qkvlo, const int* cu, bf16_t* out, bf16_t* outlo,
                              float* lse, int B, int H, int d, hipStream_t s) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("attn_cls_fwd", ProfInfo(), &ea, &eb);
    hipExtLaunchKernelGGL(attn_cls_fwd, dim3(B * H), dim3(128), 0, s, ea, eb, 0, qkv, qkvlo, cu, out, outlo, lse, H, d,
                          1.f / sqrtf((float)DH));
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_attn_cls_bwd(const bf16_t* qkv, const bf16_t* qkvlo, const int* cu, const bf16_t* out,
                              const bf16_t* outlo, const bf16_t* dout, const float* lse, bf16_t* dqkv, int B, int H,
                              int d, hipStream_t s) {
    FO_CHECK(d == H * DH, "attention: d=%d must equal heads*%d", d, DH);
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("attn_cls_bwd", ProfInfo(), &ea, &eb);
    hipExtLaunchKernelGGL(attn_cls_bwd, dim3(B * H), dim3(128), 0, s, ea, eb, 0, qkv, qkvlo, cu, out, outlo, dout, lse,
                          dqkv, H, d, 1.f / sqrtf((float)DH));
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
