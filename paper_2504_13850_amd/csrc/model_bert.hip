// Config 4: the BERT-base-shaped server network (10 post-LN encoder layers,
// d = 768, 12 heads of 64, FFN 3072 with exact GELU, tanh pooler on the first
// token, linear 768 -> 2), one training iteration of the activation branch
// of Alg. 4 on bf16 MFMA GEMMs with fp32 accumulation and fp32 master weights.
// The forward GEMMs are compensated products (bf16 high + low parts of both
// operands, three MFMA passes): through ten layers plain bf16 operands move
// the logits by 2-3% of their size, the compensated forward by ~1e-5.  The
// backward GEMMs use the high parts only.
//
// Variable-length batches run packed: only the sum(len_b) = T valid tokens
// are stored and computed ([T][d] row-major, sequence b at rows cu[b]..).
// Because padded keys are masked out of every attention and the loss reads
// only the first token, padded positions never influence the loss: packing
// gives the same loss, logits and gradients as the padded formulation.  T
// stays on the device (cu[B]); grids are sized for B*L rows and the work
// past T exits early, so a step needs no host synchronisation.
#include "gemm.h"
#include "model.h"

namespace fo {
namespace {

constexpr int D = 768, NH = 12, FF = 3072, NL = 10, L = 128, NC = 2;
// Workgroups of a layer's grouped weight-gradient launch (side stream): fewer
// than its tiles, so that the input-gradient chain on the main stream keeps
// workgroup slots on every CU.
constexpr int kWgradMaxWG = 256;
constexpr int64_t kLayer = (int64_t)3 * D * D + 3 * D + (int64_t)D * D + D + 2 * D + (int64_t)FF * D + FF +
                           (int64_t)D * FF + D + 2 * D;
constexpr int64_t kParams = NL * kLayer + (int64_t)D * D + D + (int64_t)NC * D + NC;

struct LayerOff {
    int64_t wqkv, bqkv, wo, bo, g1, b1, w1, bf1, w2, bf2, g2, b2;
};

struct LayerAct {
    bf16_t *qkv, *qkvlo;                // projection output, bf16 high and low parts
    bf16_t *O, *Olo, *Hb, *Hlo, *dgelu1, *G, *Glo;  // dgelu1 = GELU'(FFN1 pre-activation)
    float *lse, *u1, *mean1, *rstd1, *Hf, *u2, *mean2, *rstd2;
};

struct Plan {
    int rows;  // max_batch * L
    int* cu;   // [2 max_batch + 2]; cu[B] = T, cu[B + 1] = B, then the sequences by decreasing length
    LayerOff off[NL];
    int64_t pool_w, pool_b, cls_w, cls_b;
    bf16_t* Xb[NL + 1];
    bf16_t* Xlo[NL + 1];  // low parts (layer 0's input is exactly bf16: none)
    float* Xf[NL + 1];
    LayerAct a[NL];
    float *dY[2], *du2f, *dHf, *du1f;
    // operands of the weight gradients, one set per layer parity: the gradients
    // of layer l run on the side stream while the main stream goes on to l - 1
    bf16_t *du2b[2], *dA1[2], *du1b[2], *dqkv[2];
    bf16_t* dO;
    float *splitws, *slws;
    // column-sum partials per layer parity, finished on the side stream: the FFN1
    // bias gradient (colwsF), the two norms' dgamma / dbeta / bias gradient
    // (lnpart[parity][0] LN2, [1] LN1); colws2: the side stream's own (bqkv);
    // colws2m: the main stream's, for the first layer's (the backward's last)
    float *colwsF[2], *lnpart[2][2], *colws2, *colws2m;
    float *pooled, *dz, *dpool, *dxc;
    float* xres;  // the last layer's residual input at the first tokens, [B][D]
    // parameter ranges whose SGD update is not fused into a weight-gradient
    // product (biases, norm parameters, pooler, classifier): device [n][2]
    int64_t* sgd_chunks = nullptr;
    int n_sgd_chunks = 0;
    hipStream_t side = nullptr;      // weight gradients of the backward
    hipEvent_t ev_fork = nullptr;    // main -> side: an operand is ready
    hipEvent_t ev_done[2] = {};      // side -> main: a parity's operands are free again
    hipEvent_t ev_join = nullptr;    // side -> main: every weight gradient is written
    hipEvent_t ev_cols = nullptr;    // side -> main: the column sums of every layer but the first are written
};

// ------------------------------------------------------------------ kernels
// Packed offsets cu[0..B] (cu[B] = T), cu[B + 1] = B, and from cu + B + 2 the
// sequences by decreasing length (ties by index): the launch order of the
// attention workgroups.  The clamped lengths go to LDS (dynamic, B ints); a
// thread per sequence computes its rank, one thread the prefix sum.
// Lengths outside [1, Lmax] are clamped (every access then stays in bounds)
// and counted into *bad_out.
__global__ void __launch_bounds__(256) build_cu_kernel(const StepIn* __restrict__ in, int B, int Lmax,
                                                       int* __restrict__ cu, float* __restrict__ bad_out) {
    extern __shared__ int lens[];
    const int32_t* __restrict__ lengths = in->lengths;
    __shared__ int bad;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        const int len = lengths[b];
        if (len < 1 || len > Lmax) atomicAdd(&bad, 1);
        lens[b] = len < 1 ? 1 : (len > Lmax ? Lmax : len);
    }
    __syncthreads();
    if (threadIdx.x == 0) *bad_out = (float)bad;
    if (threadIdx.x == 0) {
        int acc = 0;
        for (int b = 0; b < B; ++b) {
            cu[b] = acc;
            acc += lens[b];
        }
        cu[B] = acc;
        cu[B + 1] = B;  // the row count of the last layer's first-token rows
    }
    int* order = cu + B + 2;
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        const int lb = lens[b];
        int rank = 0;
        for (int c = 0; c < B; ++c) rank += lens[c] > lb || (lens[c] == lb && c < b);
        order[rank] = b;
    }
}

// padded [B][L][D] bf16 -> packed rows (bf16 and fp32 copies)
__global__ void __launch_bounds__(256) pack_kernel(const StepIn* __restrict__ in, const int* __restrict__ cu, int B,
                                                   bf16_t* __restrict__ xb, float* __restrict__ xf) {
    const bf16_t* __restrict__ x = static_cast<const bf16_t*>(in->x);
    const int64_t total = (int64_t)B * L * (D / 8);
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        int c8 = (int)(idx % (D / 8));
        int64_t bp = idx / (D / 8);
        int b = (int)(bp / L), pos = (int)(bp % L);
        if (pos >= cu[b + 1] - cu[b]) continue;
        int64_t row = cu[b] + pos;
        uint4 v = reinterpret_cast<const uint4*>(x + bp * D)[c8];
        reinterpret_cast<uint4*>(xb + row * D)[c8] = v;
        float* f = xf + row * D + c8 * 8;
        uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            f[2 * e] = bf2f((bf16_t)(w[e] & 0xFFFFu));
            f[2 * e + 1] = bf2f((bf16_t)(w[e] >> 16));
        }
    }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}


// y = gamma * (u - mean) * rstd + beta over each row of D; one wave per row.
// LayerNorm over rows of D = 768: one wave per row, each lane four adjacent
// columns 4 lane + 256 k (k = 0..2) with 16-byte loads and stores.
constexpr int PER4 = D / 256;
__device__ __forceinline__ f32x4 ld4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ void st4(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
__device__ __forceinline__ void st4bf(bf16_t* p, f32x4 v) {
    *reinterpret_cast<uint2*>(p) = make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
}
__device__ __forceinline__ f32x4 bf4lo(f32x4 v) {  // v - bf16(v), elementwise
    f32x4 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = v[q] - bf2f(f2bf(v[q]));
    return r;
}

// The lane's PER4 column groups (4 lane + 256 k .. + 3) of row `row` of a product
// whose split-K reduction was deferred to this consumer, summed over its S
// active slices (the reduction pass's order) plus bias and residual; S = 1: the
// product's own output.  S is a template parameter so that every load of the
// row is in flight before the first add.
template <int S>
__device__ __forceinline__ void split_row(const SplitRows& src, int row, int lane, f32x4 (&x)[PER4]) {
    if constexpr (S == 1) {
#pragma unroll
        for (int k = 0; k < PER4; ++k) x[k] = ld4(src.x + (int64_t)row * D + 4 * lane + 256 * k);
    } else {
        const int64_t full = (int64_t)src.M * D;
        f32x4 p[PER4][S], bb[PER4], rr[PER4];
        const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < PER4; ++k) {
            const int c = 4 * lane + 256 * k;
#pragma unroll
            for (int z = 0; z < S; ++z) p[k][z] = ld4(src.ws + z * full + (int64_t)row * D + c);
            bb[k] = src.bias ? ld4(src.bias + c) : zero;
            rr[k] = src.resid ? ld4(src.resid + (int64_t)row * D + c) : zero;
        }
#pragma unroll
        for (int k = 0; k < PER4; ++k) {
            f32x4 v = p[k][0];
            int z = 1;
#pragma unroll
            for (; z + 3 < S; z += 4) v += (p[k][z] + p[k][z + 1]) + (p[k][z + 2] + p[k][z + 3]);
#pragma unroll
            for (; z < S; ++z) v += p[k][z];
            x[k] = (v + bb[k]) + rr[k];
        }
    }
}
__device__ __forceinline__ void load_split_row(const SplitRows& src, int S, int row, int lane, f32x4 (&x)[PER4]) {
    switch (S) {
        case 2: split_row<2>(src, row, lane, x); break;
        case 3: split_row<3>(src, row, lane, x); break;
        case 4: split_row<4>(src, row, lane, x); break;
        case 8: split_row<8>(src, row, lane, x); break;  // the last layer's first-token products
        case 1: split_row<1>(src, row, lane, x); break;
        default: {  // other slice counts: loads issued four at a time
            const int64_t full = (int64_t)src.M * D;
            const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < PER4; ++k) {
                const int c = 4 * lane + 256 * k;
                const float* p = src.ws + (int64_t)row * D + c;
                f32x4 v = ld4(p);
                int z = 1;
                for (; z + 3 < S; z += 4)
                    v += (ld4(p + z * full) + ld4(p + (z + 1) * full)) + (ld4(p + (z + 2) * full) + ld4(p + (z + 3) * full));
                for (; z < S; ++z) v += ld4(p + z * full);
                x[k] = (v + (src.bias ? ld4(src.bias + c) : zero)) +
                       (src.resid ? ld4(src.resid + (int64_t)row * D + c) : zero);
            }
        }
    }
}

// The input row u comes from `src` (a product whose split-K reduction is
// summed here when deferred; the sum is then also stored to u_store, the
// copy the backward reads).
__global__ void __launch_bounds__(256) ln_fwd_kernel(const SplitRows src, float* __restrict__ u_store,
                                                     const float* __restrict__ g, const float* __restrict__ beta,
                                                     const int* __restrict__ Tdev, float* __restrict__ yf,
                                                     bf16_t* __restrict__ yb, bf16_t* __restrict__ ylo,
                                                     float* __restrict__ mean, float* __restrict__ rstd) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int T = *Tdev;
    if (row >= T) return;
    const int S = src.active(T);
    // the norm's parameters are loaded with the row, not after its reductions
    f32x4 gg[PER4], bb[PER4];
#pragma unroll
    for (int k = 0; k < PER4; ++k) {
        gg[k] = ld4(g + 4 * lane + 256 * k);
        bb[k] = ld4(beta + 4 * lane + 256 * k);
    }
    f32x4 x[PER4];
    load_split_row(src, S, row, lane, x);
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < PER4; ++k) {
        if (S > 1) st4(u_store + (int64_t)row * D + 4 * lane + 256 * k, x[k]);
        s += (x[k][0] + x[k][1]) + (x[k][2] + x[k][3]);
    }
    const float mu = wave_sum(s) * (1.f / D);
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < PER4; ++k) {
        x[k] -= mu;
#pragma unroll
        for (int q = 0; q < 4; ++q) v = fmaf(x[k][q], x[k][q], v);
    }
    const float rs = rsqrtf(wave_sum(v) * (1.f / D) + 1e-5f);
#pragma unroll
    for (int k = 0; k < PER4; ++k) {
        const int c = 4 * lane + 256 * k;
        f32x4 y;
#pragma unroll
        for (int q = 0; q < 4; ++q) y[q] = fmaf(x[k][q] * rs, gg[k][q], bb[k][q]);
        st4(yf + (int64_t)row * D + c, y);
        st4bf(yb + (int64_t)row * D + c, y);
        st4bf(ylo + (int64_t)row * D + c, bf4lo(y));
    }
    if (lane == 0) {
        mean[row] = mu;
        rstd[row] = rs;
    }
}
// dx = rstd * (gdy - mean(gdy) - xhat * mean(gdy * xhat)), gdy = dy * gamma.
// A block takes LNB_ROWS consecutive rows (a quarter per wave, all of a wave's
// rows loaded first) and also writes column partial sums of the norm's
// parameter gradients and of dx: part[block][0][c] = sum dy * xhat (dgamma),
// part[block][1][c] = sum dy (dbeta), part[block][2][c] = sum dx (the bias
// gradient of the sublayer whose sum with the residual this norm normalises).
constexpr int LNB_ROWS = 4;
__global__ void __launch_bounds__(256) ln_bwd_kernel(const SplitRows dy, const float* __restrict__ u,
                                                     const float* __restrict__ mean, const float* __restrict__ rstd,
                                                     const float* __restrict__ g, const int* __restrict__ Tdev,
                                                     float* __restrict__ dxf, bf16_t* __restrict__ dxb,
                                                     float* __restrict__ part) {
    __builtin_amdgcn_s_setprio(2);  // on the input-gradient chain (see gemm_rk_krt_dma_kernel)
    constexpr int RW = LNB_ROWS / 4;  // rows per wave
    __shared__ float red[4][D];
    const int T = *Tdev;
    const int r0 = blockIdx.x * LNB_ROWS;
    if (r0 >= T) return;  // uniform
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int S = dy.active(T);
    f32x4 gam[PER4], pg[PER4], pb[PER4], px[PER4];
#pragma unroll
    for (int k = 0; k < PER4; ++k) {
        gam[k] = ld4(g + 4 * lane + 256 * k);
        pg[k] = pb[k] = px[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    f32x4 dv[RW][PER4], uv[RW][PER4];
    float mu[RW], rs[RW];
#pragma unroll
    for (int i = 0; i < RW; ++i) {
        const int row = min(r0 + wave * RW + i, T - 1);  // rows past T load row T - 1 and are skipped
        mu[i] = mean[row];
        rs[i] = rstd[row];
        load_split_row(dy, S, row, lane, dv[i]);
#pragma unroll
        for (int k = 0; k < PER4; ++k) uv[i][k] = ld4(u + (int64_t)row * D + 4 * lane + 256 * k);
    }
#pragma unroll
    for (int i = 0; i < RW; ++i) {
        const int row = r0 + wave * RW + i;
        if (row >= T) break;
        f32x4 xh[PER4], gd[PER4];
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int k = 0; k < PER4; ++k) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float d = dv[i][k][q];
                xh[k][q] = (uv[i][k][q] - mu[i]) * rs[i];
                gd[k][q] = d * gam[k][q];
                pg[k][q] = fmaf(d, xh[k][q], pg[k][q]);
                pb[k][q] += d;
                s1 += gd[k][q];
                s2 = fmaf(gd[k][q], xh[k][q], s2);
            }
        }
        s1 = wave_sum(s1) * (1.f / D);
        s2 = wave_sum(s2) * (1.f / D);
#pragma unroll
        for (int k = 0; k < PER4; ++k) {
            const int c = 4 * lane + 256 * k;
            f32x4 dx;
#pragma unroll
            for (int q = 0; q < 4; ++q) dx[q] = rs[i] * (gd[k][q] - s1 - xh[k][q] * s2);
            px[k] += dx;
            st4(dxf + (int64_t)row * D + c, dx);
            st4bf(dxb + (int64_t)row * D + c, dx);
        }
    }
    float* out = part + (int64_t)blockIdx.x * 3 * D;
#pragma unroll
    for (int q = 0; q < 3; ++q) {
#pragma unroll
        for (int k = 0; k < PER4; ++k)
            *reinterpret_cast<f32x4*>(&red[wave][4 * lane + 256 * k]) = q == 0 ? pg[k] : (q == 1 ? pb[k] : px[k]);
        __syncthreads();
        for (int c = threadIdx.x; c < D; c += 256)
            out[q * D + c] = (red[0][c] + red[1][c]) + (red[2][c] + red[3][c]);
        __syncthreads();
    }
}

__global__ void __launch_bounds__(256) gather_cls_kernel(const float* __restrict__ X, const int* __restrict__ cu,
                                                         int B, float* __restrict__ xc) {
    const int b = blockIdx.x;
    for (int c = threadIdx.x; c < D; c += blockDim.x) xc[(int64_t)b * D + c] = X[(int64_t)cu[b] * D + c];
}

__global__ void __launch_bounds__(256) scatter_cls_kernel(const float* __restrict__ dxc, const int* __restrict__ cu,
                                                          int B, float* __restrict__ dY) {
    const int b = blockIdx.x;
    for (int c = threadIdx.x; c < D; c += blockDim.x) dY[(int64_t)cu[b] * D + c] = dxc[(int64_t)b * D + c];
}

// ------------------------------------------------------------------ plan
// Maximum K slices of a forward / input-gradient product over the packed rows;
// the kernel takes as many of them as the device-side row count needs to fill
// the CUs (fused epilogue in the reduction pass).  K is the product's full
// reduction length, with the compensated segments.
int split_rows(int K) {
    int s = 4;
    while (s > 1 && K / s < 256) --s;
    return s;
}

// The ranges of the flat parameter vector that the final SGD pass updates:
// everything except the four weight matrices of each layer, whose update runs
// in the epilogue of their weight-gradient products.  Ranges are cut into
// chunks of at most 4096 (one block each).
constexpr int kSgdChunk = 4096;
constexpr int kMaxSgdChunks = 512;
std::vector<int64_t> sgd_ranges(const LayerOff* off, int64_t pool_w) {
    std::vector<int64_t> r;
    auto add = [&](int64_t a, int64_t b) {
        for (int64_t o = a; o < b; o += kSgdChunk) {
            r.push_back(o);
            r.push_back(std::min<int64_t>(kSgdChunk, b - o));
        }
    };
    for (int l = 0; l < NL; ++l) {
        const LayerOff& f = off[l];
        add(f.bqkv, f.wo);  // bqkv
        add(f.bo, f.w1);    // bo, ln1 gamma, beta
        add(f.bf1, f.w2);   // bf1
        add(f.bf2, l + 1 < NL ? off[l + 1].wqkv : pool_w);  // bf2, ln2 gamma, beta
    }
    add(pool_w, kParams);  // pooler and classifier
    return r;
}

size_t ws_bytes(const fo_model* m) {
    const size_t R = (size_t)m->max_batch * L, B = (size_t)m->max_batch;
    size_t s = 0;
    auto add = [&](size_t b) { s += (b + 255) & ~size_t(255); };
    add(sizeof(Plan));
    add(4 * (2 * B + 2));
    for (int l = 0; l <= NL; ++l) {
        add(2 * R * D);
        add(2 * R * D);
        add(4 * R * D);
    }
    for (int l = 0; l < NL; ++l) {
        add(2 * R * 3 * D); add(2 * R * 3 * D);     // qkv, qkvlo
        add(2 * R * D); add(2 * R * D);             // O, Olo
        add(2 * R * D); add(2 * R * D);             // Hb, Hlo
        add(2 * R * FF);                            // dgelu1
        add(2 * R * FF); add(2 * R * FF);           // G, Glo
        add(4 * B * NH * L);                        // lse
        add(4 * R * D); add(4 * R); add(4 * R);     // u1, mean1, rstd1
        add(4 * R * D);                             // Hf
        add(4 * R * D); add(4 * R); add(4 * R);     // u2, mean2, rstd2
    }
    add(4 * R * D); add(4 * R * D);                 // dY[2]
    add(4 * R * D); add(4 * R * D); add(4 * R * D); // du2f, dHf, du1f
    for (int p = 0; p < 2; ++p) {
        add(2 * R * D); add(2 * R * FF); add(2 * R * D); add(2 * R * 3 * D);  // du2b, dA1, du1b, dqkv
    }
    add(2 * R * D);                                 // dO
    // split-K partials of the forward and input-gradient products (weight
    // gradients run unsplit, grouped per layer)
    add(std::max(gemm_ws_bytes((int)R, D, 4), gemm_ws_bytes((int)B, FF, 4)));
    for (int q = 0; q < 2; ++q) add(4 * colsum_ws_floats((int)R, FF));
    add(4 * colsum_ws_floats((int)R, 3 * D));
    add(4 * colsum_ws_floats((int)R, 3 * D));
    for (int q = 0; q < 4; ++q) add(4 * (size_t)cdiv(R, LNB_ROWS) * 3 * D);
    add(4 * small_linear_ws_floats((int)B, D, D));
    add(4 * B * D); add(4 * B * NC); add(4 * B * D); add(4 * B * D); add(4 * B * D);
    add(16 * kMaxSgdChunks);
    return s;
}

fo_status init(fo_model* m) {
    Plan* P = new (std::nothrow) Plan();
    if (!P) return FO_ENOMEM;
    m->plan = P;
    const size_t R = (size_t)m->max_batch * L, B = (size_t)m->max_batch;
    P->rows = (int)R;
    int64_t o = 0;
    for (int l = 0; l < NL; ++l) {
        LayerOff& f = P->off[l];
        f.wqkv = o; o += (int64_t)3 * D * D;
        f.bqkv = o; o += 3 * D;
        f.wo = o; o += (int64_t)D * D;
        f.bo = o; o += D;
        f.g1 = o; o += D;
        f.b1 = o; o += D;
        f.w1 = o; o += (int64_t)FF * D;
        f.bf1 = o; o += FF;
        f.w2 = o; o += (int64_t)D * FF;
        f.bf2 = o; o += D;
        f.g2 = o; o += D;
        f.b2 = o; o += D;
    }
    P->pool_w = o; o += (int64_t)D * D;
    P->pool_b = o; o += D;
    P->cls_w = o; o += (int64_t)NC * D;
    P->cls_b = o; o += NC;
    if (o != kParams) {
        set_error("bert: layout mismatch");
        return FO_EINVAL;
    }
    Arena& a = m->arena;
    a.take<char>(sizeof(Plan));
    P->cu = a.take<int>(2 * B + 2);
    for (int l = 0; l <= NL; ++l) {
        P->Xb[l] = a.take<bf16_t>(R * D);
        P->Xlo[l] = a.take<bf16_t>(R * D);
        P->Xf[l] = a.take<float>(R * D);
    }
    for (int l = 0; l < NL; ++l) {
        LayerAct& t = P->a[l];
        t.qkv = a.take<bf16_t>(R * 3 * D);
        t.qkvlo = a.take<bf16_t>(R * 3 * D);
        t.O = a.take<bf16_t>(R * D);
        t.Olo = a.take<bf16_t>(R * D);
        t.Hb = a.take<bf16_t>(R * D);
        t.Hlo = a.take<bf16_t>(R * D);
        t.dgelu1 = a.take<bf16_t>(R * FF);
        t.G = a.take<bf16_t>(R * FF);
        t.Glo = a.take<bf16_t>(R * FF);
        t.lse = a.take<float>(B * NH * L);
        t.u1 = a.take<float>(R * D);
        t.mean1 = a.take<float>(R);
        t.rstd1 = a.take<float>(R);
        t.Hf = a.take<float>(R * D);
        t.u2 = a.take<float>(R * D);
        t.mean2 = a.take<float>(R);
        t.rstd2 = a.take<float>(R);
    }
    P->dY[0] = a.take<float>(R * D);
    P->dY[1] = a.take<float>(R * D);
    P->du2f = a.take<float>(R * D);
    P->dHf = a.take<float>(R * D);
    P->du1f = a.take<float>(R * D);
    for (int p = 0; p < 2; ++p) {
        P->du2b[p] = a.take<bf16_t>(R * D);
        P->dA1[p] = a.take<bf16_t>(R * FF);
        P->du1b[p] = a.take<bf16_t>(R * D);
        P->dqkv[p] = a.take<bf16_t>(R * 3 * D);
    }
    P->dO = a.take<bf16_t>(R * D);
    const size_t sw = std::max(gemm_ws_bytes((int)R, D, 4), gemm_ws_bytes((int)B, FF, 4));
    P->splitws = a.take<float>(sw / 4 + 1);
    for (int q = 0; q < 2; ++q) P->colwsF[q] = a.take<float>(colsum_ws_floats((int)R, FF));
    P->colws2 = a.take<float>(colsum_ws_floats((int)R, 3 * D));
    P->colws2m = a.take<float>(colsum_ws_floats((int)R, 3 * D));
    for (int q = 0; q < 4; ++q) P->lnpart[q / 2][q % 2] = a.take<float>((size_t)cdiv(R, LNB_ROWS) * 3 * D);
    P->slws = a.take<float>(small_linear_ws_floats((int)B, D, D));
    P->pooled = a.take<float>(B * D);
    P->dz = a.take<float>(B * NC);
    P->dpool = a.take<float>(B * D);
    P->dxc = a.take<float>(B * D);
    P->xres = a.take<float>(B * D);
    P->sgd_chunks = a.take<int64_t>(2 * kMaxSgdChunks);
    if (!P->sgd_chunks) {
        set_error("bert: workspace arena too small");
        return FO_ENOMEM;
    }
    {
        const std::vector<int64_t> r = sgd_ranges(P->off, P->pool_w);
        P->n_sgd_chunks = (int)(r.size() / 2);
        FO_CHECK(P->n_sgd_chunks <= kMaxSgdChunks, "bert: %d SGD ranges", P->n_sgd_chunks);
        FO_HIP(hipMemcpy(P->sgd_chunks, r.data(), r.size() * sizeof(int64_t), hipMemcpyHostToDevice));
    }
    if (!P->dxc) {
        set_error("bert: workspace arena too small");
        return FO_ENOMEM;
    }
    // default priority, no implicit ordering with the null stream
    FO_HIP(hipStreamCreateWithFlags(&P->side, hipStreamNonBlocking));
    for (hipEvent_t* e : {&P->ev_fork, &P->ev_done[0], &P->ev_done[1], &P->ev_join, &P->ev_cols})
        FO_HIP(hipEventCreateWithFlags(e, hipEventDisableTiming));
    return FO_OK;
}


#define TRY(x)                           \
    do {                                 \
        fo_status st_ = (x);             \
        if (st_ != FO_OK) return st_;    \
    } while (0)

// C[rows][N] = A[rows][K] W^T (+ epilogue): the forward of a linear layer as a
// compensated product (A = A + Alo, W = W + Wlo in bf16 parts; Alo == NULL
// when A is exactly bf16).
GemmDesc lin_fwd(int rows, const bf16_t* A, const bf16_t* Alo, int K, const bf16_t* W, const bf16_t* Wlo, int N) {
    GemmDesc d;
    d.M = rows; d.N = N; d.K = K;
    d.amode = OP_RK; d.A = A; d.A2 = Alo; d.lda = K;
    d.bmode = OP_RK; d.B = W; d.B2 = Wlo; d.ldb = K;
    d.nseg = Alo ? 3 : 2;
    return d;
}

// Backward of a norm: dx (fp32 and bf16) plus dgamma, dbeta and the column
// sum of dx (into dbias_below).
// The rows of a GEMM's output as its consumer reads them when the GEMM leaves
// its split-K reduction to that consumer (Cf, ldcf = ldr = N).
SplitRows deferred_rows(const GemmDesc& g) {
    SplitRows r;
    r.x = g.Cf;
    r.ws = g.splits > 1 ? g.ws : nullptr;
    r.bias = g.bias;
    r.resid = g.resid;
    r.M = g.M;
    r.N = g.N;
    r.splits = g.splits;
    r.ktot = g.nseg * (g.nseg > 1 ? (int)cdiv(g.K, 64) * 64 : g.K);
    return r;
}
SplitRows plain_rows(const float* x, int M) {
    SplitRows r;
    r.x = x;
    r.M = M;
    r.N = D;
    return r;
}

fo_status ln_bwd(const SplitRows& dy, const float* u, const float* mean, const float* rstd, const float* gamma,
                 const int* Tdev, int rows, float* dxf, bf16_t* dxb, float* part, hipStream_t s) {
    hipLaunchKernelGGL(ln_bwd_kernel, dim3(cdiv(rows, LNB_ROWS)), dim3(256), 0, s, dy, u, mean, rstd, gamma, Tdev,
                       dxf, dxb, part);
    FO_LAUNCHED();
    return FO_OK;
}
fo_status step(fo_model* m, const fo_acts* acts, const int32_t* labels) {
    Plan* P = (Plan*)m->plan;
    hipStream_t s = m->stream;
    const int B = acts->batch, rows = B * L;
    const int* Tdev = P->cu + B;
    const bf16_t* W = m->w16;
    const bf16_t* Wl = m->w16lo;
    const float* prm = m->params;
    float* grd = m->grads;

    hipLaunchKernelGGL(build_cu_kernel, dim3(1), dim3(256), sizeof(int) * B, s, m->dev_in, B, L, P->cu,
                       m->loss + 2);
    {
        int64_t total = (int64_t)rows * (D / 8);
        int grid = (int)std::min<int64_t>(cdiv(total, 256), 8192);
        hipLaunchKernelGGL(pack_kernel, dim3(grid), dim3(256), 0, s, m->dev_in, P->cu, B, P->Xb[0],
                           P->Xf[0]);
    }
    FO_LAUNCHED();

    // ---------------- forward (Alg. 4: forward pass of M_s)
    // The loss reads the last layer's output at the first token of each
    // sequence only, so that layer runs its key / value projection over every
    // token and everything after it (first-token attention, output projection,
    // norms, FFN) over the B first-token rows, compactly ([B][D], row b =
    // sequence b).  The result is exact: no other row of the last layer reaches
    // the loss.
    const int* Bdev = P->cu + B + 1;  // device copy of B
    for (int l = 0; l < NL; ++l) {
        const LayerOff& f = P->off[l];
        LayerAct& t = P->a[l];
        const bool cls = l == NL - 1;
        GemmDesc q = lin_fwd(rows, P->Xb[l], l ? P->Xlo[l] : nullptr, D, W + f.wqkv, Wl + f.wqkv, 3 * D);
        q.Mdev = Tdev;
        q.bias = prm + f.bqkv;
        q.Cb = t.qkv; q.Cb2 = t.qkvlo; q.ldcb = 3 * D;
        TRY(gemm(q, s));
        // rows of the rest of the layer: every token, or the B first tokens
        const int M = cls ? B : rows;
        const int* Mdev = cls ? Bdev : Tdev;
        const dim3 lng((unsigned)cdiv(M, 4));
        if (cls) {
            TRY(launch_attn_cls_fwd(t.qkv, t.qkvlo, P->cu, t.O, t.Olo, t.lse, B, NH, D, s));
            hipLaunchKernelGGL(gather_cls_kernel, dim3(B), dim3(256), 0, s, P->Xf[l], P->cu, B, P->xres);
            FO_LAUNCHED();
        } else {
            TRY(launch_attn_fwd(t.qkv, t.qkvlo, P->cu, t.O, t.Olo, t.lse, B, NH, D, s, P->cu + B + 2));
        }
        GemmDesc o = lin_fwd(M, t.O, t.Olo, D, W + f.wo, Wl + f.wo, D);
        o.Mdev = Mdev;
        o.splits = cls ? 8 : 2; o.ws = P->splitws;  // (two slices time like four and halve the LayerNorm's reads)
        o.bias = prm + f.bo;
        o.resid = cls ? P->xres : P->Xf[l]; o.ldr = D;
        o.Cf = t.u1; o.ldcf = D;
        o.defer_reduce = true;  // summed by the LayerNorm below
        TRY(gemm(o, s));
        hipLaunchKernelGGL(ln_fwd_kernel, lng, dim3(256), 0, s, deferred_rows(o), t.u1, prm + f.g1, prm + f.b1, Mdev,
                           t.Hf, t.Hb, t.Hlo, t.mean1, t.rstd1);
        GemmDesc f1 = lin_fwd(M, t.Hb, t.Hlo, D, W + f.w1, Wl + f.w1, FF);
        f1.Mdev = Mdev;
        if (cls) { f1.splits = 4; f1.ws = P->splitws; }  // (B rows: K slices for parallelism)
        f1.bias = prm + f.bf1;
        f1.act = ACT_GELU; f1.dact_out = t.dgelu1; f1.ldm = FF;
        f1.Cb = t.G; f1.Cb2 = t.Glo; f1.ldcb = FF;
        TRY(gemm(f1, s));
        GemmDesc f2 = lin_fwd(M, t.G, t.Glo, FF, W + f.w2, Wl + f.w2, D);
        f2.Mdev = Mdev;
        f2.splits = cls ? 8 : split_rows(3 * FF); f2.ws = P->splitws;
        f2.bias = prm + f.bf2;
        f2.resid = t.Hf; f2.ldr = D;
        f2.Cf = t.u2; f2.ldcf = D;
        f2.defer_reduce = true;
        TRY(gemm(f2, s));
        hipLaunchKernelGGL(ln_fwd_kernel, lng, dim3(256), 0, s, deferred_rows(f2), t.u2, prm + f.g2, prm + f.b2, Mdev,
                           P->Xf[l + 1], P->Xb[l + 1], P->Xlo[l + 1], t.mean2, t.rstd2);
        FO_LAUNCHED();
    }

    // ---------------- head: pooler on the first token (row b of the last
    // layer's compact output), classifier, loss f_s
    const float* xcls = P->Xf[NL];
    TRY(launch_small_linear_fwd(xcls, prm + P->pool_w, prm + P->pool_b, P->pooled, B, D, D, true, s));
    TRY(launch_small_linear_fwd(P->pooled, prm + P->cls_w, prm + P->cls_b, m->logits, B, D, NC, false, s));
    TRY(launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, NC, s));

    // ---------------- backward (Alg. 4: backward pass of M_s)
    TRY(launch_small_linear_bwd(P->dz, P->pooled, prm + P->cls_w, P->pooled, grd + P->cls_w, grd + P->cls_b,
                                P->dpool, B, D, NC, P->slws, s));
    TRY(launch_small_linear_bwd(P->dpool, xcls, prm + P->pool_w, nullptr, grd + P->pool_w, grd + P->pool_b, P->dxc,
                                B, D, D, P->slws, s));

    // Weight gradients: the four products of layer l go to the side stream
    // together, after the main stream has issued layer l's input-gradient chain
    // (each weight-gradient product also applies the SGD update to its weight in
    // its epilogue, so it must follow the input-gradient product that reads that
    // weight).  They run while the main stream carries on with layer l - 1.  One
    // fork and one wait per layer: every cross-stream edge of a captured graph
    // costs several microseconds of idle GPU.  Layer l's operands sit in the
    // parity l % 2 buffers, which layer l - 2 reuses only after the side stream
    // has finished with them.
    hipStream_t s2 = P->side;
    const float lr = m->lr;
    float* prmw = m->params;
    bf16_t* w16 = m->w16;
    bf16_t* w16lo = m->w16lo;
    auto wgrad = [&](int M_, int N_, const bf16_t* A_, const bf16_t* B_, int64_t off, int K_, const int* Kdev_) {
        GemmDesc w;  // dW = A^T B over K_ rows -> grads; theta -= lr dW; bf16 parts
        w.M = M_; w.N = N_; w.K = K_; w.Kdev = Kdev_;
        w.amode = OP_KR; w.A = A_; w.lda = M_;
        w.bmode = OP_KR; w.B = B_; w.ldb = N_;
        w.Cf = grd + off; w.ldcf = N_;
        w.sgd_theta = prmw + off;
        w.sgd_hi = w16 + off;
        w.sgd_lo = w16lo + off;
        w.sgd_lr = lr;
        return w;
    };
    int cur = 0;
    SplitRows dy_rows;  // the LN2 backward's input: the deferred dX of the layer above
    for (int l = NL - 1; l >= 0; --l) {
        const LayerOff& f = P->off[l];
        LayerAct& t = P->a[l];
        const int pb = l & 1;
        bf16_t *du2b = P->du2b[pb], *dA1 = P->dA1[pb], *du1b = P->du1b[pb], *dqkv = P->dqkv[pb];
        if (l + 2 < NL) FO_HIP(hipStreamWaitEvent(s, P->ev_done[pb], 0));
        // the last layer runs on its B first-token rows (compact) down to the
        // attention, whose backward reaches every key and value row
        const bool cls = l == NL - 1;
        const int M = cls ? B : rows;
        const int* Mdev = cls ? Bdev : Tdev;
        if (cls) dy_rows = plain_rows(P->dxc, B);
        // LN2
        TRY(ln_bwd(dy_rows, t.u2, t.mean2, t.rstd2, prm + f.g2, Mdev, M, P->du2f, du2b, P->lnpart[pb][0], s));
        // FFN2: dG = du2 W2, times GELU' of the FFN1 pre-activation -> dA1; db1
        {
            GemmDesc d;
            d.M = M; d.N = FF; d.K = D; d.Mdev = Mdev;
            d.amode = OP_RK; d.A = du2b; d.lda = D;
            d.bmode = OP_KR; d.B = W + f.w2; d.ldb = FF;
            d.dact = t.dgelu1; d.ldm = FF;
            d.Cb = dA1; d.ldcb = FF;
            d.colpart = P->colwsF[pb];
            TRY(gemm(d, s));
        }
        SplitRows dh_rows;
        // FFN1: dH = du2 + dA1 W1
        {
            GemmDesc d;
            d.M = M; d.N = D; d.K = FF; d.Mdev = Mdev;
            d.amode = OP_RK; d.A = dA1; d.lda = FF;
            d.bmode = OP_KR; d.B = W + f.w1; d.ldb = D;
            d.resid = P->du2f; d.ldr = D;
            d.Cf = P->dHf; d.ldcf = D;
            d.splits = cls ? 8 : 2; d.ws = P->splitws;  // (two slices: half the partials for the LayerNorm to read)
            d.defer_reduce = true;  // summed by the LN1 backward
            TRY(gemm(d, s));
            dh_rows = deferred_rows(d);
        }
        // LN1
        TRY(ln_bwd(dh_rows, t.u1, t.mean1, t.rstd1, prm + f.g1, Mdev, M, P->du1f, du1b, P->lnpart[pb][1], s));
        // output projection: dO = du1 Wo
        {
            GemmDesc d;
            d.M = M; d.N = D; d.K = D; d.Mdev = Mdev;
            d.amode = OP_RK; d.A = du1b; d.lda = D;
            d.bmode = OP_KR; d.B = W + f.wo; d.ldb = D;
            d.Cb = P->dO; d.ldcb = D;  // (unsplit: faster than split-K plus its reduction here)
            if (cls) { d.splits = 4; d.ws = P->splitws; }  // (B rows: K slices for parallelism)
            TRY(gemm(d, s));
        }
        const float* du1_full = P->du1f;  // du1 over every row, the residual of dX
        if (cls) {
            TRY(launch_attn_cls_bwd(t.qkv, t.qkvlo, P->cu, t.O, t.Olo, P->dO, t.lse, dqkv, B, NH, D, s));
            // du1 is nonzero at the first tokens only
            TRY(launch_fill(P->dHf, (int64_t)rows * D, 0.f, s));
            hipLaunchKernelGGL(scatter_cls_kernel, dim3(B), dim3(256), 0, s, P->du1f, P->cu, B, P->dHf);
            FO_LAUNCHED();
            du1_full = P->dHf;
        } else {
            TRY(launch_attn_bwd(t.qkv, P->cu, t.O, P->dO, t.lse, dqkv, B, NH, D, s, P->cu + B + 2));
        }
        // input projection: dX = du1 + dqkv Wqkv (skipped for the first server layer), dbqkv
        if (l > 0) {
            GemmDesc d;
            d.M = rows; d.N = D; d.K = 3 * D; d.Mdev = Tdev;
            d.amode = OP_RK; d.A = dqkv; d.lda = 3 * D;
            d.bmode = OP_KR; d.B = W + f.wqkv; d.ldb = D;
            d.resid = du1_full; d.ldr = D;
            d.Cf = P->dY[cur ^ 1]; d.ldcf = D;
            d.splits = 2; d.ws = P->splitws;  // (as for FFN1)
            d.defer_reduce = true;  // summed by the next layer's LN2 backward
            TRY(gemm(d, s));
            dy_rows = deferred_rows(d);
        }
        // the layer's parameter gradients off the input-gradient chain: bias and
        // norm gradients from their partials, then the weight gradients with
        // their SGD updates.  After the first layer's chain the main stream has
        // nothing left but the final SGD pass, so it takes that layer's column
        // sums itself while the side stream runs the weight gradients.
        const bool last = l == 0;
        hipStream_t cs = last ? s : s2;
        float* colws = last ? P->colws2m : P->colws2;
        TRY(order_after(s2, s, P->ev_fork));
        TRY(launch_colsum_partial(dqkv, 3 * D, rows, Tdev, 3 * D, colws, cs));
        {
            // one launch finishes LN2's dgamma / dbeta / dbias of FFN2, the FFN1 bias,
            // LN1's dgamma / dbeta / dbias of the output projection and the QKV bias
            ColJobs cj;
            cj.n = 4;
            auto ln_job = [&](ColJob& J, const float* part, float* dg, float* db, float* dbias) {
                J.part = part; J.rows = M; J.rows_dev = Mdev; J.rows_per_part = LNB_ROWS; J.N = 3 * D;
                J.out.p[0] = dg; J.out.p[1] = db; J.out.p[2] = dbias; J.out.seg = D;
            };
            ln_job(cj.j[0], P->lnpart[pb][0], grd + f.g2, grd + f.b2, grd + f.bf2);
            ln_job(cj.j[1], P->lnpart[pb][1], grd + f.g1, grd + f.b1, grd + f.bo);
            ColJob& jf = cj.j[2];
            jf.part = P->colwsF[pb]; jf.rows = M; jf.rows_dev = Mdev; jf.rows_per_part = 128; jf.N = FF;
            jf.out.p[0] = grd + f.bf1; jf.out.seg = FF;
            ColJob& jq = cj.j[3];
            jq.part = colws; jq.rows = rows; jq.rows_dev = Tdev; jq.rows_per_part = colsum_rows_per_part();
            jq.N = 3 * D;
            jq.out.p[0] = grd + f.bqkv; jq.out.seg = 3 * D;
            TRY(launch_colsum_finish_multi(cj, cs));
            if (l == 1) FO_HIP(hipEventRecord(P->ev_cols, s2));
        }
        // the layer's four weight gradients in one launch, each tile over the
        // whole K (the packed rows, or the B first-token rows of the last layer)
        GemmDesc wg[4];
        const int Kw = cls ? B : rows;
        const int* Kwdev = cls ? nullptr : Tdev;
        wg[0] = wgrad(D, FF, du2b, t.G, f.w2, Kw, Kwdev);          // dW2 = du2^T G
        wg[1] = wgrad(FF, D, dA1, t.Hb, f.w1, Kw, Kwdev);          // dW1 = dA1^T H
        wg[2] = wgrad(D, D, du1b, t.O, f.wo, Kw, Kwdev);           // dWo = du1^T O
        wg[3] = wgrad(3 * D, D, dqkv, P->Xb[l], f.wqkv, rows, Tdev);  // dWqkv = dqkv^T X
        // (the last group has the GPU to itself: no cap on its workgroups)
        TRY(gemm_group(wg, 4, s2, last ? 0 : kWgradMaxWG));
        FO_HIP(hipEventRecord(P->ev_done[pb], s2));
        cur ^= 1;
    }
    FO_LAUNCHED();
    // ---------------- SGD (Alg. 4: theta_s <- theta_s - gamma_s grad) of the
    // parameters not updated by their weight-gradient product (biases, norms,
    // pooler, classifier; disjoint from the weight matrices the side stream is
    // still updating); refreshes the bf16 shadow.  It needs every layer's column
    // sums: the first layer's are on this stream, the others before ev_cols.
    static_assert(NL >= 2, "the column sums of the layers above the first finish on the side stream");
    FO_HIP(hipStreamWaitEvent(s, P->ev_cols, 0));
    TRY(launch_sgd_chunks(m->params, m->grads, m->w16, m->w16lo, P->sgd_chunks, P->n_sgd_chunks, m->lr, s));
    return order_after(s, s2, P->ev_join);
}

void destroy(fo_model* m) {
    Plan* P = (Plan*)m->plan;
    if (P) {
        for (hipEvent_t e : {P->ev_fork, P->ev_done[0], P->ev_done[1], P->ev_join, P->ev_cols})
            if (e) (void)hipEventDestroy(e);
        if (P->side) (void)hipStreamDestroy(P->side);
    }
    delete P;
    m->plan = nullptr;
}

}  // namespace

int64_t bert_param_count() { return kParams; }

const Family* family_bert() {
    static const Family f = {(int64_t)L * D * 2, ws_bytes, init, step, destroy};
    return &f;
}

}  // namespace fo
