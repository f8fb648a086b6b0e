// Configs 7 and 8: the server part of the paper's Transformer-6 and
// Transformer-12 (Table 4) split after their embedding, one training
// iteration of the activation branch of Alg. 4 in fp32:
//   for each encoder layer (d = 100, FFN 100, post-norm):
//     qkv = x Wqkv^T + b;  O = softmax(q k^T / sqrt(dh), keys >= length masked) v per head;
//     h = LN1(x + O Wo^T + bo);  y = LN2(h + ReLU(h W1^T + b1) W2^T + b2)
//   z = y[:, 0] Wc^T + bc (the first token), mean cross-entropy, backward, SGD.
// Transformer-6 has 5 heads of width 20 on 64-token batches, Transformer-12
// 50 heads of width 2 on 256-token batches.
//
// The model is small (d = 100): the products run as LDS-tiled fp32 FMA
// (64 x 64 output tiles, a deterministic split over K for the long weight-
// gradient reductions), attention as one thread per query (forward, and the
// dQ phase of the backward) or per key (the dK, dV phase) over K, V or Q, dO
// staged in LDS, LayerNorm as one wave per row.  Batches stay padded
// [B][L][d]; queries past a sequence's length are computed like the others
// (nothing reads them, so their gradients are zero) and keys past it are masked.
#include "gemm.h"
#include "model.h"

namespace fo {

namespace {

constexpr int D = 100, FF = 100, NCLS = 2;
constexpr float LN_EPS = 1e-5f;

struct Arch {
    int layers, heads, L;
};
Arch arch_of(int cid) { return cid == 7 ? Arch{6, 5, 64} : Arch{12, 50, 256}; }

inline int nblk(int64_t n) { return (int)cdiv(n, 256); }

using Gf = GemmF32;

// ------------------------------------------------------------------ attention
// Lengths as the kernels use them: clamped to [1, L]; the number of lengths
// outside that range goes to *bad (the model's error flag).
__global__ void lengths_check(const StepIn* __restrict__ in, int B, int L, float* __restrict__ bad) {
    int n = 0;
    for (int b = threadIdx.x; b < B; b += blockDim.x) n += in->lengths[b] < 1 || in->lengths[b] > L;
    for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o);
    if (threadIdx.x == 0) *bad = (float)n;
}
__device__ __forceinline__ int seq_len(const StepIn* in, int b, int L) { return min(max(in->lengths[b], 1), L); }

// One workgroup per (sequence, head); thread i is query i.  Keys and values of
// the head in LDS; an online softmax over the valid keys (running maximum,
// rescaled sum and output), then O and lse = max + log(sum).
template <int DH>
__global__ void __launch_bounds__(256) attn_small_fwd(const float* __restrict__ qkv, const StepIn* __restrict__ in,
                                                      float* __restrict__ O, float* __restrict__ lse, int H, int L,
                                                      float scale) {
    extern __shared__ float sm[];
    float* Ks = sm;
    float* Vs = sm + L * DH;
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int len = seq_len(in, b, L);
    const int64_t row0 = (int64_t)b * L, ld = 3 * D;
    for (int e = threadIdx.x; e < len * DH; e += blockDim.x) {
        const int j = e / DH, c = e % DH;
        Ks[e] = qkv[(row0 + j) * ld + D + h * DH + c];
        Vs[e] = qkv[(row0 + j) * ld + 2 * D + h * DH + c];
    }
    __syncthreads();
    const int i = threadIdx.x;
    if (i >= L) return;
    float q[DH], acc[DH];
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        q[c] = qkv[(row0 + i) * ld + h * DH + c] * scale;
        acc[c] = 0.f;
    }
    float mx = -INFINITY, sum = 0.f;
    for (int j = 0; j < len; ++j) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < DH; ++c) s = fmaf(q[c], Ks[j * DH + c], s);
        const float mn = fmaxf(mx, s);
        // the hardware exponential (v_exp_f32 on x log2 e): its error on these
        // arguments (<= 0 after the running-max shift) is far below the fp32 path's
        const float f = __expf(mx - mn), p = __expf(s - mn);  // exp(-inf) = 0 on the first key
        sum = sum * f + p;
#pragma unroll
        for (int c = 0; c < DH; ++c) acc[c] = fmaf(acc[c], f, p * Vs[j * DH + c]);
        mx = mn;
    }
    const float inv = 1.f / sum;
#pragma unroll
    for (int c = 0; c < DH; ++c) O[(row0 + i) * D + h * DH + c] = acc[c] * inv;
    lse[(int64_t)blockIdx.x * L + i] = mx + logf(sum);
}

// Backward, with P = softmax(S), D_i = dO_i . O_i, dS_ij = P_ij (dO_i . V_j - D_i):
// phase 1, thread = query i: dQ_i = scale sum_j dS_ij K_j (K, V in LDS);
// phase 2, thread = key j: dK_j = scale sum_i dS_ij Q_i, dV_j = sum_i P_ij dO_i
// over every query (Q, dO, lse, D in LDS).  Keys past the length get zero.
template <int DH>
__global__ void __launch_bounds__(256) attn_small_bwd(const float* __restrict__ qkv, const StepIn* __restrict__ in,
                                                      const float* __restrict__ O, const float* __restrict__ dO,
                                                      const float* __restrict__ lse, float* __restrict__ dqkv, int H,
                                                      int L, float scale) {
    extern __shared__ float sm[];
    float* T0 = sm;                // K, then Q
    float* T1 = sm + L * DH;       // V, then dO
    float* Ls = sm + 2 * L * DH;   // lse
    float* Ds = Ls + L;            // D
    const int b = blockIdx.x / H, h = blockIdx.x % H;
    const int len = seq_len(in, b, L);
    const int64_t row0 = (int64_t)b * L, ld = 3 * D;
    const int t = threadIdx.x;
    for (int e = t; e < len * DH; e += blockDim.x) {
        const int j = e / DH, c = e % DH;
        T0[e] = qkv[(row0 + j) * ld + D + h * DH + c];
        T1[e] = qkv[(row0 + j) * ld + 2 * D + h * DH + c];
    }
    float dsum = 0.f, li = 0.f;
    float q[DH], g[DH];
    if (t < L) {
#pragma unroll
        for (int c = 0; c < DH; ++c) {
            q[c] = qkv[(row0 + t) * ld + h * DH + c];
            g[c] = dO[(row0 + t) * D + h * DH + c];
            dsum = fmaf(g[c], O[(row0 + t) * D + h * DH + c], dsum);
        }
        li = lse[(int64_t)blockIdx.x * L + t];
    }
    __syncthreads();
    if (t < L) {
        float dq[DH];
#pragma unroll
        for (int c = 0; c < DH; ++c) dq[c] = 0.f;
        for (int j = 0; j < len; ++j) {
            float s = 0.f, dp = 0.f;
#pragma unroll
            for (int c = 0; c < DH; ++c) {
                s = fmaf(q[c], T0[j * DH + c], s);
                dp = fmaf(g[c], T1[j * DH + c], dp);
            }
            const float p = __expf(s * scale - li), ds = p * (dp - dsum);
#pragma unroll
            for (int c = 0; c < DH; ++c) dq[c] = fmaf(ds, T0[j * DH + c], dq[c]);
        }
#pragma unroll
        for (int c = 0; c < DH; ++c) dqkv[(row0 + t) * ld + h * DH + c] = dq[c] * scale;
    }
    __syncthreads();  // phase 2 overwrites K, V with Q, dO
    if (t < L) {
#pragma unroll
        for (int c = 0; c < DH; ++c) {
            T0[t * DH + c] = q[c];
            T1[t * DH + c] = g[c];
        }
        Ls[t] = li;
        Ds[t] = dsum;
    }
    __syncthreads();
    if (t >= L) return;
    float kj[DH], vj[DH], dk[DH], dv[DH];
    const bool valid = t < len;
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        kj[c] = valid ? qkv[(row0 + t) * ld + D + h * DH + c] : 0.f;
        vj[c] = valid ? qkv[(row0 + t) * ld + 2 * D + h * DH + c] : 0.f;
        dk[c] = dv[c] = 0.f;
    }
    if (valid)
        for (int i = 0; i < L; ++i) {
            float s = 0.f, dp = 0.f;
#pragma unroll
            for (int c = 0; c < DH; ++c) {
                s = fmaf(T0[i * DH + c], kj[c], s);
                dp = fmaf(T1[i * DH + c], vj[c], dp);
            }
            const float p = __expf(s * scale - Ls[i]), ds = p * (dp - Ds[i]);
#pragma unroll
            for (int c = 0; c < DH; ++c) {
                dk[c] = fmaf(ds, T0[i * DH + c], dk[c]);
                dv[c] = fmaf(p, T1[i * DH + c], dv[c]);
            }
        }
#pragma unroll
    for (int c = 0; c < DH; ++c) {
        dqkv[(row0 + t) * ld + D + h * DH + c] = dk[c] * scale;
        dqkv[(row0 + t) * ld + 2 * D + h * DH + c] = dv[c];
    }
}

// ------------------------------------------------------------------ LayerNorm (d = 100, one wave per row)
__global__ void __launch_bounds__(256) ln_small_fwd(const float* __restrict__ u, const float* __restrict__ gam,
                                                    const float* __restrict__ bet, float* __restrict__ y,
                                                    float* __restrict__ xhat, float* __restrict__ rstd, int rows) {
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6), l = threadIdx.x & 63;
    if (r >= rows) return;
    const float* x = u + (int64_t)r * D;
    const float a = x[l], c = l + 64 < D ? x[l + 64] : 0.f;
    float s = a + c;
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    const float mu = s / D, da = a - mu, dc = l + 64 < D ? c - mu : 0.f;
    float v = da * da + dc * dc;
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    const float rs = 1.f / sqrtf(v / D + LN_EPS);
    const int64_t o0 = (int64_t)r * D;
    xhat[o0 + l] = da * rs;
    y[o0 + l] = da * rs * gam[l] + bet[l];
    if (l + 64 < D) {
        xhat[o0 + l + 64] = dc * rs;
        y[o0 + l + 64] = dc * rs * gam[l + 64] + bet[l + 64];
    }
    if (l == 0) rstd[r] = rs;
}

// dx = rstd (dy g - mean(dy g) - xhat mean(dy g xhat)) (+ add); also dy * xhat
// into gx for the scale gradient's column sums.
__global__ void __launch_bounds__(256) ln_small_bwd(const float* __restrict__ dy, const float* __restrict__ xhat,
                                                    const float* __restrict__ rstd, const float* __restrict__ gam,
                                                    float* __restrict__ dx, float* __restrict__ gx, int rows) {
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6), l = threadIdx.x & 63;
    if (r >= rows) return;
    const int64_t o0 = (int64_t)r * D;
    const bool two = l + 64 < D;
    const float ya = dy[o0 + l], yc = two ? dy[o0 + l + 64] : 0.f;
    const float xa = xhat[o0 + l], xc = two ? xhat[o0 + l + 64] : 0.f;
    const float ga = ya * gam[l], gc = two ? yc * gam[l + 64] : 0.f;
    float s1 = ga + gc, s2 = ga * xa + gc * xc;
    for (int o = 32; o > 0; o >>= 1) {
        s1 += __shfl_xor(s1, o);
        s2 += __shfl_xor(s2, o);
    }
    s1 /= D;
    s2 /= D;
    const float rs = rstd[r];
    dx[o0 + l] = rs * (ga - s1 - xa * s2);
    gx[o0 + l] = ya * xa;
    if (two) {
        dx[o0 + l + 64] = rs * (gc - s1 - xc * s2);
        gx[o0 + l + 64] = yc * xc;
    }
}

// ------------------------------------------------------------------ plan
struct LayerP {
    const float *wqkv, *bqkv, *wo, *bo, *g1, *b1n, *w1, *b1, *w2, *b2, *g2, *b2n;
    float *gwqkv, *gbqkv, *gwo, *gbo, *gg1, *gb1n, *gw1, *gb1, *gw2, *gb2, *gg2, *gb2n;
    // saved activations
    float *qkv, *O, *lse, *xh1, *rs1, *h1, *f, *xh2, *rs2, *y;
};

struct Plan {
    Arch a;
    LayerP* ly;        // [layers] (host array)
    const float *wc, *bc;
    float *gwc, *gbc;
    float *dz, *dy, *du2, *df, *dh1, *du1, *dO, *dqkv, *dx, *gx, *gx1;
    float* part;       // split-K slices
    float* colws;      // column-sum workspace
    float* sumws;      // partial rows of a layer's kLayerSums column sums
    float* wgpart;     // the weight gradients' K slices of every layer (layer_wgrad_part each)
    size_t part_floats;
};

constexpr int kMaxSlices = 16;
// column sums per layer in the backward: the biases of the four products and
// the two norms' gain and shift
constexpr int kLayerSums = 8;

// K slices of a weight gradient (K = the R packed rows)
int wgrad_slices(int64_t R) { return (int)std::min<int64_t>(kMaxSlices, std::max<int64_t>(1, R / 256)); }
// Floats of a layer's weight-gradient slices (its four products, each rounded
// up to 64 floats), kept until the step sums them all before the update.
size_t layer_wgrad_part(int64_t R) {
    const int S = wgrad_slices(R);
    if (S <= 1) return 0;
    auto r64 = [](size_t n) { return (n + 63) / 64 * 64; };
    return r64((size_t)S * D * FF) + r64((size_t)S * FF * D) + r64((size_t)S * D * D) + r64((size_t)S * 3 * D * D);
}

size_t ws_bytes(const fo_model* m) {
    const Arch a = arch_of(m->cid);
    const size_t R = (size_t)m->max_batch * a.L, Bm = m->max_batch;
    size_t s = 0;
    auto add = [&](size_t b) { s += (b + 255) & ~size_t(255); };
    add(sizeof(Plan));
    for (int l = 0; l < a.layers; ++l) {
        add(4 * R * 3 * D);              // qkv
        add(4 * R * D);                  // O
        add(4 * Bm * a.heads * a.L);     // lse
        add(4 * R * D);                  // xh1
        add(4 * R);                      // rs1
        add(4 * R * D);                  // h1
        add(4 * R * FF);                 // f
        add(4 * R * D);                  // xh2
        add(4 * R);                      // rs2
        add(4 * R * D);                  // y
    }
    add(4 * Bm * NCLS);                                               // dz
    for (int i = 0; i < 8; ++i) add(4 * R * 3 * D);                   // dy, du2, df, dh1, du1, dO, dqkv, dx (+gx)
    add(4 * R * D);                                                   // gx
    add(4 * R * D);                                                   // gx1
    add(4 * (size_t)kMaxSlices * 3 * D * D);                          // part
    add(4 * colsum_ws_floats((int)R, 3 * D));                         // colws
    add(4 * kLayerSums * colsum_ws_floats((int)R, 3 * D));            // sumws
    add(4 * a.layers * layer_wgrad_part((int64_t)R));                 // wgpart
    return s;
}

fo_status init(fo_model* m) {
    Plan* P = new (std::nothrow) Plan();
    if (!P) return FO_ENOMEM;
    m->plan = P;
    P->a = arch_of(m->cid);
    P->ly = new (std::nothrow) LayerP[P->a.layers];
    if (!P->ly) return FO_ENOMEM;
    const size_t R = (size_t)m->max_batch * P->a.L, Bm = m->max_batch;
    const float* p = m->params;
    float* g = m->grads;
    auto take = [&](const float*& w, float*& gw, size_t n) {
        w = p;
        gw = g;
        p += n;
        g += n;
    };
    Arena& ar = m->arena;
    ar.take<char>(sizeof(Plan));
    for (int l = 0; l < P->a.layers; ++l) {
        LayerP& L = P->ly[l];
        take(L.wqkv, L.gwqkv, 3 * D * D);
        take(L.bqkv, L.gbqkv, 3 * D);
        take(L.wo, L.gwo, D * D);
        take(L.bo, L.gbo, D);
        take(L.g1, L.gg1, D);
        take(L.b1n, L.gb1n, D);
        take(L.w1, L.gw1, FF * D);
        take(L.b1, L.gb1, FF);
        take(L.w2, L.gw2, D * FF);
        take(L.b2, L.gb2, D);
        take(L.g2, L.gg2, D);
        take(L.b2n, L.gb2n, D);
        L.qkv = ar.take<float>(R * 3 * D);
        L.O = ar.take<float>(R * D);
        L.lse = ar.take<float>(Bm * P->a.heads * P->a.L);
        L.xh1 = ar.take<float>(R * D);
        L.rs1 = ar.take<float>(R);
        L.h1 = ar.take<float>(R * D);
        L.f = ar.take<float>(R * FF);
        L.xh2 = ar.take<float>(R * D);
        L.rs2 = ar.take<float>(R);
        L.y = ar.take<float>(R * D);
    }
    take(P->wc, P->gwc, NCLS * D);
    take(P->bc, P->gbc, NCLS);
    P->dz = ar.take<float>(Bm * NCLS);
    float** bufs[8] = {&P->dy, &P->du2, &P->df, &P->dh1, &P->du1, &P->dO, &P->dqkv, &P->dx};
    for (float** b : bufs) *b = ar.take<float>(R * 3 * D);
    P->gx = ar.take<float>(R * D);
    P->gx1 = ar.take<float>(R * D);
    P->part_floats = (size_t)kMaxSlices * 3 * D * D;
    P->part = ar.take<float>(P->part_floats);
    P->colws = ar.take<float>(colsum_ws_floats((int)R, 3 * D));
    P->sumws = ar.take<float>(kLayerSums * colsum_ws_floats((int)R, 3 * D));
    P->wgpart = ar.take<float>(std::max<size_t>(1, P->a.layers * layer_wgrad_part((int64_t)R)));
    if (!P->wgpart) {
        set_error("tfsmall: workspace arena too small");
        return FO_ENOMEM;
    }
    return FO_OK;
}

struct Ctx {
    hipStream_t s;
    Plan* P;
};

// C = epi(sum_k A(m, k) B(n, k)) (see GemmF32); S slices over K for long reductions.
fo_status gemm(const Ctx& c, const Gf& g) { return launch_gemm_f32(g, c.P->part, c.P->part_floats, c.s); }

Gf prod(const float* A, int64_t am, int64_t ak, const float* B, int64_t bn, int64_t bk, float* C, int64_t ldc, int M,
        int N, int K) {
    Gf g{};
    g.A = A;
    g.am = am;
    g.ak = ak;
    g.B = B;
    g.bn = bn;
    g.bk = bk;
    g.C = C;
    g.ldc = ldc;
    g.M = M;
    g.N = N;
    g.K = K;
    g.S = 1;
    return g;
}

// y[r][n] = x[r][:] . W[n][:] + b[n] (+ add[r][n], ReLU), W [N][K]
Gf linear(const float* x, const StepIn* inx, const float* W, const float* b, float* y, int R, int N, int K) {
    Gf g = prod(x, K, 1, W, K, 1, y, N, R, N, K);
    g.inA = inx;
    g.bias = b;
    return g;
}
// dx[r][k] = dy[r][:] . W[:][k] (+ add), W [N][K]
Gf linear_dx(const float* dy, const float* W, float* dx, int R, int N, int K) {
    return prod(dy, N, 1, W, 1, K, dx, K, R, K, N);
}
// dW[n][k] = sum_r dy[r][n] x[r][k] (x = the batch when inx is set).  Nothing
// reads dW before the update, so its K slices stay at *part (which advances)
// and join `sums`, added up for every layer in one launch at the end of the
// backward instead of one reduction launch per product.
fo_status linear_dw(const Ctx& c, const float* dy, const float* x, const StepIn* inx, float* dW, int R, int N, int K,
                    SplitJobs& sums, float*& part) {
    Gf g = prod(dy, 1, N, x, 1, K, dW, K, N, K, R);
    g.inB = inx;
    g.S = wgrad_slices(R);
    if (g.S <= 1) return gemm(c, g);
    FO_CHECK(sums.n < kSplitJobsMax, "tfsmall: more than %d deferred weight-gradient sums", kSplitJobsMax);
    g.defer = 1;
    const size_t n = (size_t)g.S * N * K;
    SplitJob& j = sums.j[sums.n++];
    j.ws = part; j.C = dW; j.ldc = K; j.S = g.S; j.M = N; j.N = K;
    const fo_status st = launch_gemm_f32(g, part, n, c.s);
    part += (n + 63) / 64 * 64;
    return st;
}
fo_status colsum(const Ctx& c, const float* X, int R, int N, float* out) {
    return launch_colsum(X, N, R, nullptr, N, out, c.P->colws, c.s);
}

fo_status step(fo_model* m, const fo_acts* acts, const int32_t* labels) {
    (void)labels;  // read through m->dev_in
    Plan* P = (Plan*)m->plan;
    const Arch a = P->a;
    const int B = acts->batch, L = a.L, R = B * L, H = a.heads, dh = D / H;
    const float scale = 1.f / sqrtf((float)dh);
    const Ctx c{m->stream, P};
    hipStream_t s = m->stream;
    fo_status st = FO_OK;
#define TRY(x)                   \
    do {                         \
        st = (x);                \
        if (st != FO_OK) return st; \
    } while (0)
    hipLaunchKernelGGL(lengths_check, dim3(1), dim3(64), 0, s, m->dev_in, B, L, m->loss + 2);
    FO_LAUNCHED();
    const size_t fwd_lds = sizeof(float) * 2 * L * dh, bwd_lds = sizeof(float) * (2 * L * dh + 2 * L);
    // forward (Alg. 4: forward pass of M_s)
    for (int l = 0; l < a.layers; ++l) {
        LayerP& Y = P->ly[l];
        const float* x = l ? P->ly[l - 1].y : nullptr;
        const StepIn* inx = l ? nullptr : m->dev_in;
        TRY(gemm(c, linear(x, inx, Y.wqkv, Y.bqkv, Y.qkv, R, 3 * D, D)));
        if (dh == 20)
            hipLaunchKernelGGL(attn_small_fwd<20>, dim3(B * H), dim3(256), fwd_lds, s, Y.qkv, m->dev_in, Y.O, Y.lse,
                               H, L, scale);
        else
            hipLaunchKernelGGL(attn_small_fwd<2>, dim3(B * H), dim3(256), fwd_lds, s, Y.qkv, m->dev_in, Y.O, Y.lse,
                               H, L, scale);
        FO_LAUNCHED();
        Gf go = linear(Y.O, nullptr, Y.wo, Y.bo, P->dx, R, D, D);  // u1 = x + O Wo^T + bo (into dx as scratch)
        go.add = x;
        go.inAdd = inx;
        go.ldadd = D;
        TRY(gemm(c, go));
        hipLaunchKernelGGL(ln_small_fwd, dim3((int)cdiv(R, 4)), dim3(256), 0, s, P->dx, Y.g1, Y.b1n, Y.h1, Y.xh1, Y.rs1,
                           R);
        FO_LAUNCHED();
        Gf g1 = linear(Y.h1, nullptr, Y.w1, Y.b1, Y.f, R, FF, D);
        g1.relu = 1;
        TRY(gemm(c, g1));
        Gf g2 = linear(Y.f, nullptr, Y.w2, Y.b2, P->dx, R, D, FF);  // u2 = h1 + f W2^T + b2
        g2.add = Y.h1;
        g2.ldadd = D;
        TRY(gemm(c, g2));
        hipLaunchKernelGGL(ln_small_fwd, dim3((int)cdiv(R, 4)), dim3(256), 0, s, P->dx, Y.g2, Y.b2n, Y.y, Y.xh2, Y.rs2,
                           R);
        FO_LAUNCHED();
    }
    // classifier on the first token, loss f_s (Eq. 5)
    const float* ytop = P->ly[a.layers - 1].y;
    Gf gz = prod(ytop, (int64_t)L * D, 1, P->wc, D, 1, m->logits, NCLS, B, NCLS, D);  // rows b at token 0
    gz.bias = P->bc;
    TRY(gemm(c, gz));
    TRY(launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, NCLS, s));
    // backward (Alg. 4: backward pass of M_s)
    float* dy = P->dy;  // gradient of the current layer's output
    float* dx = P->dx;  // gradient of its input
    // dWc[c][k] = sum_b dz[b][c] y[b, 0, k]; dy[b, 0, :] = dz[b] Wc, zero elsewhere
    TRY(gemm(c, prod(P->dz, 1, NCLS, ytop, 1, (int64_t)L * D, P->gwc, D, NCLS, D, B)));
    TRY(colsum(c, P->dz, B, NCLS, P->gbc));
    TRY(launch_fill(dy, (int64_t)R * D, 0.f, s));
    TRY(gemm(c, prod(P->dz, NCLS, 1, P->wc, 1, D, dy, (int64_t)L * D, B, D, NCLS)));
    SplitJobs wsums;
    float* wpart = P->wgpart;
    for (int l = a.layers - 1; l >= 0; --l) {
        LayerP& Y = P->ly[l];
        const float* x = l ? P->ly[l - 1].y : nullptr;
        const StepIn* inx = l ? nullptr : m->dev_in;
        // LN2
        hipLaunchKernelGGL(ln_small_bwd, dim3((int)cdiv(R, 4)), dim3(256), 0, s, dy, Y.xh2, Y.rs2, Y.g2, P->du2,
                           P->gx, R);
        FO_LAUNCHED();
        // The layer's eight column sums (biases, norm gains and shifts) run as
        // one pass at the end of the layer, over buffers that stay intact until then.
        ColSums sums;
        const size_t sw = colsum_ws_floats(R, 3 * D);
        auto sum = [&](const float* X, int N, float* out) {
            sums.add(X, N, R, N, P->sumws + sums.parts.n * sw, out);
        };
        sum(P->gx, D, Y.gg2);
        sum(dy, D, Y.gb2n);
        // FFN2 and FFN1 (ReLU mask from the stored activation)
        TRY(linear_dw(c, P->du2, Y.f, nullptr, Y.gw2, R, D, FF, wsums, wpart));
        sum(P->du2, D, Y.gb2);
        Gf gdf = linear_dx(P->du2, Y.w2, P->df, R, D, FF);
        gdf.mask = Y.f;
        gdf.ldmask = FF;
        TRY(gemm(c, gdf));
        TRY(linear_dw(c, P->df, Y.h1, nullptr, Y.gw1, R, FF, D, wsums, wpart));
        sum(P->df, FF, Y.gb1);
        Gf gdh = linear_dx(P->df, Y.w1, P->dh1, R, FF, D);  // dh1 = du2 + df W1
        gdh.add = P->du2;
        gdh.ldadd = D;
        TRY(gemm(c, gdh));
        // LN1
        hipLaunchKernelGGL(ln_small_bwd, dim3((int)cdiv(R, 4)), dim3(256), 0, s, P->dh1, Y.xh1, Y.rs1, Y.g1, P->du1,
                           P->gx1, R);
        FO_LAUNCHED();
        sum(P->gx1, D, Y.gg1);
        sum(P->dh1, D, Y.gb1n);
        // output projection
        TRY(linear_dw(c, P->du1, Y.O, nullptr, Y.gwo, R, D, D, wsums, wpart));
        sum(P->du1, D, Y.gbo);
        TRY(gemm(c, linear_dx(P->du1, Y.wo, P->dO, R, D, D)));
        // attention
        if (dh == 20)
            hipLaunchKernelGGL(attn_small_bwd<20>, dim3(B * H), dim3(256), bwd_lds, s, Y.qkv, m->dev_in, Y.O, P->dO,
                               Y.lse, P->dqkv, H, L, scale);
        else
            hipLaunchKernelGGL(attn_small_bwd<2>, dim3(B * H), dim3(256), bwd_lds, s, Y.qkv, m->dev_in, Y.O, P->dO,
                               Y.lse, P->dqkv, H, L, scale);
        FO_LAUNCHED();
        // QKV projection (no input gradient for the first server layer: nothing is sent back)
        TRY(linear_dw(c, P->dqkv, x, inx, Y.gwqkv, R, 3 * D, D, wsums, wpart));
        sum(P->dqkv, 3 * D, Y.gbqkv);
        TRY(launch_colsums(sums, s));
        if (l > 0) {
            Gf gx = linear_dx(P->dqkv, Y.wqkv, dx, R, 3 * D, D);  // dx = du1 + dqkv Wqkv
            gx.add = P->du1;
            gx.ldadd = D;
            TRY(gemm(c, gx));
            std::swap(dy, dx);
        }
    }
    if (wsums.n) TRY(launch_splitk_sum_multi(wsums, s));
#undef TRY
    // SGD (Alg. 4)
    return launch_sgd(m->params, m->grads, nullptr, nullptr, nullptr, m->n_params, m->lr, 0.f, s);
}

void destroy(fo_model* m) {
    Plan* P = (Plan*)m->plan;
    if (P) delete[] P->ly;
    delete P;
    m->plan = nullptr;
}

}  // namespace

int64_t tfsmall_param_count(int32_t cid) {
    const Arch a = arch_of(cid);
    const int64_t per = 3LL * D * D + 3 * D + (int64_t)D * D + D + 2 * D + (int64_t)FF * D + FF + (int64_t)D * FF + D +
                        2 * D;
    return a.layers * per + (int64_t)NCLS * D + NCLS;
}

const Family* family_tfsmall7() {
    static const Family f = {(int64_t)64 * D * 4, ws_bytes, init, step, destroy};
    return &f;
}
const Family* family_tfsmall8() {
    static const Family f = {(int64_t)256 * D * 4, ws_bytes, init, step, destroy};
    return &f;
}

}  // namespace fo
