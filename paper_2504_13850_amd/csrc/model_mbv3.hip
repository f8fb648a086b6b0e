// Config 10: the server part of the paper's MobileNetV3-Large (Table 4) split
// after its seventh bottleneck, one training iteration of the activation
// branch of Alg. 4 in fp32 on [80, 4, 4] inputs (NCHW at the boundary):
//   eight bottlenecks: expansion 1x1 conv + BN + hard-swish, depthwise k x k
//   conv (stride 1 or 2) + BN + hard-swish, squeeze-excitation on four (global
//   mean, fc + ReLU, fc + hard-sigmoid, channel scale), projection 1x1 conv +
//   BN, plus the input when the shape is kept;
//   1x1 conv to 960 + BN + hard-swish, global mean, fc 1280 + hard-swish,
//   fc 200; mean cross-entropy, backward, SGD.
// Activations are NHWC rows [B*H*W][C]; the 1x1 convolutions and the fc layers
// run on the fp32 product kernel, batch norm is one workgroup per channel
// (batch statistics, with the activation and the residual fused), the
// depthwise convolution one thread per output (forward) or input (input
// gradient) and one workgroup per channel for its weight gradient.
#include "gemm.h"
#include "model.h"

namespace fo {

namespace {

constexpr int CIN = 80, HIN = 4, CLAST = 960, F1 = 1280, NCLS = 200, NBLK = 8;
constexpr float BN_EPS = 1e-5f;
constexpr int kMaxSlices = 16;

struct Blk {
    int k, e, co, se, stride;
};
constexpr Blk kBlk[NBLK] = {{3, 200, 80, 0, 1}, {3, 184, 80, 0, 1}, {3, 184, 80, 0, 1}, {3, 480, 112, 1, 1},
                            {3, 672, 112, 1, 1}, {5, 672, 160, 1, 2}, {5, 960, 160, 1, 1}, {5, 960, 160, 1, 1}};
// squeeze width: e / 4 to a multiple of 8, at least 8, not below 90% of e / 4
constexpr int se_width(int e) {
    return (e / 4 + 4) / 8 * 8 < 8 ? 8
           : ((e / 4 + 4) / 8 * 8 < 0.9 * (e / 4) ? (e / 4 + 4) / 8 * 8 + 8 : (e / 4 + 4) / 8 * 8);
}

inline int nblk(int64_t n) { return (int)cdiv(n, 256); }

__device__ __forceinline__ float hswish(float x) { return x * fminf(fmaxf(x + 3.f, 0.f), 6.f) * (1.f / 6.f); }
__device__ __forceinline__ float hswish_d(float x) { return x < -3.f ? 0.f : (x > 3.f ? 1.f : (2.f * x + 3.f) / 6.f); }
__device__ __forceinline__ float hsig(float x) { return fminf(fmaxf(x + 3.f, 0.f), 6.f) * (1.f / 6.f); }
__device__ __forceinline__ float hsig_d(float x) { return x > -3.f && x < 3.f ? 1.f / 6.f : 0.f; }

// [B][C][HW] (the batch) -> rows [B*HW][C]
__global__ void __launch_bounds__(256) nchw_rows(const StepIn* __restrict__ in, float* __restrict__ y, int B, int C,
                                                 int HW) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)B * C * HW) return;
    const int c = (int)(i % C);
    const int64_t r = i / C;
    const int b = (int)(r / HW), p = (int)(r % HW);
    y[i] = ((const float*)in->x)[((int64_t)b * C + c) * HW + p];
}

// rows a BatchNorm thread keeps in registers (up to 256 x BN_REG_ROWS rows per
// channel read once; more rows take the three-pass loops)
constexpr int BN_REG_ROWS = 8;

__device__ __forceinline__ float block_sum(float v, float* red) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    return red[0] + red[1] + red[2] + red[3];
}

// Block c: batch statistics of column c of z [R][C] (two passes), xhat, then
// y = act(gamma xhat + beta) (+ add), act 0 = none, 1 = hard-swish
__global__ void __launch_bounds__(256) bn_rows_fwd(const float* __restrict__ z, const float* __restrict__ gam,
                                                   const float* __restrict__ bet, float* __restrict__ xhat,
                                                   float* __restrict__ y, float* __restrict__ rstd_out,
                                                   const float* __restrict__ add, int R, int C, int act) {
    __shared__ float red[4];
    const int c = blockIdx.x;
    if (R <= 256 * BN_REG_ROWS) {
        // the thread's rows (r = t + 256 i, i < n) read once, kept in registers
        // for the mean, the variance and the output
        const int n = (R + 255) / 256;
        float zv[BN_REG_ROWS];
#pragma unroll
        for (int i = 0; i < BN_REG_ROWS; ++i)
            if (i < n) zv[i] = z[(int64_t)min((int)threadIdx.x + 256 * i, R - 1) * C + c];
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < BN_REG_ROWS; ++i)
            if (i < n && threadIdx.x + 256 * i < R) s += zv[i];
        const float mu = block_sum(s, red) / R;
        float v = 0.f;
#pragma unroll
        for (int i = 0; i < BN_REG_ROWS; ++i)
            if (i < n && threadIdx.x + 256 * i < R) {
                const float d = zv[i] - mu;
                v = fmaf(d, d, v);
            }
        const float rs = 1.f / sqrtf(block_sum(v, red) / R + BN_EPS);
        const float gc = gam[c], bc = bet[c];
#pragma unroll
        for (int i = 0; i < BN_REG_ROWS; ++i) {
            const int r = threadIdx.x + 256 * i;
            if (i < n && r < R) {
                const int64_t o = (int64_t)r * C + c;
                const float xh = (zv[i] - mu) * rs;
                const float u = fmaf(gc, xh, bc);
                xhat[o] = xh;
                y[o] = (act ? hswish(u) : u) + (add ? add[o] : 0.f);
            }
        }
        if (threadIdx.x == 0) rstd_out[c] = rs;
        return;
    }
    float s = 0.f;
    for (int r = threadIdx.x; r < R; r += 256) s += z[(int64_t)r * C + c];
    const float mu = block_sum(s, red) / R;
    float v = 0.f;
    for (int r = threadIdx.x; r < R; r += 256) {
        const float d = z[(int64_t)r * C + c] - mu;
        v = fmaf(d, d, v);
    }
    const float rs = 1.f / sqrtf(block_sum(v, red) / R + BN_EPS);
    for (int r = threadIdx.x; r < R; r += 256) {
        const int64_t o = (int64_t)r * C + c;
        const float xh = (z[o] - mu) * rs;
        const float u = fmaf(gam[c], xh, bet[c]);
        xhat[o] = xh;
        y[o] = (act ? hswish(u) : u) + (add ? add[o] : 0.f);
    }
    if (threadIdx.x == 0) rstd_out[c] = rs;
}

// Block c: du = dy act'(gamma xhat + beta); dgamma = sum du xhat, dbeta = sum du,
// dz = gamma rstd (du - dbeta / R - xhat dgamma / R)
__global__ void __launch_bounds__(256) bn_rows_bwd(const float* __restrict__ dy, const float* __restrict__ xhat,
                                                   const float* __restrict__ gam, const float* __restrict__ bet,
                                                   const float* __restrict__ rstd, float* __restrict__ dz,
                                                   float* __restrict__ dgam, float* __restrict__ dbet, int R, int C,
                                                   int act) {
    __shared__ float red[4];
    const int c = blockIdx.x;
    const float g = gam[c], bb = bet[c];
    if (R <= 256 * BN_REG_ROWS) {
        // the thread's rows read once (dy, xhat), du kept in registers
        const int n = (R + 255) / 256;
        float duv[BN_REG_ROWS], xv[BN_REG_ROWS];
#pragma unroll
        for (int i = 0; i < BN_REG_ROWS; ++i)
            if (i < n) {
                const int64_t o = (int64_t)min((int)threadIdx.x + 256 * i, R - 1) * C + c;
                xv[i] = xhat[o];
                duv[i] = dy[o];
            }
        float sg = 0.f, sb = 0.f;
#pragma unroll
        for (int i = 0; i < BN_REG_ROWS; ++i)
            if (i < n && threadIdx.x + 256 * i < R) {
                const float du = act ? duv[i] * hswish_d(fmaf(g, xv[i], bb)) : duv[i];
                duv[i] = du;
                sg = fmaf(du, xv[i], sg);
                sb += du;
            }
        const float dg = block_sum(sg, red), db = block_sum(sb, red);
        const float k = g * rstd[c];
#pragma unroll
        for (int i = 0; i < BN_REG_ROWS; ++i) {
            const int r = threadIdx.x + 256 * i;
            if (i < n && r < R) dz[(int64_t)r * C + c] = k * (duv[i] - db / R - xv[i] * dg / R);
        }
        if (threadIdx.x == 0) {
            dgam[c] = dg;
            dbet[c] = db;
        }
        return;
    }
    float sg = 0.f, sb = 0.f;
    for (int r = threadIdx.x; r < R; r += 256) {
        const int64_t o = (int64_t)r * C + c;
        const float du = act ? dy[o] * hswish_d(fmaf(g, xhat[o], bb)) : dy[o];
        sg = fmaf(du, xhat[o], sg);
        sb += du;
    }
    const float dg = block_sum(sg, red), db = block_sum(sb, red);
    const float k = g * rstd[c];
    for (int r = threadIdx.x; r < R; r += 256) {
        const int64_t o = (int64_t)r * C + c;
        const float du = act ? dy[o] * hswish_d(fmaf(g, xhat[o], bb)) : dy[o];
        dz[o] = k * (du - db / R - xhat[o] * dg / R);
    }
    if (threadIdx.x == 0) {
        dgam[c] = dg;
        dbet[c] = db;
    }
}

// depthwise k x k, stride s, padding k / 2; x rows [B*H*W][C], y rows [B*Ho*Wo][C],
// weights [C][k][k]
__global__ void __launch_bounds__(256) dw_fwd(const float* __restrict__ x, const float* __restrict__ w,
                                              float* __restrict__ y, int B, int H, int C, int k, int s) {
    const int Ho = (H + 2 * (k / 2) - k) / s + 1;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)B * Ho * Ho * C) return;
    const int c = (int)(i % C);
    const int64_t r = i / C;
    const int b = (int)(r / (Ho * Ho)), oy = (int)(r / Ho % Ho), ox = (int)(r % Ho);
    // the taps (k <= 5) in order: inputs and weights loaded first from clamped
    // coordinates, the taps outside the filter or the image add zero
    float xv[25], wv[25];
#pragma unroll
    for (int q = 0; q < 25; ++q) {
        const int ky = min(q / 5, k - 1), kx = min(q % 5, k - 1);
        const int yy = min(max(oy * s + ky - k / 2, 0), H - 1), xx = min(max(ox * s + kx - k / 2, 0), H - 1);
        xv[q] = x[(((int64_t)b * H + yy) * H + xx) * C + c];
        wv[q] = w[(c * k + ky) * k + kx];
    }
    float acc = 0.f;
#pragma unroll
    for (int q = 0; q < 25; ++q) {
        const int ky = q / 5, kx = q % 5;
        const int yy = oy * s + ky - k / 2, xx = ox * s + kx - k / 2;
        const bool in = ky < k && kx < k && yy >= 0 && yy < H && xx >= 0 && xx < H;
        if (in) acc = fmaf(xv[q], wv[q], acc);
    }
    y[i] = acc;
}
// dx[b, yy, xx, c] = sum over the outputs whose window holds (yy, xx) of dy w
__global__ void __launch_bounds__(256) dw_bwd_x(const float* __restrict__ dy, const float* __restrict__ w,
                                                float* __restrict__ dx, int B, int H, int C, int k, int s) {
    const int Ho = (H + 2 * (k / 2) - k) / s + 1;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)B * H * H * C) return;
    const int c = (int)(i % C);
    const int64_t r = i / C;
    const int b = (int)(r / (H * H)), yy = (int)(r / H % H), xx = (int)(r % H);
    // the taps (k <= 5) in order, operands loaded first from clamped
    // coordinates; taps that reach no output pixel add nothing
    float gv[25], wv[25];
#pragma unroll
    for (int q = 0; q < 25; ++q) {
        const int ky = min(q / 5, k - 1), kx = min(q % 5, k - 1);
        const int oy = min(max(yy + k / 2 - ky, 0) / s, Ho - 1), ox = min(max(xx + k / 2 - kx, 0) / s, Ho - 1);
        gv[q] = dy[(((int64_t)b * Ho + oy) * Ho + ox) * C + c];
        wv[q] = w[(c * k + ky) * k + kx];
    }
    float acc = 0.f;
#pragma unroll
    for (int q = 0; q < 25; ++q) {
        const int ky = q / 5, kx = q % 5;
        const int ty = yy + k / 2 - ky, tx = xx + k / 2 - kx;  // = oy * s, ox * s
        const bool in = ky < k && kx < k && ty >= 0 && tx >= 0 && ty % s == 0 && tx % s == 0 && ty / s < Ho &&
                        tx / s < Ho;
        if (in) acc = fmaf(gv[q], wv[q], acc);
    }
    dx[i] = acc;
}
// Block c: dw[c][tap] = sum over outputs of dy x at the tap (k <= 5)
__global__ void __launch_bounds__(256) dw_bwd_w(const float* __restrict__ dy, const float* __restrict__ x,
                                                float* __restrict__ dw, int B, int H, int C, int k, int s) {
    __shared__ float part[25][257];
    const int Ho = (H + 2 * (k / 2) - k) / s + 1, c = blockIdx.x, t = threadIdx.x;
    float acc[25];
#pragma unroll
    for (int q = 0; q < 25; ++q) acc[q] = 0.f;
    for (int p = t; p < B * Ho * Ho; p += 256) {
        const int b = p / (Ho * Ho), oy = p / Ho % Ho, ox = p % Ho;
        const float g = dy[(int64_t)p * C + c];
        // every tap's input first (coordinates clamped into the image, so each
        // load is valid), then the products of the taps inside the image: a
        // bound test before each load makes each wait for the previous one
        float xv[25];
#pragma unroll
        for (int q = 0; q < 25; ++q) {
            const int ky = q / 5, kx = q % 5;
            const int yy = min(max(oy * s + ky - k / 2, 0), H - 1), xx = min(max(ox * s + kx - k / 2, 0), H - 1);
            xv[q] = ky < k && kx < k ? x[(((int64_t)b * H + yy) * H + xx) * C + c] : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 25; ++q) {
            const int ky = q / 5, kx = q % 5;
            const int yy = oy * s + ky - k / 2, xx = ox * s + kx - k / 2;
            const bool in = ky < k && kx < k && yy >= 0 && yy < H && xx >= 0 && xx < H;
            if (in) acc[q] = fmaf(g, xv[q], acc[q]);
        }
    }
#pragma unroll
    for (int q = 0; q < 25; ++q) part[q][t] = acc[q];
    __syncthreads();
    if (t < k * k) {
        const int q = (t / k) * 5 + t % k;
        float v = 0.f;
        for (int j = 0; j < 256; ++j) v += part[q][j];
        dw[(int64_t)c * k * k + t] = v;
    }
}

// m[b][c] = mean over the HW rows of sample b of a [B*HW][C]
__global__ void __launch_bounds__(256) rows_mean(const float* __restrict__ a, float* __restrict__ m, int B, int HW,
                                                 int C) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= B * C) return;
    const int b = i / C, c = i % C;
    float v = 0.f;
    for (int p = 0; p < HW; ++p) v += a[((int64_t)b * HW + p) * C + c];
    m[i] = v / HW;
}
// out[r][c] = a[r][c] hard-sigmoid(t[b][c])
__global__ void __launch_bounds__(256) se_scale(const float* __restrict__ a, const float* __restrict__ t,
                                                float* __restrict__ out, int B, int HW, int C) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)B * HW * C) return;
    const int c = (int)(i % C), b = (int)(i / C / HW);
    out[i] = a[i] * hsig(t[b * C + c]);
}
// dt[b][c] = hard-sigmoid'(t) sum over HW of dout a
__global__ void __launch_bounds__(256) se_dt(const float* __restrict__ dout, const float* __restrict__ a,
                                             const float* __restrict__ t, float* __restrict__ dt, int B, int HW,
                                             int C) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= B * C) return;
    const int b = i / C, c = i % C;
    float v = 0.f;
    for (int p = 0; p < HW; ++p) {
        const int64_t o = ((int64_t)b * HW + p) * C + c;
        v = fmaf(dout[o], a[o], v);
    }
    dt[i] = v * hsig_d(t[i]);
}
// da[r][c] = (t ? dout hard-sigmoid(t[b][c]) : 0) + dm[b][c] / HW
__global__ void __launch_bounds__(256) rows_bcast_add(const float* __restrict__ dout, const float* __restrict__ t,
                                                      const float* __restrict__ dm, float* __restrict__ da, int B,
                                                      int HW, int C) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)B * HW * C) return;
    const int c = (int)(i % C), b = (int)(i / C / HW);
    da[i] = (t ? dout[i] * hsig(t[b * C + c]) : 0.f) + dm[b * C + c] / HW;
}
// hard-swish forward (y from x) or backward (dx = dy hswish'(x)), elementwise
__global__ void __launch_bounds__(256) hswish_ew(const float* __restrict__ x, const float* __restrict__ dy,
                                                 float* __restrict__ out, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    out[i] = dy ? dy[i] * hswish_d(x[i]) : hswish(x[i]);
}

struct BlkP {
    const float *wex, *g1, *b1, *wdw, *g2, *b2, *wse1, *bse1, *wse2, *bse2, *wpr, *g3, *b3;
    float *gwex, *gg1, *gb1, *gwdw, *gg2, *gb2, *gwse1, *gbse1, *gwse2, *gbse2, *gwpr, *gg3, *gb3;
    int H, Ho;                                     // input and output side
    float *xh1, *a1, *xh2, *a2, *m, *q, *t, *a2s, *xh3, *y, *rs1, *rs2, *rs3;
};

struct Plan {
    BlkP bk[NBLK];
    const float *wl, *gl, *bl, *wf1, *bf1, *wf2, *bf2;
    float *gwl, *ggl, *gbl, *gwf1, *gbf1, *gwf2, *gbf2;
    float *x0, *zl, *xhl, *al, *rsl, *gp, *fpre, *f, *dz, *df, *dg, *z, *d0, *d1, *d2, *dm, *dt, *dq, *part, *colws;
    size_t part_floats;
    float* wgpart;  // the weight gradients' K slices until the update (wgrad_part_floats)
    size_t wgpart_floats;
};

// K slices of a weight gradient over R rows
int wgrad_slices(int64_t R) { return (int)std::min<int64_t>(kMaxSlices, std::max<int64_t>(1, R / 64)); }
// Floats for the weight gradients' K slices of one step, an upper bound (every
// product at the largest row count, each rounded up to 64 floats): the slices
// stay until the step sums them all before the update.
size_t wgrad_part_floats(int B) {
    const int64_t Rmax = (int64_t)B * HIN * HIN;
    const size_t S = wgrad_slices(Rmax), Sb = wgrad_slices(B);
    auto r64 = [](size_t n) { return (n + 63) / 64 * 64; };
    size_t n = r64(Sb * NCLS * F1) + r64(Sb * F1 * CLAST);
    int ci = CIN;
    for (int j = 0; j < NBLK; ++j) {
        const Blk& b = kBlk[j];
        n += r64(S * b.co * b.e) + r64(S * b.e * ci);
        if (b.se) n += 2 * r64(Sb * b.e * se_width(b.e));
        ci = b.co;
    }
    return n + r64(S * CLAST * ci);
}

size_t ws_floats(int B) {
    const size_t R = (size_t)B * HIN * HIN;
    size_t s = 0;
    auto add = [&](size_t n) { s += (4 * n + 255) / 256 * 64; };  // floats, 256-byte rounded
    for (int j = 0; j < NBLK; ++j) {
        const Blk& b = kBlk[j];
        add(R * b.e * 2);          // xh1, a1 (input side, at most R rows)
        add(R * b.e * 3);          // xh2, a2, a2s
        add((size_t)B * b.e * 3);  // m, t (+ q)
        add(R * b.co * 2);         // xh3, y
        add(3 * (size_t)b.e);      // rstd
    }
    add(R * CIN);                       // x0
    add(R * CLAST * 3);                 // zl, xhl, al
    add(CLAST);                         // rsl
    add((size_t)B * (CLAST + 2 * F1 + NCLS + F1 + CLAST));  // gp, fpre, f, dz, df, dg
    add(R * 960 * 4);                   // z, d0, d1, d2
    add((size_t)B * 960 * 3);           // dm, dt, dq
    add((size_t)kMaxSlices * CLAST * 200 + (size_t)kMaxSlices * F1 * CLAST / 4);  // part
    add(colsum_ws_floats(B, F1));       // colws
    add(wgrad_part_floats(B));          // wgpart
    return s;
}

size_t ws_bytes(const fo_model* m) { return sizeof(Plan) + 256 + 4 * ws_floats(m->max_batch) + 256 * 256; }

fo_status init(fo_model* m) {
    Plan* P = new (std::nothrow) Plan();
    if (!P) return FO_ENOMEM;
    m->plan = P;
    const int B = m->max_batch;
    const size_t R = (size_t)B * HIN * HIN;
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
    int ci = CIN, H = HIN;
    for (int j = 0; j < NBLK; ++j) {
        const Blk& b = kBlk[j];
        BlkP& K = P->bk[j];
        K.H = H;
        K.Ho = (H + 2 * (b.k / 2) - b.k) / b.stride + 1;
        take(K.wex, K.gwex, (size_t)b.e * ci);
        take(K.g1, K.gg1, b.e);
        take(K.b1, K.gb1, b.e);
        take(K.wdw, K.gwdw, (size_t)b.e * b.k * b.k);
        take(K.g2, K.gg2, b.e);
        take(K.b2, K.gb2, b.e);
        if (b.se) {
            const int S = se_width(b.e);
            take(K.wse1, K.gwse1, (size_t)S * b.e);
            take(K.bse1, K.gbse1, S);
            take(K.wse2, K.gwse2, (size_t)b.e * S);
            take(K.bse2, K.gbse2, b.e);
        }
        take(K.wpr, K.gwpr, (size_t)b.co * b.e);
        take(K.g3, K.gg3, b.co);
        take(K.b3, K.gb3, b.co);
        const size_t Ri = (size_t)B * H * H, Ro = (size_t)B * K.Ho * K.Ho;
        K.xh1 = ar.take<float>(Ri * b.e);
        K.a1 = ar.take<float>(Ri * b.e);
        K.xh2 = ar.take<float>(Ro * b.e);
        K.a2 = ar.take<float>(Ro * b.e);
        K.a2s = ar.take<float>(Ro * b.e);
        K.m = ar.take<float>((size_t)B * b.e);
        K.q = ar.take<float>((size_t)B * b.e);
        K.t = ar.take<float>((size_t)B * b.e);
        K.xh3 = ar.take<float>(Ro * b.co);
        K.y = ar.take<float>(Ro * b.co);
        K.rs1 = ar.take<float>(b.e);
        K.rs2 = ar.take<float>(b.e);
        K.rs3 = ar.take<float>(b.e);
        ci = b.co;
        H = K.Ho;
    }
    take(P->wl, P->gwl, (size_t)CLAST * ci);
    take(P->gl, P->ggl, CLAST);
    take(P->bl, P->gbl, CLAST);
    take(P->wf1, P->gwf1, (size_t)F1 * CLAST);
    take(P->bf1, P->gbf1, F1);
    take(P->wf2, P->gwf2, (size_t)NCLS * F1);
    take(P->bf2, P->gbf2, NCLS);
    P->x0 = ar.take<float>(R * CIN);
    P->zl = ar.take<float>(R * CLAST);
    P->xhl = ar.take<float>(R * CLAST);
    P->al = ar.take<float>(R * CLAST);
    P->rsl = ar.take<float>(CLAST);
    P->gp = ar.take<float>((size_t)B * CLAST);
    P->fpre = ar.take<float>((size_t)B * F1);
    P->f = ar.take<float>((size_t)B * F1);
    P->dz = ar.take<float>((size_t)B * NCLS);
    P->df = ar.take<float>((size_t)B * F1);
    P->dg = ar.take<float>((size_t)B * CLAST);
    P->z = ar.take<float>(R * 960);
    P->d0 = ar.take<float>(R * 960);
    P->d1 = ar.take<float>(R * 960);
    P->d2 = ar.take<float>(R * 960);
    P->dm = ar.take<float>((size_t)B * 960);
    P->dt = ar.take<float>((size_t)B * 960);
    P->dq = ar.take<float>((size_t)B * 960);
    P->part_floats = (size_t)kMaxSlices * CLAST * 200 + (size_t)kMaxSlices * F1 * CLAST / 4;
    P->part = ar.take<float>(P->part_floats);
    P->colws = ar.take<float>(colsum_ws_floats(B, F1));
    P->wgpart_floats = wgrad_part_floats(B);
    P->wgpart = ar.take<float>(P->wgpart_floats);
    if (!P->wgpart) {
        set_error("mbv3: workspace arena too small");
        return FO_ENOMEM;
    }
    return FO_OK;
}

GemmF32 prod(const float* A, int64_t am, int64_t ak, const float* B, int64_t bn, int64_t bk, float* C, int64_t ldc,
             int M, int N, int K) {
    GemmF32 g{};
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
    g.auto_split = 1;
    return g;
}

fo_status step(fo_model* m, const fo_acts* acts, const int32_t* labels) {
    (void)labels;  // read through m->dev_in
    Plan* P = (Plan*)m->plan;
    hipStream_t s = m->stream;
    const int B = acts->batch;
    fo_status st = FO_OK;
    auto gemm = [&](const GemmF32& g) { return launch_gemm_f32(g, P->part, P->part_floats, s); };
    // y[r][n] = x[r][:] . W[n][:] (+ bias, ReLU) for W [N][K]
    auto linear = [&](const float* x, const float* W, const float* bias, float* y, int R, int N, int K, int relu) {
        GemmF32 g = prod(x, K, 1, W, K, 1, y, N, R, N, K);
        g.bias = bias;
        g.relu = relu;
        return gemm(g);
    };
    // dW[n][k] = sum_r dy[r][n] x[r][k].  Nothing reads dW before the update,
    // so its K slices stay in wgpart and join `wsums`, added up for every
    // product in one launch at the end of the backward.
    SplitJobs wsums;
    size_t wused = 0;
    auto linear_dw = [&](const float* dy, const float* x, float* dW, int R, int N, int K) -> fo_status {
        GemmF32 g = prod(dy, 1, N, x, 1, K, dW, K, N, K, R);
        g.S = wgrad_slices(R);
        if (g.S <= 1) return gemm(g);
        const size_t n = (size_t)g.S * N * K;
        FO_CHECK(wsums.n < kSplitJobsMax && wused + n <= P->wgpart_floats,
                 "mbv3: deferred weight-gradient slices exceed their workspace");
        g.defer = 1;
        SplitJob& j = wsums.j[wsums.n++];
        j.ws = P->wgpart + wused; j.C = dW; j.ldc = K; j.S = g.S; j.M = N; j.N = K;
        const fo_status r = launch_gemm_f32(g, P->wgpart + wused, n, s);
        wused += (n + 63) / 64 * 64;
        return r;
    };
    // dx[r][k] = dy[r][:] . W[:][k] (+ add, times mask > 0)
    auto linear_dx = [&](const float* dy, const float* W, float* dx, int R, int N, int K, const float* add,
                         const float* mask) {
        GemmF32 g = prod(dy, N, 1, W, 1, K, dx, K, R, K, N);
        g.add = add;
        g.ldadd = K;
        g.mask = mask;
        g.ldmask = K;
        return gemm(g);
    };
    auto bnf = [&](const float* z, const float* gm, const float* bt, float* xh, float* y, float* rs, const float* add,
                   int R, int C, int act) {
        hipLaunchKernelGGL(bn_rows_fwd, dim3(C), dim3(256), 0, s, z, gm, bt, xh, y, rs, add, R, C, act);
        FO_LAUNCHED();
        return FO_OK;
    };
    auto bnb = [&](const float* dy, const float* xh, const float* gm, const float* bt, const float* rs, float* dz,
                   float* dgm, float* dbt, int R, int C, int act) {
        hipLaunchKernelGGL(bn_rows_bwd, dim3(C), dim3(256), 0, s, dy, xh, gm, bt, rs, dz, dgm, dbt, R, C, act);
        FO_LAUNCHED();
        return FO_OK;
    };
#define TRY(x)                      \
    do {                            \
        st = (x);                   \
        if (st != FO_OK) return st; \
    } while (0)
    // forward (Alg. 4: forward pass of M_s)
    hipLaunchKernelGGL(nchw_rows, dim3(nblk((int64_t)B * CIN * HIN * HIN)), dim3(256), 0, s, m->dev_in, P->x0, B, CIN,
                       HIN * HIN);
    FO_LAUNCHED();
    const float* x = P->x0;
    int ci = CIN;
    for (int j = 0; j < NBLK; ++j) {
        const Blk& b = kBlk[j];
        BlkP& K = P->bk[j];
        const int Ri = B * K.H * K.H, Ro = B * K.Ho * K.Ho, HWo = K.Ho * K.Ho;
        TRY(linear(x, K.wex, nullptr, P->z, Ri, b.e, ci, 0));
        TRY(bnf(P->z, K.g1, K.b1, K.xh1, K.a1, K.rs1, nullptr, Ri, b.e, 1));
        hipLaunchKernelGGL(dw_fwd, dim3(nblk((int64_t)Ro * b.e)), dim3(256), 0, s, K.a1, K.wdw, P->z, B, K.H, b.e, b.k,
                           b.stride);
        FO_LAUNCHED();
        TRY(bnf(P->z, K.g2, K.b2, K.xh2, K.a2, K.rs2, nullptr, Ro, b.e, 1));
        const float* h = K.a2;
        if (b.se) {
            const int S = se_width(b.e);
            hipLaunchKernelGGL(rows_mean, dim3(nblk((int64_t)B * b.e)), dim3(256), 0, s, K.a2, K.m, B, HWo, b.e);
            FO_LAUNCHED();
            TRY(linear(K.m, K.wse1, K.bse1, K.q, B, S, b.e, 1));
            TRY(linear(K.q, K.wse2, K.bse2, K.t, B, b.e, S, 0));
            hipLaunchKernelGGL(se_scale, dim3(nblk((int64_t)Ro * b.e)), dim3(256), 0, s, K.a2, K.t, K.a2s, B, HWo,
                               b.e);
            FO_LAUNCHED();
            h = K.a2s;
        }
        TRY(linear(h, K.wpr, nullptr, P->z, Ro, b.co, b.e, 0));
        const bool res = b.stride == 1 && ci == b.co;
        TRY(bnf(P->z, K.g3, K.b3, K.xh3, K.y, K.rs3, res ? x : nullptr, Ro, b.co, 0));
        x = K.y;
        ci = b.co;
    }
    const int Rl = B * P->bk[NBLK - 1].Ho * P->bk[NBLK - 1].Ho, HWl = Rl / B;
    TRY(linear(x, P->wl, nullptr, P->zl, Rl, CLAST, ci, 0));
    TRY(bnf(P->zl, P->gl, P->bl, P->xhl, P->al, P->rsl, nullptr, Rl, CLAST, 1));
    hipLaunchKernelGGL(rows_mean, dim3(nblk((int64_t)B * CLAST)), dim3(256), 0, s, P->al, P->gp, B, HWl, CLAST);
    FO_LAUNCHED();
    TRY(linear(P->gp, P->wf1, P->bf1, P->fpre, B, F1, CLAST, 0));
    hipLaunchKernelGGL(hswish_ew, dim3(nblk((int64_t)B * F1)), dim3(256), 0, s, P->fpre, nullptr, P->f,
                       (int64_t)B * F1);
    FO_LAUNCHED();
    TRY(linear(P->f, P->wf2, P->bf2, m->logits, B, NCLS, F1, 0));
    TRY(launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, NCLS, s));
    // backward (Alg. 4: backward pass of M_s)
    TRY(linear_dw(P->dz, P->f, P->gwf2, B, NCLS, F1));
    TRY(launch_colsum(P->dz, NCLS, B, nullptr, NCLS, P->gbf2, P->colws, s));
    TRY(linear_dx(P->dz, P->wf2, P->df, B, NCLS, F1, nullptr, nullptr));
    hipLaunchKernelGGL(hswish_ew, dim3(nblk((int64_t)B * F1)), dim3(256), 0, s, P->fpre, P->df, P->df,
                       (int64_t)B * F1);
    FO_LAUNCHED();
    TRY(linear_dw(P->df, P->gp, P->gwf1, B, F1, CLAST));
    TRY(launch_colsum(P->df, F1, B, nullptr, F1, P->gbf1, P->colws, s));
    TRY(linear_dx(P->df, P->wf1, P->dg, B, F1, CLAST, nullptr, nullptr));
    hipLaunchKernelGGL(rows_bcast_add, dim3(nblk((int64_t)Rl * CLAST)), dim3(256), 0, s, nullptr, nullptr, P->dg,
                       P->d1, B, HWl, CLAST);
    FO_LAUNCHED();
    TRY(bnb(P->d1, P->xhl, P->gl, P->bl, P->rsl, P->d2, P->ggl, P->gbl, Rl, CLAST, 1));
    TRY(linear_dw(P->d2, P->bk[NBLK - 1].y, P->gwl, Rl, CLAST, ci));
    float* dy = P->d0;  // gradient of the current block's output
    float *t1 = P->d1, *t2 = P->d2;  // scratch
    TRY(linear_dx(t2, P->wl, dy, Rl, CLAST, ci, nullptr, nullptr));
    for (int j = NBLK - 1; j >= 0; --j) {
        const Blk& b = kBlk[j];
        BlkP& K = P->bk[j];
        const int Ri = B * K.H * K.H, Ro = B * K.Ho * K.Ho, HWo = K.Ho * K.Ho;
        const int cin = j ? kBlk[j - 1].co : CIN;
        const float* xin = j ? P->bk[j - 1].y : P->x0;
        const bool res = b.stride == 1 && cin == b.co;
        // projection and its batch norm
        TRY(bnb(dy, K.xh3, K.g3, K.b3, K.rs3, t1, K.gg3, K.gb3, Ro, b.co, 0));
        TRY(linear_dw(t1, b.se ? K.a2s : K.a2, K.gwpr, Ro, b.co, b.e));
        TRY(linear_dx(t1, K.wpr, t2, Ro, b.co, b.e, nullptr, nullptr));  // d(h)
        if (b.se) {
            const int S = se_width(b.e);
            hipLaunchKernelGGL(se_dt, dim3(nblk((int64_t)B * b.e)), dim3(256), 0, s, t2, K.a2, K.t, P->dt, B, HWo,
                               b.e);
            FO_LAUNCHED();
            TRY(linear_dw(P->dt, K.q, K.gwse2, B, b.e, S));
            TRY(launch_colsum(P->dt, b.e, B, nullptr, b.e, K.gbse2, P->colws, s));
            TRY(linear_dx(P->dt, K.wse2, P->dq, B, b.e, S, nullptr, K.q));  // times (q > 0)
            TRY(linear_dw(P->dq, K.m, K.gwse1, B, S, b.e));
            TRY(launch_colsum(P->dq, S, B, nullptr, S, K.gbse1, P->colws, s));
            TRY(linear_dx(P->dq, K.wse1, P->dm, B, S, b.e, nullptr, nullptr));
            hipLaunchKernelGGL(rows_bcast_add, dim3(nblk((int64_t)Ro * b.e)), dim3(256), 0, s, t2, K.t, P->dm,
                               t1, B, HWo, b.e);
            FO_LAUNCHED();
            std::swap(t1, t2);  // d(a2) in t2
        }
        // depthwise conv and its batch norm (hard-swish)
        TRY(bnb(t2, K.xh2, K.g2, K.b2, K.rs2, t1, K.gg2, K.gb2, Ro, b.e, 1));
        hipLaunchKernelGGL(dw_bwd_w, dim3(b.e), dim3(256), 0, s, t1, K.a1, K.gwdw, B, K.H, b.e, b.k, b.stride);
        hipLaunchKernelGGL(dw_bwd_x, dim3(nblk((int64_t)Ri * b.e)), dim3(256), 0, s, t1, K.wdw, t2, B, K.H,
                           b.e, b.k, b.stride);
        FO_LAUNCHED();
        // expansion conv and its batch norm (hard-swish)
        TRY(bnb(t2, K.xh1, K.g1, K.b1, K.rs1, t1, K.gg1, K.gb1, Ri, b.e, 1));
        TRY(linear_dw(t1, xin, K.gwex, Ri, b.e, cin));
        if (j > 0) {  // the first server layer's input gradient is never formed
            float* dx = dy == P->d0 ? P->z : P->d0;
            TRY(linear_dx(t1, K.wex, dx, Ri, b.e, cin, res ? dy : nullptr, nullptr));
            dy = dx;
        }
    }
    if (wsums.n) TRY(launch_splitk_sum_multi(wsums, s));
#undef TRY
    // SGD (Alg. 4)
    return launch_sgd(m->params, m->grads, nullptr, nullptr, nullptr, m->n_params, m->lr, 0.f, s);
}

void destroy(fo_model* m) {
    delete (Plan*)m->plan;
    m->plan = nullptr;
}

}  // namespace

int64_t mbv3_param_count() {
    int64_t n = 0;
    int ci = CIN;
    for (const Blk& b : kBlk) {
        n += (int64_t)b.e * ci + 2 * b.e + (int64_t)b.e * b.k * b.k + 2 * b.e;
        if (b.se) n += 2LL * se_width(b.e) * b.e + se_width(b.e) + b.e;
        n += (int64_t)b.co * b.e + 2 * b.co;
        ci = b.co;
    }
    return n + (int64_t)CLAST * ci + 2 * CLAST + (int64_t)F1 * CLAST + F1 + (int64_t)NCLS * F1 + NCLS;
}

const Family* family_mbv3() {
    static const Family f = {(int64_t)CIN * HIN * HIN * 4, ws_bytes, init, step, destroy};
    return &f;
}

}  // namespace fo
