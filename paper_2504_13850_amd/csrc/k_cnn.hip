// Elementwise and reduction kernels of the bf16 CNN server networks (NHWC):
// layout change at the boundary, 2x2 max pooling, global average pooling,
// training-mode batch normalisation, ReLU masks, and fp32 -> bf16 splits.
// Activations that feed a GEMM are kept as bf16 (high, low) pairs so the
// forward products can be compensated; gradients are single bf16 (plus fp32
// where a reduction reads them).
#include "kernels.h"

namespace fo {
namespace {

__device__ __forceinline__ void split_store(bf16_t* hi, bf16_t* lo, int64_t i, float v) {
    const bf16_t h = f2bf(v);
    hi[i] = h;
    if (lo) lo[i] = f2bf(v - bf2f(h));
}

// x [B][C][H][W] -> y [B][H][W][C] (bf16 bits)
__global__ void __launch_bounds__(256) nchw_to_nhwc(const bf16_t* __restrict__ x, bf16_t* __restrict__ y, int B,
                                                    int C, int HW) {
    __shared__ bf16_t tile[32][33];
    const int b = blockIdx.z;
    const int c0 = blockIdx.y * 32, p0 = blockIdx.x * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
    for (int r = ty; r < 32; r += 8) {
        int c = c0 + r, p = p0 + tx;
        tile[r][tx] = (c < C && p < HW) ? x[((int64_t)b * C + c) * HW + p] : (bf16_t)0;
    }
    __syncthreads();
    for (int r = ty; r < 32; r += 8) {
        int p = p0 + r, c = c0 + tx;
        if (c < C && p < HW) y[((int64_t)b * HW + p) * C + c] = tile[tx][r];
    }
}

// 2x2/2 max pooling of the value hi + lo; the first maximum in row-major
// window order wins; the winner's (hi, lo) pair is copied and its position kept.
__global__ void __launch_bounds__(256) maxpool_fwd(const bf16_t* __restrict__ xh, const bf16_t* __restrict__ xl,
                                                   bf16_t* __restrict__ yh, bf16_t* __restrict__ yl,
                                                   uint8_t* __restrict__ arg, int B, int H, int W, int C) {
    const int Ho = H / 2, Wo = W / 2;
    const int64_t total = (int64_t)B * Ho * Wo * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(i % C);
        int64_t r = i / C;
        const int ox = (int)(r % Wo);
        r /= Wo;
        const int oy = (int)(r % Ho);
        const int b = (int)(r / Ho);
        int64_t src[4];
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int iy = 2 * oy + (t >> 1), ix = 2 * ox + (t & 1);
            src[t] = (((int64_t)b * H + iy) * W + ix) * C + c;
            v[t] = bf2f(xh[src[t]]) + (xl ? bf2f(xl[src[t]]) : 0.f);
        }
        int a = 0;
#pragma unroll
        for (int t = 1; t < 4; ++t)
            if (v[t] > v[a]) a = t;
        yh[i] = xh[src[a]];
        if (yl) yl[i] = xl ? xl[src[a]] : (bf16_t)0;
        arg[i] = (uint8_t)a;
    }
}

// dx at the window's winner = dy (and 0 elsewhere), times [y > 0] of the
// pooled layer's own (post-ReLU) output y.  Writes fp32 and bf16.
__global__ void __launch_bounds__(256) maxpool_relu_bwd(const float* __restrict__ dy, const uint8_t* __restrict__ arg,
                                                        const bf16_t* __restrict__ y, float* __restrict__ dxf,
                                                        bf16_t* __restrict__ dxb, int B, int H, int W, int C) {
    const int64_t total = (int64_t)B * H * W * C;
    const int Ho = H / 2, Wo = W / 2;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(i % C);
        int64_t r = i / C;
        const int x = (int)(r % W);
        r /= W;
        const int yy = (int)(r % H);
        const int b = (int)(r / H);
        const int64_t o = (((int64_t)b * Ho + yy / 2) * Wo + x / 2) * C + c;
        const int pos = (yy & 1) * 2 + (x & 1);
        float g = (arg[o] == pos && bf2f(y[i]) > 0.f) ? dy[o] : 0.f;
        dxf[i] = g;
        dxb[i] = f2bf(g);
    }
}

// h[b][c] = mean over the H*W pixels of x (hi + lo)
__global__ void __launch_bounds__(256) gap_fwd(const bf16_t* __restrict__ xh, const bf16_t* __restrict__ xl,
                                               float* __restrict__ h, int B, int HW, int C) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * C) return;
    const int b = (int)(i / C), c = (int)(i % C);
    float s = 0.f;
    for (int p = 0; p < HW; ++p) {
        const int64_t k = ((int64_t)b * HW + p) * C + c;
        s += bf2f(xh[k]) + (xl ? bf2f(xl[k]) : 0.f);
    }
    h[i] = s / (float)HW;
}

// dx[b][p][c] = dh[b][c] / HW * [y > 0]
__global__ void __launch_bounds__(256) gap_relu_bwd(const float* __restrict__ dh, const bf16_t* __restrict__ y,
                                                    float* __restrict__ dxf, int B, int HW, int C) {
    const int64_t total = (int64_t)B * HW * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(i % C);
        const int b = (int)(i / ((int64_t)HW * C));
        dxf[i] = bf2f(y[i]) > 0.f ? dh[(int64_t)b * C + c] / (float)HW : 0.f;
    }
}

// ---- batch norm (training mode): per-channel statistics over the N*H*W rows
constexpr int BN_ROWS = 64;

// partial column sums of (z - shift) and (z - shift)^2; shift = z of row 0
// (a per-channel shift keeps the one-pass variance well conditioned)
__global__ void __launch_bounds__(256) bn_stats_partial(const float* __restrict__ z, int rows, int C,
                                                        float* __restrict__ part) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= C) return;
    const float sh = z[c];
    const int r0 = blockIdx.y * BN_ROWS, r1 = min(rows, r0 + BN_ROWS);
    float s = 0.f, q = 0.f;
    for (int r = r0; r < r1; ++r) {
        const float d = z[(int64_t)r * C + c] - sh;
        s += d;
        q = fmaf(d, d, q);
    }
    part[((int64_t)blockIdx.y * 2 + 0) * C + c] = s;
    part[((int64_t)blockIdx.y * 2 + 1) * C + c] = q;
}

__global__ void __launch_bounds__(256) bn_stats_finish(const float* __restrict__ z, const float* __restrict__ part,
                                                       int chunks, int rows, int C, float eps,
                                                       float* __restrict__ mean, float* __restrict__ rstd) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= C) return;
    double s = 0.0, q = 0.0;
    for (int k = 0; k < chunks; ++k) {
        s += part[((int64_t)k * 2 + 0) * C + c];
        q += part[((int64_t)k * 2 + 1) * C + c];
    }
    const double n = rows, m = s / n;
    double var = q / n - m * m;
    var = var < 0.0 ? 0.0 : var;
    mean[c] = (float)(z[c] + m);
    rstd[c] = (float)(1.0 / sqrt(var + eps));
}

// y = relu(gamma (z - mean) rstd + beta [+ residual]) -> (hi, lo) bf16
__global__ void __launch_bounds__(256) bn_apply(const float* __restrict__ z, const float* __restrict__ mean,
                                                const float* __restrict__ rstd, const float* __restrict__ g,
                                                const float* __restrict__ beta, const float* __restrict__ resf,
                                                const bf16_t* __restrict__ resh, const bf16_t* __restrict__ resl,
                                                int relu, int64_t total, int C, float* __restrict__ yf,
                                                bf16_t* __restrict__ yh, bf16_t* __restrict__ yl) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(i % C);
        float v = fmaf((z[i] - mean[c]) * rstd[c], g[c], beta[c]);
        if (resf) v += resf[i];
        if (resh) v += bf2f(resh[i]) + (resl ? bf2f(resl[i]) : 0.f);
        if (relu) v = v > 0.f ? v : 0.f;
        if (yf) yf[i] = v;
        if (yh) split_store(yh, yl, i, v);
    }
}

// dbeta = sum dy, dgamma = sum dy * xhat (partials)
__global__ void __launch_bounds__(256) bn_bwd_partial(const float* __restrict__ dy, const float* __restrict__ z,
                                                      const float* __restrict__ mean, const float* __restrict__ rstd,
                                                      int rows, int C, float* __restrict__ part) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= C) return;
    const int r0 = blockIdx.y * BN_ROWS, r1 = min(rows, r0 + BN_ROWS);
    const float m = mean[c], rs = rstd[c];
    float sb = 0.f, sg = 0.f;
    for (int r = r0; r < r1; ++r) {
        const float d = dy[(int64_t)r * C + c];
        sb += d;
        sg = fmaf(d, (z[(int64_t)r * C + c] - m) * rs, sg);
    }
    part[((int64_t)blockIdx.y * 2 + 0) * C + c] = sg;
    part[((int64_t)blockIdx.y * 2 + 1) * C + c] = sb;
}

__global__ void __launch_bounds__(256) bn_bwd_finish(const float* __restrict__ part, int chunks, int C,
                                                     float* __restrict__ dg, float* __restrict__ db) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= C) return;
    float sg = 0.f, sb = 0.f;
    for (int k = 0; k < chunks; ++k) {
        sg += part[((int64_t)k * 2 + 0) * C + c];
        sb += part[((int64_t)k * 2 + 1) * C + c];
    }
    dg[c] = sg;
    db[c] = sb;
}

// dz = gamma rstd (dy - dbeta/N - xhat dgamma/N) -> fp32 and bf16
__global__ void __launch_bounds__(256) bn_bwd_apply(const float* __restrict__ dy, const float* __restrict__ z,
                                                    const float* __restrict__ mean, const float* __restrict__ rstd,
                                                    const float* __restrict__ g, const float* __restrict__ dg,
                                                    const float* __restrict__ db, int rows, int C,
                                                    float* __restrict__ dzf, bf16_t* __restrict__ dzb) {
    const int64_t total = (int64_t)rows * C;
    const float inv = 1.f / (float)rows;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(i % C);
        const float xh = (z[i] - mean[c]) * rstd[c];
        const float v = g[c] * rstd[c] * (dy[i] - db[c] * inv - xh * dg[c] * inv);
        if (dzf) dzf[i] = v;
        if (dzb) dzb[i] = f2bf(v);
    }
}

// d = dy * [y > 0] (fp32), optionally adding a second gradient
__global__ void __launch_bounds__(256) relu_mask(const float* __restrict__ dy, const float* __restrict__ add,
                                                 const bf16_t* __restrict__ y, int64_t total, float* __restrict__ d) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        float v = dy[i] + (add ? add[i] : 0.f);
        d[i] = bf2f(y[i]) > 0.f ? v : 0.f;
    }
}

__global__ void __launch_bounds__(256) to_bf16(const float* __restrict__ x, bf16_t* __restrict__ y, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        y[i] = f2bf(x[i]);
}

inline int grid_for(int64_t n) { return (int)std::min<int64_t>(cdiv(n, 256), 8192); }

}  // namespace

fo_status launch_nchw_to_nhwc(const bf16_t* x, bf16_t* y, int B, int C, int HW, hipStream_t s) {
    hipLaunchKernelGGL(nchw_to_nhwc, dim3(cdiv(HW, 32), cdiv(C, 32), B), dim3(256), 0, s, x, y, B, C, HW);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_maxpool_fwd(const bf16_t* xh, const bf16_t* xl, bf16_t* yh, bf16_t* yl, uint8_t* arg, int B, int H,
                             int W, int C, hipStream_t s) {
    hipLaunchKernelGGL(maxpool_fwd, dim3(grid_for((int64_t)B * H * W * C / 4)), dim3(256), 0, s, xh, xl, yh, yl, arg,
                       B, H, W, C);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_maxpool_relu_bwd(const float* dy, const uint8_t* arg, const bf16_t* y, float* dxf, bf16_t* dxb, int B,
                                  int H, int W, int C, hipStream_t s) {
    hipLaunchKernelGGL(maxpool_relu_bwd, dim3(grid_for((int64_t)B * H * W * C)), dim3(256), 0, s, dy, arg, y, dxf, dxb,
                       B, H, W, C);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_gap_fwd(const bf16_t* xh, const bf16_t* xl, float* h, int B, int HW, int C, hipStream_t s) {
    hipLaunchKernelGGL(gap_fwd, dim3(cdiv((int64_t)B * C, 256)), dim3(256), 0, s, xh, xl, h, B, HW, C);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_gap_relu_bwd(const float* dh, const bf16_t* y, float* dxf, int B, int HW, int C, hipStream_t s) {
    hipLaunchKernelGGL(gap_relu_bwd, dim3(grid_for((int64_t)B * HW * C)), dim3(256), 0, s, dh, y, dxf, B, HW, C);
    FO_LAUNCHED();
    return FO_OK;
}

size_t bn_ws_floats(int rows, int C) { return (size_t)cdiv(rows, BN_ROWS) * 2 * C; }

fo_status launch_bn_stats(const float* z, int rows, int C, float eps, float* mean, float* rstd, float* ws,
                          hipStream_t s) {
    const int chunks = (int)cdiv(rows, BN_ROWS);
    hipLaunchKernelGGL(bn_stats_partial, dim3(cdiv(C, 256), chunks), dim3(256), 0, s, z, rows, C, ws);
    hipLaunchKernelGGL(bn_stats_finish, dim3(cdiv(C, 256)), dim3(256), 0, s, z, ws, chunks, rows, C, eps, mean, rstd);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_bn_apply(const float* z, const float* mean, const float* rstd, const float* g, const float* beta,
                          const float* resf, const bf16_t* resh, const bf16_t* resl, bool relu, int rows, int C,
                          float* yf, bf16_t* yh, bf16_t* yl, hipStream_t s) {
    const int64_t total = (int64_t)rows * C;
    hipLaunchKernelGGL(bn_apply, dim3(grid_for(total)), dim3(256), 0, s, z, mean, rstd, g, beta, resf, resh, resl,
                       relu ? 1 : 0, total, C, yf, yh, yl);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_bn_bwd(const float* dy, const float* z, const float* mean, const float* rstd, const float* g,
                        int rows, int C, float* dg, float* db, float* dzf, bf16_t* dzb, float* ws, hipStream_t s) {
    const int chunks = (int)cdiv(rows, BN_ROWS);
    hipLaunchKernelGGL(bn_bwd_partial, dim3(cdiv(C, 256), chunks), dim3(256), 0, s, dy, z, mean, rstd, rows, C, ws);
    hipLaunchKernelGGL(bn_bwd_finish, dim3(cdiv(C, 256)), dim3(256), 0, s, ws, chunks, C, dg, db);
    hipLaunchKernelGGL(bn_bwd_apply, dim3(grid_for((int64_t)rows * C)), dim3(256), 0, s, dy, z, mean, rstd, g, dg, db,
                       rows, C, dzf, dzb);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_relu_mask(const float* dy, const float* add, const bf16_t* y, int64_t n, float* d, hipStream_t s) {
    hipLaunchKernelGGL(relu_mask, dim3(grid_for(n)), dim3(256), 0, s, dy, add, y, n, d);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_to_bf16(const float* x, bf16_t* y, int64_t n, hipStream_t s) {
    hipLaunchKernelGGL(to_bf16, dim3(grid_for(n)), dim3(256), 0, s, x, y, n);
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
