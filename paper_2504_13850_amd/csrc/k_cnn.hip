// Elementwise and reduction kernels of the bf16 CNN server networks (NHWC):
// layout change at the boundary, 2x2 max pooling, global average pooling,
// training-mode batch normalisation (with the ReLU around it), and fp32 ->
// bf16 splits.
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

// x [B][C][H][W] -> y [B][H][W][C] (bf16 bits); x is the step's batch (in->x)
__global__ void __launch_bounds__(256) nchw_to_nhwc(const StepIn* __restrict__ in, bf16_t* __restrict__ y, int B,
                                                    int C, int HW) {
    __shared__ bf16_t tile[32][33];
    const bf16_t* __restrict__ x = static_cast<const bf16_t*>(in->x);
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
        // the four taps' high (and low) parts, each in one uniform branch, before the first use
        bf16_t hv[4], lv[4] = {};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int iy = 2 * oy + (t >> 1), ix = 2 * ox + (t & 1);
            hv[t] = xh[(((int64_t)b * H + iy) * W + ix) * C + c];
        }
        if (xl) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int iy = 2 * oy + (t >> 1), ix = 2 * ox + (t & 1);
                lv[t] = xl[(((int64_t)b * H + iy) * W + ix) * C + c];
            }
        }
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = bf2f(hv[t]) + (xl ? bf2f(lv[t]) : 0.f);
        int a = 0;
#pragma unroll
        for (int t = 1; t < 4; ++t)
            if (v[t] > v[a]) a = t;
        yh[i] = hv[a];
        if (yl) yl[i] = lv[a];
        arg[i] = (uint8_t)a;
    }
}

// dx at the window's winner = dy (and 0 elsewhere), times [y > 0] of the
// pooled layer's own (post-ReLU) output y.  Writes fp32 and bf16.
__global__ void __launch_bounds__(256) maxpool_relu_bwd(const float* __restrict__ dy, const uint8_t* __restrict__ arg,
                                                        const bf16_t* __restrict__ y, float* __restrict__ dxf,
                                                        bf16_t* __restrict__ dxb, int B, int H, int W, int C) {
    // one thread per pooled output (b, yo, xo, c): its four window inputs, the
    // index arithmetic done once for them
    const int Ho = H / 2, Wo = W / 2;
    const int64_t total = (int64_t)B * Ho * Wo * C;
    const int64_t rowC = (int64_t)W * C;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total; o += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(o % C);
        int64_t r = o / C;
        const int xo = (int)(r % Wo);
        r /= Wo;
        const int yo = (int)(r % Ho);
        const int b = (int)(r / Ho);
        const int64_t i0 = (((int64_t)b * H + 2 * yo) * W + 2 * xo) * C + c;
        const int64_t off[4] = {0, C, rowC, rowC + C};  // window position (yy & 1) * 2 + (x & 1)
        const int a = arg[o];
        const float g = dy[o];
        bf16_t yv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) yv[q] = y[i0 + off[q]];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float v = (a == q && bf2f(yv[q]) > 0.f) ? g : 0.f;
            dxf[i0 + off[q]] = v;
            dxb[i0 + off[q]] = f2bf(v);
        }
    }
}

// h[b][c] = mean over the H*W pixels of x (hi + lo).  Block = (sample b,
// 64 channels c0 ..): lane = channel (one 128-byte row segment per wave and
// pixel), the four waves take every fourth pixel, eight loads in flight per
// lane, the waves' sums added in wave order.
__global__ void __launch_bounds__(256) gap_fwd(const bf16_t* __restrict__ xh, const bf16_t* __restrict__ xl,
                                               float* __restrict__ h, int B, int HW, int C) {
    __shared__ float red[4][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int b = blockIdx.y, c = blockIdx.x * 64 + lane;
    float s = 0.f;
    if (c < C) {
        const int64_t base = (int64_t)b * HW * C + c;
        int p = w;
        for (; p + 28 < HW; p += 32) {
            bf16_t hv[8], lv[8] = {};
#pragma unroll
            for (int u = 0; u < 8; ++u) hv[u] = xh[base + (int64_t)(p + 4 * u) * C];
            if (xl) {  // (one uniform branch: no select right after each load)
#pragma unroll
                for (int u = 0; u < 8; ++u) lv[u] = xl[base + (int64_t)(p + 4 * u) * C];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) s += bf2f(hv[u]) + (xl ? bf2f(lv[u]) : 0.f);
        }
        for (; p < HW; p += 4) {
            const int64_t k = base + (int64_t)p * C;
            s += bf2f(xh[k]) + (xl ? bf2f(xl[k]) : 0.f);
        }
    }
    red[w][lane] = s;
    __syncthreads();
    if (w == 0 && c < C)
        h[(int64_t)b * C + c] = ((red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane])) / (float)HW;
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
// A block covers 64 channels (one per lane: each row segment is one 256-byte
// access per wave) and BN_RPB rows (its four waves take every fourth row).
// Statistics come in two launches: per row block, partial sums written to
// part[row block][2][C]; the kernel that applies them first adds up the
// partials of its own channels (in row-block order, so the result does not
// depend on scheduling).  Requires C % 64 == 0.
constexpr int BN_RPB = 32;
constexpr int BN_PER = BN_RPB / 4;  // rows per wave

// Sums the S split-K slices ws[z][row][c] of the convolution that produced
// z (S = 1: z was written by the convolution itself), stores the sum to z,
// and writes partial sums of (z - shift) and (z - shift)^2 per channel, with
// shift = the channel's value at row 0 (keeps the one-pass variance well
// conditioned; every block computes it the same way).  S is a template
// parameter (up to 8) so that all S x BN_PER loads of a lane are in flight
// together; the slices are added in index order.
template <int S>
__global__ void __launch_bounds__(256) bn_fwd_stats(const float* __restrict__ ws, float* __restrict__ z, int rows,
                                                    int C, float* __restrict__ part) {
    __shared__ float red[4][2][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane;
    const int r0 = blockIdx.y * BN_RPB;
    const int64_t full = (int64_t)rows * C;
    const float* src = S > 1 ? ws : z;
    float x[S][BN_PER + 1];  // [slice][row], the last row is row 0 (the shift)
#pragma unroll
    for (int k = 0; k < S; ++k) {
#pragma unroll
        for (int i = 0; i < BN_PER; ++i) {
            const int r = min(r0 + w + 4 * i, rows - 1);  // rows past the end load the last row and are skipped
            x[k][i] = src[k * full + (int64_t)r * C + c];
        }
        x[k][BN_PER] = src[k * full + c];
    }
    float v[BN_PER + 1];
#pragma unroll
    for (int i = 0; i <= BN_PER; ++i) {
        v[i] = x[0][i];
#pragma unroll
        for (int k = 1; k < S; ++k) v[i] += x[k][i];
    }
    const float sh = v[BN_PER];
    float sm = 0.f, sq = 0.f;
#pragma unroll
    for (int i = 0; i < BN_PER; ++i) {
        const int r = r0 + w + 4 * i;
        if (r < rows) {
            if (S > 1) z[(int64_t)r * C + c] = v[i];
            const float d = v[i] - sh;
            sm += d;
            sq = fmaf(d, d, sq);
        }
    }
    red[w][0][lane] = sm;
    red[w][1][lane] = sq;
    __syncthreads();
    if (w < 2) {
        const float t = (red[0][w][lane] + red[1][w][lane]) + (red[2][w][lane] + red[3][w][lane]);
        part[((int64_t)blockIdx.y * 2 + w) * C + c] = t;
    }
}

// y = relu(gamma (z - mean) rstd + beta [+ residual]) -> fp32 and/or (hi, lo)
// bf16.  Each block first completes the statistics of its 64 channels from
// the nrb partial rows (fp64, its waves over interleaved partial rows, then
// in wave order); row block 0 also stores mean and rstd for the backward.
__global__ void __launch_bounds__(256) bn_fwd_apply(const float* __restrict__ z, const float* __restrict__ part,
                                                    int nrb, int rows, int C, float eps, const float* __restrict__ g,
                                                    const float* __restrict__ beta, const float* __restrict__ resf,
                                                    const bf16_t* __restrict__ resh, const bf16_t* __restrict__ resl,
                                                    int relu, float* __restrict__ mean_out,
                                                    float* __restrict__ rstd_out, float* __restrict__ yf,
                                                    bf16_t* __restrict__ yh, bf16_t* __restrict__ yl) {
    __shared__ double red[4][2][64];
    __shared__ float stat[2][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane;
    double s1 = 0.0, s2 = 0.0;
    int k = w;
    for (; k + 12 < nrb; k += 16) {  // four partial rows in flight
        float a[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            a[u] = part[((int64_t)(k + 4 * u) * 2 + 0) * C + c];
            b[u] = part[((int64_t)(k + 4 * u) * 2 + 1) * C + c];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            s1 += a[u];
            s2 += b[u];
        }
    }
    for (; k < nrb; k += 4) {
        s1 += part[((int64_t)k * 2 + 0) * C + c];
        s2 += part[((int64_t)k * 2 + 1) * C + c];
    }
    red[w][0][lane] = s1;
    red[w][1][lane] = s2;
    __syncthreads();
    if (w == 0) {
        const double sm = (red[0][0][lane] + red[1][0][lane]) + (red[2][0][lane] + red[3][0][lane]);
        const double sq = (red[0][1][lane] + red[1][1][lane]) + (red[2][1][lane] + red[3][1][lane]);
        const double n = rows, m = sm / n;
        double var = sq / n - m * m;
        var = var < 0.0 ? 0.0 : var;
        const float mean = (float)(z[c] + m), rstd = (float)(1.0 / sqrt(var + eps));
        stat[0][lane] = mean;
        stat[1][lane] = rstd;
        if (blockIdx.y == 0) {
            mean_out[c] = mean;
            rstd_out[c] = rstd;
        }
    }
    __syncthreads();
    const float mean = stat[0][lane], rstd = stat[1][lane];
    const float gs = g[c] * rstd, bs = fmaf(-mean, gs, beta[c]);  // y = z gs + bs
    const int r0 = blockIdx.y * BN_RPB;
    // every row's operands first (rows clamped into the tensor), then the
    // guarded stores: a bound test before each row's loads serialises them
    // (each operand's loads in one uniform branch, so that no value needs a
    // select right after its load)
    int64_t ov[BN_PER];
    float zv[BN_PER], rv[BN_PER] = {};
    bf16_t hv[BN_PER] = {}, lv[BN_PER] = {};
#pragma unroll
    for (int i = 0; i < BN_PER; ++i) {
        ov[i] = (int64_t)min(r0 + w + 4 * i, rows - 1) * C + c;
        zv[i] = z[ov[i]];
    }
    if (resf) {
#pragma unroll
        for (int i = 0; i < BN_PER; ++i) rv[i] = resf[ov[i]];
    }
    if (resh) {
#pragma unroll
        for (int i = 0; i < BN_PER; ++i) hv[i] = resh[ov[i]];
    }
    if (resl) {
#pragma unroll
        for (int i = 0; i < BN_PER; ++i) lv[i] = resl[ov[i]];
    }
#pragma unroll
    for (int i = 0; i < BN_PER; ++i) {
        const int r = r0 + w + 4 * i;
        if (r >= rows) break;
        const int64_t o = (int64_t)r * C + c;
        float v = fmaf(zv[i], gs, bs);
        if (resf) v += rv[i];
        if (resh) v += bf2f(hv[i]) + (resl ? bf2f(lv[i]) : 0.f);
        if (relu) v = v > 0.f ? v : 0.f;
        if (yf) yf[o] = v;
        if (yh) split_store(yh, yl, o, v);
    }
}

// Backward partial sums per row block: dbeta = sum dy, dgamma = sum dy xhat,
// with dy = gout [* (mask > 0)] (the ReLU of the norm's output, when mask is
// set), which is also stored to dy_out when that is set.
__global__ void __launch_bounds__(256) bn_bwd_stats(const float* __restrict__ gout, const bf16_t* __restrict__ mask,
                                                    float* __restrict__ dy_out, const float* __restrict__ z,
                                                    const float* __restrict__ mean, const float* __restrict__ rstd,
                                                    int rows, int C, float* __restrict__ part) {
    __shared__ float red[4][2][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane;
    const int r0 = blockIdx.y * BN_RPB;
    const float m = mean[c], rs = rstd[c];
    float d[BN_PER], x[BN_PER];
#pragma unroll
    for (int i = 0; i < BN_PER; ++i) {
        const int r = r0 + w + 4 * i;
        const int64_t o = (int64_t)r * C + c;
        d[i] = r < rows ? gout[o] : 0.f;
        x[i] = r < rows ? z[o] : 0.f;
        if (mask && r < rows && !(bf2f(mask[o]) > 0.f)) d[i] = 0.f;
    }
    float sg = 0.f, sb = 0.f;
#pragma unroll
    for (int i = 0; i < BN_PER; ++i) {
        const int r = r0 + w + 4 * i;
        if (r < rows) {
            if (dy_out) dy_out[(int64_t)r * C + c] = d[i];
            sb += d[i];
            sg = fmaf(d[i], (x[i] - m) * rs, sg);
        }
    }
    red[w][0][lane] = sg;
    red[w][1][lane] = sb;
    __syncthreads();
    if (w < 2) {
        const float t = (red[0][w][lane] + red[1][w][lane]) + (red[2][w][lane] + red[3][w][lane]);
        part[((int64_t)blockIdx.y * 2 + w) * C + c] = t;
    }
}

// dz = gamma rstd (dy - dbeta / N - xhat dgamma / N) -> fp32 and/or bf16, dy as
// in bn_bwd_stats.  Each block completes dgamma and dbeta of its channels from
// the partial rows (in row-block order); row block 0 stores them.
__global__ void __launch_bounds__(256) bn_bwd_apply(const float* __restrict__ gout, const bf16_t* __restrict__ mask,
                                                    const float* __restrict__ z, const float* __restrict__ mean,
                                                    const float* __restrict__ rstd, const float* __restrict__ g,
                                                    const float* __restrict__ part, int nrb, int rows, int C,
                                                    float* __restrict__ dg_out, float* __restrict__ db_out,
                                                    float* __restrict__ dzf, bf16_t* __restrict__ dzb) {
    __shared__ float red[4][2][64];
    __shared__ float stat[2][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane;
    float sg = 0.f, sb = 0.f;
    int k = w;
    for (; k + 12 < nrb; k += 16) {  // four partial rows in flight
        float a[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            a[u] = part[((int64_t)(k + 4 * u) * 2 + 0) * C + c];
            b[u] = part[((int64_t)(k + 4 * u) * 2 + 1) * C + c];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            sg += a[u];
            sb += b[u];
        }
    }
    for (; k < nrb; k += 4) {
        sg += part[((int64_t)k * 2 + 0) * C + c];
        sb += part[((int64_t)k * 2 + 1) * C + c];
    }
    red[w][0][lane] = sg;
    red[w][1][lane] = sb;
    __syncthreads();
    if (w == 0) {
        const float tg = (red[0][0][lane] + red[1][0][lane]) + (red[2][0][lane] + red[3][0][lane]);
        const float tb = (red[0][1][lane] + red[1][1][lane]) + (red[2][1][lane] + red[3][1][lane]);
        stat[0][lane] = tg;
        stat[1][lane] = tb;
        if (blockIdx.y == 0) {
            dg_out[c] = tg;
            db_out[c] = tb;
        }
    }
    __syncthreads();
    const float inv = 1.f / (float)rows, m = mean[c], rs = rstd[c];
    const float dgn = stat[0][lane] * inv, dbn = stat[1][lane] * inv, gr = g[c] * rs;
    const int r0 = blockIdx.y * BN_RPB;
    // every row's operands first (rows clamped into the tensor), then the guarded stores
    int64_t ov[BN_PER];
    float dv[BN_PER], zv[BN_PER];
    bf16_t mv[BN_PER];
#pragma unroll
    for (int i = 0; i < BN_PER; ++i) {
        ov[i] = (int64_t)min(r0 + w + 4 * i, rows - 1) * C + c;
        dv[i] = gout[ov[i]];
        zv[i] = z[ov[i]];
        mv[i] = 0x3F80;  // 1.0
    }
    if (mask) {  // (one uniform branch: no select right after each load)
#pragma unroll
        for (int i = 0; i < BN_PER; ++i) mv[i] = mask[ov[i]];
    }
#pragma unroll
    for (int i = 0; i < BN_PER; ++i) {
        const int r = r0 + w + 4 * i;
        if (r >= rows) break;
        const int64_t o = (int64_t)r * C + c;
        float d = dv[i];
        if (mask && !(bf2f(mv[i]) > 0.f)) d = 0.f;
        const float xh = (zv[i] - m) * rs;
        const float v = gr * (d - dbn - xh * dgn);
        if (dzf) dzf[o] = v;
        if (dzb) dzb[o] = f2bf(v);
    }
}

__global__ void __launch_bounds__(256) to_bf16(const float* __restrict__ x, bf16_t* __restrict__ y, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        y[i] = f2bf(x[i]);
}

inline int grid_for(int64_t n) { return (int)std::min<int64_t>(cdiv(n, 256), 8192); }

}  // namespace

fo_status launch_nchw_to_nhwc(const StepIn* in, bf16_t* y, int B, int C, int HW, hipStream_t s) {
    hipLaunchKernelGGL(nchw_to_nhwc, dim3(cdiv(HW, 32), cdiv(C, 32), B), dim3(256), 0, s, in, y, B, C, HW);
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
    FO_CHECK(H % 2 == 0 && W % 2 == 0, "max pool backward: %d x %d input (even sizes only)", H, W);
    hipLaunchKernelGGL(maxpool_relu_bwd, dim3(grid_for((int64_t)B * (H / 2) * (W / 2) * C)), dim3(256), 0, s, dy,
                       arg, y, dxf, dxb, B, H, W, C);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_gap_fwd(const bf16_t* xh, const bf16_t* xl, float* h, int B, int HW, int C, hipStream_t s) {
    hipLaunchKernelGGL(gap_fwd, dim3(cdiv(C, 64), B), dim3(256), 0, s, xh, xl, h, B, HW, C);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_gap_relu_bwd(const float* dh, const bf16_t* y, float* dxf, int B, int HW, int C, hipStream_t s) {
    hipLaunchKernelGGL(gap_relu_bwd, dim3(grid_for((int64_t)B * HW * C)), dim3(256), 0, s, dh, y, dxf, B, HW, C);
    FO_LAUNCHED();
    return FO_OK;
}

size_t bn_ws_floats(int rows, int C) { return (size_t)cdiv(rows, BN_RPB) * 2 * C; }

fo_status launch_bn_fwd_stats(const float* ws, int S, float* z, int rows, int C, float* part, hipStream_t s) {
    FO_CHECK(C % 64 == 0 && rows >= 1, "batch norm: %d channels (multiples of 64), %d rows", C, rows);
    FO_CHECK(S == 1 || ws != nullptr, "batch norm: %d slices without a workspace", S);
    const dim3 grid(C / 64, cdiv(rows, BN_RPB));
    switch (S) {
        case 1: hipLaunchKernelGGL(bn_fwd_stats<1>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        case 2: hipLaunchKernelGGL(bn_fwd_stats<2>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        case 3: hipLaunchKernelGGL(bn_fwd_stats<3>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        case 4: hipLaunchKernelGGL(bn_fwd_stats<4>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        case 5: hipLaunchKernelGGL(bn_fwd_stats<5>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        case 6: hipLaunchKernelGGL(bn_fwd_stats<6>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        case 7: hipLaunchKernelGGL(bn_fwd_stats<7>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        case 8: hipLaunchKernelGGL(bn_fwd_stats<8>, grid, dim3(256), 0, s, ws, z, rows, C, part); break;
        default: FO_CHECK(false, "batch norm: %d split-K slices (at most 8)", S);
    }
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_bn_fwd_apply(const float* z, const float* part, int rows, int C, float eps, const float* g,
                              const float* beta, const float* resf, const bf16_t* resh, const bf16_t* resl, bool relu,
                              float* mean, float* rstd, float* yf, bf16_t* yh, bf16_t* yl, hipStream_t s) {
    FO_CHECK(C % 64 == 0 && rows >= 1, "batch norm: %d channels (multiples of 64), %d rows", C, rows);
    const int nrb = (int)cdiv(rows, BN_RPB);
    hipLaunchKernelGGL(bn_fwd_apply, dim3(C / 64, nrb), dim3(256), 0, s, z, part, nrb, rows, C, eps, g, beta, resf,
                       resh, resl, relu ? 1 : 0, mean, rstd, yf, yh, yl);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_bn_bwd(const float* gout, const bf16_t* mask, float* dy_out, const float* z, const float* mean,
                        const float* rstd, const float* g, int rows, int C, float* dg, float* db, float* dzf,
                        bf16_t* dzb, float* part, hipStream_t s) {
    FO_CHECK(C % 64 == 0 && rows >= 1, "batch norm: %d channels (multiples of 64), %d rows", C, rows);
    const int nrb = (int)cdiv(rows, BN_RPB);
    hipLaunchKernelGGL(bn_bwd_stats, dim3(C / 64, nrb), dim3(256), 0, s, gout, mask, dy_out, z, mean, rstd, rows, C,
                       part);
    hipLaunchKernelGGL(bn_bwd_apply, dim3(C / 64, nrb), dim3(256), 0, s, gout, mask, z, mean, rstd, g, part, nrb, rows,
                       C, dg, db, dzf, dzb);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_to_bf16(const float* x, bf16_t* y, int64_t n, hipStream_t s) {
    hipLaunchKernelGGL(to_bf16, dim3(grid_for(n)), dim3(256), 0, s, x, y, n);
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
