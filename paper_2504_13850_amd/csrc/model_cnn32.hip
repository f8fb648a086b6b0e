// Config 1: the tiny fp32 CNN server network, one training iteration of the
// activation branch of Alg. 4:
//   conv3x3 32->64 + bias + ReLU, maxpool 2x2, conv3x3 64->64 + bias + ReLU,
//   global average pool, linear 64->10, mean cross-entropy, backward, SGD.
// Everything is fp32 and NCHW (the boundary layout).  The network is small
// and launch-bound, so the kernels are direct loops (thread per output,
// block-reduced weight gradients); the activation gradient of the first conv
// is never formed.
#include "model.h"

namespace fo {

namespace {

constexpr int C0 = 32, C1 = 64, C2 = 64, H0 = 16, W0 = 16, H1 = 8, W1 = 8, NCLS = 10;
constexpr int64_t kW1 = (int64_t)C1 * 9 * C0, kW2 = (int64_t)C2 * 9 * C1, kFc = (int64_t)NCLS * C2;
constexpr int64_t kParams = kW1 + C1 + kW2 + C2 + kFc + NCLS;

struct Plan {
    // parameter offsets (library layout)
    const float *w1, *b1, *w2, *b2, *wf, *bf;
    float *gw1, *gb1, *gw2, *gb2, *gwf, *gbf;
    // activations [B, C, H, W]
    float *y1;       // conv1 + ReLU, [B,64,16,16]
    float *p1;       // pooled,       [B,64,8,8]
    uint8_t *arg1;   // argmax of each pool window (0..3)
    float *y2;       // conv2 + ReLU, [B,64,8,8]
    float *h;        // GAP,          [B,64]
    float *dz;       // dlogits       [B,10]
    float *dh;       // [B,64]
    float *d2;       // dpre conv2    [B,64,8,8]
    float *dp1;      // d pooled      [B,64,8,8]
    float *d1;       // dpre conv1    [B,64,16,16]
};

// y[b,co,y,x] = relu(bias[co] + sum_{ci,ky,kx} x[b,ci,y+ky-1,x+kx-1] w[co,ky,kx,ci]);
// x is the step's batch (in->x) when in is set
// part[u] += sum over channels c = u, u + 8, ... < n of a[c sa] b[c sb]: eight
// independent chains whose loads are in flight together (a single chain over
// the channels waits for each pair of loads in turn).
__device__ __forceinline__ void chan_dot(const float* __restrict__ a, int64_t sa, const float* __restrict__ b,
                                         int64_t sb, int n, float (&part)[8]) {
    int c = 0;
    for (; c + 8 <= n; c += 8) {
        float av[8], bv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            av[u] = a[(c + u) * sa];
            bv[u] = b[(c + u) * sb];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) part[u] = fmaf(av[u], bv[u], part[u]);
    }
    for (; c < n; ++c) part[c & 7] = fmaf(a[c * sa], b[c * sb], part[c & 7]);
}

__global__ void conv3x3_fwd_relu(const float* __restrict__ x_, const StepIn* __restrict__ in,
                                 const float* __restrict__ w, const float* __restrict__ bias, float* __restrict__ y,
                                 int B, int Ci, int Co, int H, int W) {
    const float* __restrict__ x = in ? static_cast<const float*>(in->x) : x_;
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    int total = B * Co * H * W;
    if (idx >= total) return;
    int xx = idx % W, yy = (idx / W) % H, co = (idx / (W * H)) % Co, b = idx / (W * H * Co);
    float acc = bias[co];
    float part[8] = {};
    for (int ky = 0; ky < 3; ++ky) {
        int iy = yy + ky - 1;
        if (iy < 0 || iy >= H) continue;
        for (int kx = 0; kx < 3; ++kx) {
            int ix = xx + kx - 1;
            if (ix < 0 || ix >= W) continue;
            const float* wp = w + ((int64_t)co * 9 + ky * 3 + kx) * Ci;
            const float* xp = x + ((int64_t)b * Ci * H + iy) * W + ix;
            chan_dot(xp, (int64_t)H * W, wp, 1, Ci, part);
        }
    }
    acc += ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
    y[idx] = acc > 0.f ? acc : 0.f;
}

// 2x2/2 max pool; the first maximum in row-major window order wins.
__global__ void maxpool2_fwd(const float* __restrict__ x, float* __restrict__ y, uint8_t* __restrict__ arg,
                             int BC, int H, int W) {
    int Ho = H / 2, Wo = W / 2;
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= BC * Ho * Wo) return;
    int ox = idx % Wo, oy = (idx / Wo) % Ho, bc = idx / (Wo * Ho);
    const float* p = x + ((int64_t)bc * H + 2 * oy) * W + 2 * ox;
    float v[4] = {p[0], p[1], p[W], p[W + 1]};
    int a = 0;
    for (int i = 1; i < 4; ++i)
        if (v[i] > v[a]) a = i;
    y[idx] = v[a];
    arg[idx] = (uint8_t)a;
}

// h[b,c] = mean over H*W of x[b,c]
__global__ void gap_fwd(const float* __restrict__ x, float* __restrict__ h, int BC, int HW) {
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= BC) return;
    float s = 0.f;
    for (int i = 0; i < HW; ++i) s += x[(int64_t)idx * HW + i];
    h[idx] = s / (float)HW;
}

// z[b,o] = bias[o] + sum_i h[b,i] w[o,i]
__global__ void linear_fwd(const float* __restrict__ h, const float* __restrict__ w,
                           const float* __restrict__ bias, float* __restrict__ z, int B, int I, int O) {
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= B * O) return;
    int o = idx % O, b = idx / O;
    float acc = bias[o];
    for (int i = 0; i < I; ++i) acc = fmaf(h[(int64_t)b * I + i], w[(int64_t)o * I + i], acc);
    z[idx] = acc;
}

// Linear backward: gw[o,i] = sum_b dz[b,o] h[b,i]; gb[o] = sum_b dz[b,o];
// dh[b,i] = sum_o dz[b,o] w[o,i].
__global__ void linear_bwd(const float* __restrict__ dz, const float* __restrict__ h,
                           const float* __restrict__ w, float* __restrict__ gw, float* __restrict__ gb,
                           float* __restrict__ dh, int B, int I, int O) {
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx < O * I) {
        int i = idx % I, o = idx / I;
        float s = 0.f;
        for (int b = 0; b < B; ++b) s = fmaf(dz[(int64_t)b * O + o], h[(int64_t)b * I + i], s);
        gw[idx] = s;
    }
    if (idx < O) {
        float s = 0.f;
        for (int b = 0; b < B; ++b) s += dz[(int64_t)b * O + idx];
        gb[idx] = s;
    }
    if (idx < B * I) {
        int i = idx % I, b = idx / I;
        float s = 0.f;
        for (int o = 0; o < O; ++o) s = fmaf(dz[(int64_t)b * O + o], w[(int64_t)o * I + i], s);
        dh[idx] = s;
    }
}

// d[b,c,y,x] = dh[b,c] / HW * [y2 > 0]
__global__ void gap_relu_bwd(const float* __restrict__ dh, const float* __restrict__ y, float* __restrict__ d,
                             int BC, int HW) {
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= BC * HW) return;
    float g = dh[idx / HW] / (float)HW;
    d[idx] = y[idx] > 0.f ? g : 0.f;
}

// Weight and bias gradient of a 3x3 pad-1 conv: one block per (co, ci),
// threads stride over (b, y, x), nine partial sums, block reduction.
// (x is the step's batch, in->x, when in is set)
__global__ void __launch_bounds__(256) conv3x3_wgrad(const float* __restrict__ d, const float* __restrict__ x_,
                                                     const StepIn* __restrict__ in, float* __restrict__ gw,
                                                     float* __restrict__ gb, int B, int Ci, int Co, int H, int W) {
    const float* __restrict__ x = in ? static_cast<const float*>(in->x) : x_;
    int ci = blockIdx.x % Ci, co = blockIdx.x / Ci;
    float acc[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) acc[t] = 0.f;
    float bacc = 0.f;
    int HW = H * W;
    // pixels p = t + 256 (2 q + h), h = 0, 1: each pair's twenty loads (the
    // gradient and nine taps of both, taps at indices clamped into the image)
    // issued together, the taps outside the image zeroed afterwards
    const int P = B * HW;
    for (int p0 = threadIdx.x; p0 < P; p0 += 2 * blockDim.x) {
        float g[2], v[2][9];
        int yy[2], xx[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int p = min(p0 + h * (int)blockDim.x, P - 1);
            const int b = p / HW;
            yy[h] = (p / W) % H;
            xx[h] = p % W;
            g[h] = d[((int64_t)b * Co + co) * HW + yy[h] * W + xx[h]];
            const float* xp = x + ((int64_t)b * Ci + ci) * HW;
#pragma unroll
            for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                for (int kx = 0; kx < 3; ++kx)
                    v[h][ky * 3 + kx] =
                        xp[min(max(yy[h] + ky - 1, 0), H - 1) * W + min(max(xx[h] + kx - 1, 0), W - 1)];
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (p0 + h * (int)blockDim.x >= P) break;
            bacc += g[h];
#pragma unroll
            for (int ky = 0; ky < 3; ++ky) {
                const int iy = yy[h] + ky - 1;
#pragma unroll
                for (int kx = 0; kx < 3; ++kx) {
                    const int ix = xx[h] + kx - 1;
                    const float vv = (iy >= 0 && iy < H && ix >= 0 && ix < W) ? v[h][ky * 3 + kx] : 0.f;
                    acc[ky * 3 + kx] = fmaf(g[h], vv, acc[ky * 3 + kx]);
                }
            }
        }
    }
    __shared__ float red[10][256];
#pragma unroll
    for (int t = 0; t < 9; ++t) red[t][threadIdx.x] = acc[t];
    red[9][threadIdx.x] = bacc;
    __syncthreads();
    for (int s = blockDim.x / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s)
            for (int t = 0; t < 10; ++t) red[t][threadIdx.x] += red[t][threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x < 9) gw[((int64_t)co * 9 + threadIdx.x) * Ci + ci] = red[threadIdx.x][0];
    if (threadIdx.x == 0 && ci == 0) gb[co] = red[9][0];
}

// dx[b,ci,y,x] = sum_{co,ky,kx} d[b,co,y-ky+1,x-kx+1] w[co,ky,kx,ci]
__global__ void conv3x3_dgrad(const float* __restrict__ d, const float* __restrict__ w, float* __restrict__ dx,
                              int B, int Ci, int Co, int H, int W) {
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= B * Ci * H * W) return;
    int xx = idx % W, yy = (idx / W) % H, ci = (idx / (W * H)) % Ci, b = idx / (W * H * Ci);
    float part[8] = {};
    for (int ky = 0; ky < 3; ++ky) {
        int oy = yy - ky + 1;
        if (oy < 0 || oy >= H) continue;
        for (int kx = 0; kx < 3; ++kx) {
            int ox = xx - kx + 1;
            if (ox < 0 || ox >= W) continue;
            const float* dp = d + ((int64_t)b * Co * H + oy) * W + ox;
            const float* wp = w + (int64_t)(ky * 3 + kx) * Ci + ci;
            chan_dot(dp, (int64_t)H * W, wp, (int64_t)9 * Ci, Co, part);
        }
    }
    dx[idx] = ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
}

// d1[b,c,Y,X] = dp[b,c,Y/2,X/2] if (Y,X) was the window's argmax, times [y1 > 0]
__global__ void maxpool2_relu_bwd(const float* __restrict__ dp, const uint8_t* __restrict__ arg,
                                  const float* __restrict__ y, float* __restrict__ d, int BC, int H, int W) {
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= BC * H * W) return;
    int xx = idx % W, yy = (idx / W) % H, bc = idx / (W * H);
    int o = (bc * (H / 2) + yy / 2) * (W / 2) + xx / 2;
    int pos = (yy & 1) * 2 + (xx & 1);
    float g = (arg[o] == pos) ? dp[o] : 0.f;
    d[idx] = y[idx] > 0.f ? g : 0.f;
}

inline int nb(int64_t n) { return (int)cdiv(n, 256); }

size_t ws_bytes(const fo_model* m) {
    size_t B = (size_t)m->max_batch, s = 0;
    auto add = [&](size_t b) { s += (b + 255) & ~size_t(255); };
    add(sizeof(Plan));
    add(4 * B * C1 * H0 * W0);  // y1
    add(4 * B * C1 * H1 * W1);  // p1
    add(B * C1 * H1 * W1);      // arg1
    add(4 * B * C2 * H1 * W1);  // y2
    add(4 * B * C2);            // h
    add(4 * B * NCLS);          // dz
    add(4 * B * C2);            // dh
    add(4 * B * C2 * H1 * W1);  // d2
    add(4 * B * C1 * H1 * W1);  // dp1
    add(4 * B * C1 * H0 * W0);  // d1
    return s;
}

fo_status init(fo_model* m) {
    Plan* P = new (std::nothrow) Plan();
    if (!P) return FO_ENOMEM;
    m->plan = P;
    size_t B = (size_t)m->max_batch;
    const float* p = m->params;
    float* g = m->grads;
    P->w1 = p; P->gw1 = g; p += kW1; g += kW1;
    P->b1 = p; P->gb1 = g; p += C1; g += C1;
    P->w2 = p; P->gw2 = g; p += kW2; g += kW2;
    P->b2 = p; P->gb2 = g; p += C2; g += C2;
    P->wf = p; P->gwf = g; p += kFc; g += kFc;
    P->bf = p; P->gbf = g;
    Arena& a = m->arena;
    a.take<char>(sizeof(Plan));
    P->y1 = a.take<float>(B * C1 * H0 * W0);
    P->p1 = a.take<float>(B * C1 * H1 * W1);
    P->arg1 = a.take<uint8_t>(B * C1 * H1 * W1);
    P->y2 = a.take<float>(B * C2 * H1 * W1);
    P->h = a.take<float>(B * C2);
    P->dz = a.take<float>(B * NCLS);
    P->dh = a.take<float>(B * C2);
    P->d2 = a.take<float>(B * C2 * H1 * W1);
    P->dp1 = a.take<float>(B * C1 * H1 * W1);
    P->d1 = a.take<float>(B * C1 * H0 * W0);
    if (!P->d1) {
        set_error("cnn32: workspace arena too small");
        return FO_ENOMEM;
    }
    return FO_OK;
}

fo_status step(fo_model* m, const fo_acts* acts, const int32_t* labels) {
    Plan* P = (Plan*)m->plan;
    hipStream_t s = m->stream;
    const int B = acts->batch;  // (the batch's data is read through m->dev_in)
    // forward (Alg. 4: forward pass of M_s, loss f_s)
    hipLaunchKernelGGL(conv3x3_fwd_relu, dim3(nb((int64_t)B * C1 * H0 * W0)), dim3(256), 0, s, nullptr, m->dev_in,
                       P->w1, P->b1,
                       P->y1, B, C0, C1, H0, W0);
    hipLaunchKernelGGL(maxpool2_fwd, dim3(nb((int64_t)B * C1 * H1 * W1)), dim3(256), 0, s, P->y1, P->p1, P->arg1,
                       B * C1, H0, W0);
    hipLaunchKernelGGL(conv3x3_fwd_relu, dim3(nb((int64_t)B * C2 * H1 * W1)), dim3(256), 0, s, P->p1, nullptr,
                       P->w2, P->b2,
                       P->y2, B, C1, C2, H1, W1);
    hipLaunchKernelGGL(gap_fwd, dim3(nb(B * C2)), dim3(256), 0, s, P->y2, P->h, B * C2, H1 * W1);
    hipLaunchKernelGGL(linear_fwd, dim3(nb(B * NCLS)), dim3(256), 0, s, P->h, P->wf, P->bf, m->logits, B, C2, NCLS);
    FO_LAUNCHED();
    fo_status st = launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, NCLS, s);
    if (st != FO_OK) return st;
    // backward (Alg. 4: backward pass of M_s)
    int64_t lin_threads = (int64_t)(NCLS * C2 > B * C2 ? NCLS * C2 : B * C2);
    hipLaunchKernelGGL(linear_bwd, dim3(nb(lin_threads)), dim3(256), 0, s, P->dz, P->h, P->wf, P->gwf, P->gbf, P->dh,
                       B, C2, NCLS);
    hipLaunchKernelGGL(gap_relu_bwd, dim3(nb((int64_t)B * C2 * H1 * W1)), dim3(256), 0, s, P->dh, P->y2, P->d2,
                       B * C2, H1 * W1);
    hipLaunchKernelGGL(conv3x3_wgrad, dim3(C2 * C1), dim3(256), 0, s, P->d2, P->p1, nullptr, P->gw2, P->gb2, B, C1,
                       C2, H1,
                       W1);
    hipLaunchKernelGGL(conv3x3_dgrad, dim3(nb((int64_t)B * C1 * H1 * W1)), dim3(256), 0, s, P->d2, P->w2, P->dp1, B,
                       C1, C2, H1, W1);
    hipLaunchKernelGGL(maxpool2_relu_bwd, dim3(nb((int64_t)B * C1 * H0 * W0)), dim3(256), 0, s, P->dp1, P->arg1,
                       P->y1, P->d1, B * C1, H0, W0);
    hipLaunchKernelGGL(conv3x3_wgrad, dim3(C1 * C0), dim3(256), 0, s, P->d1, nullptr, m->dev_in, P->gw1, P->gb1, B,
                       C0, C1, H0, W0);
    FO_LAUNCHED();
    // SGD (Alg. 4: theta_s <- theta_s - gamma_s grad)
    return launch_sgd(m->params, m->grads, nullptr, nullptr, nullptr, m->n_params, m->lr, 0.f, s);
}

void destroy(fo_model* m) {
    delete (Plan*)m->plan;
    m->plan = nullptr;
}

}  // namespace

int64_t cnn32_param_count() { return kParams; }

const Family* family_cnn32() {
    static const Family f = {(int64_t)C0 * H0 * W0 * 4, ws_bytes, init, step, destroy};
    return &f;
}

}  // namespace fo
