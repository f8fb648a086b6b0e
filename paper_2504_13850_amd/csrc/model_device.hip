// Config 6: one local training iteration of a device (Alg. 1) for the VGG-16
// split of configs 2 and 5, with the auxiliary network that gives the device
// its own loss (Sec. 3.2.2):
//
//   device network M_d:   conv3x3 3->64 + ReLU, conv3x3 64->64 + ReLU, 2x2 max pool
//                         -> the activations xi [B][64][16][16] sent to the server
//   auxiliary network:    conv3x3 64->64 + ReLU on xi (a layer of the type of M_d's
//                         last layer), global average pool, dense 64 -> 10
//   local loss f_d:       mean softmax cross-entropy; backward through both
//                         networks (no gradient for the input data); SGD on the
//                         device and auxiliary parameters with rate gamma_d.
//
// Inputs are fp32 NCHW 32x32 RGB mini-batches.  The first convolution (three
// input channels, 0.23 GFLOP at B = 64) runs as a direct fp32 kernel; the
// two 64-channel convolutions run on the bf16 MFMA implicit-GEMM kernels,
// compensated in the forward, high parts in the backward, as on the server.
// Activations are NHWC internally; xi leaves as bf16 NCHW, the layout the
// server's step takes.
#include "gemm.h"
#include "model.h"

namespace fo {

fo_status launch_maxpool_fwd(const bf16_t* xh, const bf16_t* xl, bf16_t* yh, bf16_t* yl, uint8_t* arg, int B, int H,
                             int W, int C, hipStream_t s);
fo_status launch_maxpool_relu_bwd(const float* dy, const uint8_t* arg, const bf16_t* y, float* dxf, bf16_t* dxb, int B,
                                  int H, int W, int C, hipStream_t s);
fo_status launch_gap_fwd(const bf16_t* xh, const bf16_t* xl, float* h, int B, int HW, int C, hipStream_t s);
fo_status launch_gap_relu_bwd(const float* dh, const bf16_t* y, float* dxf, int B, int HW, int C, hipStream_t s);
fo_status launch_to_bf16(const float* x, bf16_t* y, int64_t n, hipStream_t s);

namespace {

#define TRY(x)                           \
    do {                                 \
        fo_status st_ = (x);             \
        if (st_ != FO_OK) return st_;    \
    } while (0)

constexpr int CI = 3, C = 64, H0 = 32, H1 = 16, NCLS = 10;
constexpr int KK = 9 * C;  // reduction length of a 64-channel 3x3 conv
// parameter offsets (library layout: conv weights [Cout][kh][kw][Cin], then bias)
constexpr int64_t W1 = 0, B1 = W1 + (int64_t)C * 9 * CI, W2 = B1 + C, B2 = W2 + (int64_t)C * KK, WA = B2 + C,
                  BA = WA + (int64_t)C * KK, WF = BA + C, BF = WF + (int64_t)NCLS * C, kParams = BF + NCLS;

// conv1 weight gradient: image rows per block of the partial-sum pass
constexpr int W1_ROWS = 4;

struct Plan {
    int B;
    bf16_t *h1h, *h1l;      // conv1 output after ReLU, NHWC [B][32][32][64]
    bf16_t *h2h, *h2l;      // conv2 output after ReLU
    bf16_t *xih, *xil;      // max pool output: the activations xi, NHWC [B][16][16][64]
    uint8_t* arg;           // the pool's winners
    bf16_t *ah, *al;        // auxiliary conv output after ReLU
    float *g, *dz, *dg;     // pooled features [B][64], dlogits, their gradient
    float *da, *dxi, *dh2f, *dh1;
    bf16_t *dab, *dh2b;
    float *splitws, *colws, *slws, *w1part;
    int split_af, split_aw, split_ad, split_2w;
};

// K slices of a product: enough for about 512 workgroups over its output
// tiles, at most max_s, each slice at least 256 long.  The weight gradients
// here have five 128 x 128 tiles (64 x 576) over K = B * H * W pixels, so they
// take up to 64 slices.
int split_for(int M, int N, int K, int max_s = 8) {
    int tiles = (int)(cdiv(M, 128) * cdiv(N, 128));
    int s = std::max(1, std::min(max_s, 512 / std::max(tiles, 1)));
    while (s > 1 && (int64_t)K / s < 256) --s;
    return s;
}

// ------------------------------------------------------------------ kernels
// conv1 forward: x = the step's batch (in->x), fp32 NCHW [B][3][32][32];
// y = ReLU(b + conv3x3(x, w)) as NHWC (high, low) bf16, one output per thread
// with the channel fastest (coalesced stores; the 27 inputs of a pixel are
// shared by its 64 threads).
__global__ void __launch_bounds__(256) conv1_fwd(const StepIn* __restrict__ in, const float* __restrict__ w,
                                                 const float* __restrict__ bias, bf16_t* __restrict__ yh,
                                                 bf16_t* __restrict__ yl, int B) {
    static_assert(C == 64, "a wave is the 64 channels of one pixel");
    const float* __restrict__ x = static_cast<const float*>(in->x);
    // the weights as [tap][channel] in LDS: a wave's 64 lanes read one row
    // (w itself is [channel][tap], 27 floats apart from lane to lane)
    __shared__ float wl[9 * CI][C];
    for (int t = threadIdx.x; t < 9 * CI * C; t += blockDim.x) wl[t % (9 * CI)][t / (9 * CI)] = w[t];
    __syncthreads();
    const int64_t total = (int64_t)B * H0 * H0 * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int co = (int)(i % C);
        const int64_t p = i / C;
        const int xx = (int)(p % H0), yy = (int)((p / H0) % H0), b = (int)(p / (H0 * H0));
        // the 27 inputs loaded together at indices clamped into the image, the
        // taps outside it skipped afterwards (a border test before each tap's
        // loads made every tap wait for its own)
        float xv[9 * CI];
#pragma unroll
        for (int ky = 0; ky < 3; ++ky)
#pragma unroll
            for (int kx = 0; kx < 3; ++kx)
#pragma unroll
                for (int ci = 0; ci < CI; ++ci)
                    xv[(ky * 3 + kx) * CI + ci] =
                        x[(((int64_t)b * CI + ci) * H0 + min(max(yy + ky - 1, 0), H0 - 1)) * H0 +
                          min(max(xx + kx - 1, 0), H0 - 1)];
        float acc = bias[co];
#pragma unroll
        for (int ky = 0; ky < 3; ++ky) {
            const int iy = yy + ky - 1;
            if (iy < 0 || iy >= H0) continue;
#pragma unroll
            for (int kx = 0; kx < 3; ++kx) {
                const int ix = xx + kx - 1;
                if (ix < 0 || ix >= H0) continue;
#pragma unroll
                for (int ci = 0; ci < CI; ++ci)
                    acc = fmaf(xv[(ky * 3 + kx) * CI + ci], wl[(ky * 3 + kx) * CI + ci][co], acc);
            }
        }
        const float v = acc > 0.f ? acc : 0.f;
        const bf16_t h = f2bf(v);
        yh[i] = h;
        yl[i] = f2bf(v - bf2f(h));
    }
}

// The activations that leave the device: xi (high parts) NHWC -> bf16 NCHW into in->out.
__global__ void __launch_bounds__(256) acts_out_nchw(const StepIn* __restrict__ in, const bf16_t* __restrict__ xi,
                                                     int B) {
    bf16_t* __restrict__ out = static_cast<bf16_t*>(in->out);
    __shared__ bf16_t tile[32][33];
    const int b = blockIdx.z, c0 = blockIdx.y * 32, p0 = blockIdx.x * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
    constexpr int HW = H1 * H1;
    for (int r = ty; r < 32; r += 8) tile[r][tx] = xi[((int64_t)b * HW + p0 + r) * C + c0 + tx];
    __syncthreads();
    for (int r = ty; r < 32; r += 8) out[((int64_t)b * C + c0 + r) * HW + p0 + tx] = tile[tx][r];
}

// conv1 weight and bias gradients, pass 1: block = W1_ROWS image rows of one
// sample (their input rows, with the padding, staged once in LDS), lane =
// output channel co, the four waves take every fourth pixel; per lane the 27
// weight sums dh1[p][co] x[b][ci][y + ky - 1][x + kx - 1] and the bias sum
// dh1[p][co] (coalesced 256-byte rows of dh1; the input values are LDS
// broadcasts), written as part[block][28][64].
__global__ void __launch_bounds__(256) conv1_wgrad_partial(const StepIn* __restrict__ in,
                                                           const float* __restrict__ dh1, float* __restrict__ part) {
    const float* __restrict__ x = static_cast<const float*>(in->x);
    __shared__ float xs[CI][W1_ROWS + 2][H0 + 2];
    __shared__ float red[4][28][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    constexpr int strips = H0 / W1_ROWS;
    const int b = blockIdx.x / strips, y0 = (blockIdx.x % strips) * W1_ROWS;
    for (int i = threadIdx.x; i < CI * (W1_ROWS + 2) * (H0 + 2); i += 256) {
        const int ci = i / ((W1_ROWS + 2) * (H0 + 2)), r = (i / (H0 + 2)) % (W1_ROWS + 2), cx = i % (H0 + 2);
        const int iy = y0 + r - 1, ix = cx - 1;
        xs[ci][r][cx] = (iy >= 0 && iy < H0 && ix >= 0 && ix < H0) ? x[(((int64_t)b * CI + ci) * H0 + iy) * H0 + ix]
                                                                    : 0.f;
    }
    __syncthreads();
    float acc[28];
#pragma unroll
    for (int t = 0; t < 28; ++t) acc[t] = 0.f;
    for (int j = w; j < W1_ROWS * H0; j += 4) {
        const int r = j / H0, xx = j % H0;
        const float d = dh1[(((int64_t)b * H0 + y0 + r) * H0 + xx) * C + lane];
        acc[27] += d;
#pragma unroll
        for (int ky = 0; ky < 3; ++ky)
#pragma unroll
            for (int kx = 0; kx < 3; ++kx)
#pragma unroll
                for (int ci = 0; ci < CI; ++ci)
                    acc[(ky * 3 + kx) * CI + ci] = fmaf(d, xs[ci][r + ky][xx + kx], acc[(ky * 3 + kx) * CI + ci]);
    }
#pragma unroll
    for (int t = 0; t < 28; ++t) red[w][t][lane] = acc[t];
    __syncthreads();
    for (int i = threadIdx.x; i < 28 * 64; i += 256) {
        const int t = i / 64, c = i % 64;
        part[((int64_t)blockIdx.x * 28 + t) * 64 + c] = (red[0][t][c] + red[1][t][c]) + (red[2][t][c] + red[3][t][c]);
    }
}

// pass 2: one wave per output (28 x 64 of them: 27 weights and the bias per
// channel), its lanes over the partial rows, then a wave sum in a fixed order
// -> dW1 [co][ky][kx][ci] and db1.
__global__ void __launch_bounds__(256) conv1_wgrad_finish(const float* __restrict__ part, int nblk,
                                                          float* __restrict__ gw, float* __restrict__ gb) {
    const int lane = threadIdx.x & 63;
    const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (o >= 28 * 64) return;  // (uniform per wave)
    const int t = o / 64, c = o % 64;
    float s = 0.f;
    for (int k = lane; k < nblk; k += 64) s += part[((int64_t)k * 28 + t) * 64 + c];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if (lane == 0) {
        if (t < 27) gw[(int64_t)c * 27 + t] = s;  // t = (ky * 3 + kx) * 3 + ci: the [co][ky][kx][ci] order
        else gb[c] = s;
    }
}

// ------------------------------------------------------------------ GEMM wrappers
ConvGeom geom(int B, int H) {
    ConvGeom g;
    g.Bn = B; g.H = H; g.W = H; g.Ci = C;
    g.Ho = H; g.Wo = H; g.Co = C;
    g.kh = 3; g.kw = 3; g.stride = 1; g.pad = 1;
    return g;
}

// y = ReLU(b + conv3x3(x)) as a compensated implicit GEMM, NHWC (high, low) out
fo_status conv_fwd(fo_model* m, const Plan* P, int B, int H, const bf16_t* xh, const bf16_t* xl, int64_t w, int64_t b,
                   int splits, bf16_t* yh, bf16_t* yl) {
    GemmDesc d;
    d.M = B * H * H; d.N = C; d.K = KK;
    d.amode = OP_CONV_FWD; d.A = xh; d.A2 = xl;
    d.bmode = OP_RK; d.B = m->w16 + w; d.B2 = m->w16lo + w; d.ldb = KK;
    d.nseg = 3;
    d.g = geom(B, H);
    d.bias = m->params + b;
    d.act = ACT_RELU;
    d.Cb = yh; d.Cb2 = yl; d.ldcb = C;
    d.splits = splits; d.ws = P->splitws;
    return gemm(d, m->stream);
}

// dW = sum over pixels dy (x) x (weight layout [Cout][kh][kw][Cin])
fo_status conv_wgrad(fo_model* m, const Plan* P, int B, int H, const bf16_t* dyb, const bf16_t* xh, int64_t w,
                     int splits) {
    GemmDesc d;
    d.M = C; d.N = KK; d.K = B * H * H;
    d.amode = OP_KR; d.A = dyb; d.lda = C;
    d.bmode = OP_CONV_DWX; d.B = xh;
    d.g = geom(B, H);
    d.Cf = m->grads + w; d.ldcf = KK;
    d.splits = splits; d.ws = P->splitws;
    return gemm(d, m->stream);
}

// dx = conv^T(dy) (fp32), times [mask > 0] when mask is set
fo_status conv_dgrad(fo_model* m, const Plan* P, int B, int H, const bf16_t* dyb, int64_t w, const bf16_t* mask,
                     int splits, float* dxf) {
    GemmDesc d;
    d.M = B * H * H; d.N = C; d.K = KK;
    d.amode = OP_CONV_DX; d.A = dyb;
    d.bmode = OP_CONV_DXW; d.B = m->w16 + w;
    d.g = geom(B, H);
    d.mask = mask; d.ldm = C;
    d.Cf = dxf; d.ldcf = C;
    d.splits = splits; d.ws = P->splitws;
    return gemm(d, m->stream);
}

// ------------------------------------------------------------------ plan
size_t ws_bytes(const fo_model* m) {
    const size_t B = (size_t)m->max_batch, n0 = B * H0 * H0 * C, n1 = B * H1 * H1 * C;
    size_t s = 0;
    auto add = [&](size_t b) { s += (b + 255) & ~size_t(255); };
    add(sizeof(Plan) + 256);
    for (int i = 0; i < 4; ++i) add(2 * n0);            // h1, h2 (high, low)
    add(2 * n1); add(2 * n1); add(n1);                  // xi (high, low), pool winners
    add(2 * n1); add(2 * n1);                           // a (high, low)
    add(4 * B * C); add(4 * B * NCLS); add(4 * B * C);  // g, dz, dg
    add(4 * n1); add(4 * n1); add(4 * n0); add(4 * n0); // da, dxi, dh2f, dh1
    add(2 * n1); add(2 * n0);                           // dab, dh2b
    const int Bi = (int)B;
    size_t sw = 0;
    sw = std::max(sw, gemm_ws_bytes(Bi * H1 * H1, C, split_for(Bi * H1 * H1, C, 3 * KK)));
    sw = std::max(sw, gemm_ws_bytes(C, KK, split_for(C, KK, Bi * H1 * H1, 64)));
    sw = std::max(sw, gemm_ws_bytes(Bi * H1 * H1, C, split_for(Bi * H1 * H1, C, KK)));
    sw = std::max(sw, gemm_ws_bytes(C, KK, split_for(C, KK, Bi * H0 * H0, 64)));
    add(sw + 256);
    add(4 * colsum_ws_floats(Bi * H0 * H0, C));
    add(4 * small_linear_ws_floats(Bi, C, NCLS));
    add(4 * B * (H0 / W1_ROWS) * 28 * 64);
    return s;
}

fo_status init(fo_model* m) {
    Plan* P = new (std::nothrow) Plan();
    if (!P) return FO_ENOMEM;
    m->plan = P;
    const int B = m->max_batch;
    P->B = B;
    const size_t n0 = (size_t)B * H0 * H0 * C, n1 = (size_t)B * H1 * H1 * C;
    Arena& a = m->arena;
    a.take<char>(sizeof(Plan) + 256);
    P->h1h = a.take<bf16_t>(n0); P->h1l = a.take<bf16_t>(n0);
    P->h2h = a.take<bf16_t>(n0); P->h2l = a.take<bf16_t>(n0);
    P->xih = a.take<bf16_t>(n1); P->xil = a.take<bf16_t>(n1);
    P->arg = a.take<uint8_t>(n1);
    P->ah = a.take<bf16_t>(n1); P->al = a.take<bf16_t>(n1);
    P->g = a.take<float>((size_t)B * C); P->dz = a.take<float>((size_t)B * NCLS); P->dg = a.take<float>((size_t)B * C);
    P->da = a.take<float>(n1); P->dxi = a.take<float>(n1); P->dh2f = a.take<float>(n0); P->dh1 = a.take<float>(n0);
    P->dab = a.take<bf16_t>(n1); P->dh2b = a.take<bf16_t>(n0);
    P->split_af = split_for(B * H1 * H1, C, 3 * KK);
    P->split_aw = split_for(C, KK, B * H1 * H1, 64);
    P->split_ad = split_for(B * H1 * H1, C, KK);
    P->split_2w = split_for(C, KK, B * H0 * H0, 64);
    size_t sw = 0;
    sw = std::max(sw, gemm_ws_bytes(B * H1 * H1, C, P->split_af));
    sw = std::max(sw, gemm_ws_bytes(C, KK, P->split_aw));
    sw = std::max(sw, gemm_ws_bytes(B * H1 * H1, C, P->split_ad));
    sw = std::max(sw, gemm_ws_bytes(C, KK, P->split_2w));
    P->splitws = a.take<float>(sw / 4 + 64);
    P->colws = a.take<float>(colsum_ws_floats(B * H0 * H0, C));
    P->slws = a.take<float>(small_linear_ws_floats(B, C, NCLS));
    P->w1part = a.take<float>((size_t)B * (H0 / W1_ROWS) * 28 * 64);
    if (!P->w1part) {
        set_error("device model: workspace arena too small");
        return FO_ENOMEM;
    }
    return FO_OK;
}

// ------------------------------------------------------------------ the step
fo_status step(fo_model* m, const fo_acts* acts, const int32_t* labels) {
    (void)labels;  // the batch is read through m->dev_in
    Plan* P = (Plan*)m->plan;
    hipStream_t s = m->stream;
    const int B = acts->batch;
    const float* prm = m->params;
    float* grd = m->grads;
    const int rows0 = B * H0 * H0, rows1 = B * H1 * H1;
    // ---- forward of the device network M_d (Alg. 1: forward pass, activations)
    {
        const int64_t total = (int64_t)rows0 * C;
        // 1024 blocks (4 per CU) walk the outputs: each block's weight table
        // in LDS serves 16 outputs per thread (8192 blocks: 2 each, 0.335 ms
        // per step against 0.325)
        const int grid = (int)std::min<int64_t>(cdiv(total, 256), 1024);
        hipLaunchKernelGGL(conv1_fwd, dim3(grid), dim3(256), 0, s, m->dev_in, prm + W1, prm + B1, P->h1h, P->h1l, B);
        FO_LAUNCHED();
    }
    TRY(conv_fwd(m, P, B, H0, P->h1h, P->h1l, W2, B2, 1, P->h2h, P->h2l));
    TRY(launch_maxpool_fwd(P->h2h, P->h2l, P->xih, P->xil, P->arg, B, H0, H0, C, s));
    hipLaunchKernelGGL(acts_out_nchw, dim3(H1 * H1 / 32, C / 32, B), dim3(256), 0, s, m->dev_in, P->xih, B);
    FO_LAUNCHED();
    // ---- forward of the auxiliary network on xi and the local loss f_d
    TRY(conv_fwd(m, P, B, H1, P->xih, P->xil, WA, BA, P->split_af, P->ah, P->al));
    TRY(launch_gap_fwd(P->ah, P->al, P->g, B, H1 * H1, C, s));
    TRY(launch_small_linear_fwd(P->g, prm + WF, prm + BF, m->logits, B, C, NCLS, false, s));
    TRY(launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, NCLS, s));
    // ---- backward of the auxiliary network
    TRY(launch_small_linear_bwd(P->dz, P->g, prm + WF, nullptr, grd + WF, grd + BF, P->dg, B, C, NCLS, P->slws, s));
    TRY(launch_gap_relu_bwd(P->dg, P->ah, P->da, B, H1 * H1, C, s));
    TRY(launch_to_bf16(P->da, P->dab, (int64_t)rows1 * C, s));
    TRY(conv_wgrad(m, P, B, H1, P->dab, P->xih, WA, P->split_aw));
    TRY(launch_colsum(P->da, C, rows1, nullptr, C, grd + BA, P->colws, s));
    TRY(conv_dgrad(m, P, B, H1, P->dab, WA, nullptr, P->split_ad, P->dxi));
    // ---- backward of the device network (through the pool and conv2's ReLU)
    TRY(launch_maxpool_relu_bwd(P->dxi, P->arg, P->h2h, P->dh2f, P->dh2b, B, H0, H0, C, s));
    TRY(conv_wgrad(m, P, B, H0, P->dh2b, P->h1h, W2, P->split_2w));
    TRY(launch_colsum(P->dh2f, C, rows0, nullptr, C, grd + B2, P->colws, s));
    TRY(conv_dgrad(m, P, B, H0, P->dh2b, W2, P->h1h, 1, P->dh1));  // times conv1's ReLU mask
    {
        const int nblk = B * (H0 / W1_ROWS);
        hipLaunchKernelGGL(conv1_wgrad_partial, dim3(nblk), dim3(256), 0, s, m->dev_in, P->dh1, P->w1part);
        hipLaunchKernelGGL(conv1_wgrad_finish, dim3(28 * 64 / 4), dim3(256), 0, s, P->w1part, nblk, grd + W1, grd + B1);
        FO_LAUNCHED();
    }
    // ---- SGD on the device and auxiliary parameters (rate gamma_d)
    return launch_sgd(m->params, m->grads, nullptr, m->w16, m->w16lo, m->n_params, m->lr, 0.f, s);
}

void destroy(fo_model* m) {
    delete (Plan*)m->plan;
    m->plan = nullptr;
}

}  // namespace

int64_t device_param_count() { return kParams; }

const Family* family_device() {
    static const Family f = {(int64_t)CI * H0 * H0 * 4, ws_bytes, init, step, destroy};
    return &f;
}

}  // namespace fo
