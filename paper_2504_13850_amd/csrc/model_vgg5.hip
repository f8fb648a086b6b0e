// Config 9: the server part of the paper's VGG-5 (Table 4) split after its
// second pool, one training iteration of the activation branch of Alg. 4 in
// fp32 on [64, 8, 8] inputs (NCHW at the boundary):
//   conv3x3 64->64 (no bias) -> batch norm (batch statistics) -> ReLU ->
//   maxpool 2x2 -> flatten (C, H, W) -> fc 1024->128 + ReLU -> fc 128->10,
//   mean cross-entropy, backward, SGD.
// The convolution runs as an explicit im2col matrix [B*64][576] (k = (ky, kx,
// ci), the weight layout's order) times the weights on the fp32 product
// kernel, its output NHWC; batch norm is one workgroup per channel; the pool
// writes its output in (C, H, W) order so the flatten is the identity.  The
// input gradient of the convolution is never formed (nothing goes back to the
// devices).
#include "model.h"

namespace fo {

namespace {

constexpr int CI = 64, CO = 64, HW = 8, HP = 4, KC = 9 * CI, F1 = 128, NCLS = 10, NF = CO * HP * HP;
constexpr float BN_EPS = 1e-5f;
constexpr int64_t kParams = (int64_t)CO * KC + 2 * CO + (int64_t)F1 * NF + F1 + (int64_t)NCLS * F1 + NCLS;
constexpr int kMaxSlices = 16;

inline int nblk(int64_t n) { return (int)cdiv(n, 256); }

// col[r][(ky*3 + kx)*CI + ci] = x[b][ci][y+ky-1][x+kx-1] (0 outside), r = (b*8 + y)*8 + x
__global__ void __launch_bounds__(256) im2col_kernel(const StepIn* __restrict__ in, float* __restrict__ col, int B) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)B * HW * HW * KC) return;
    const int k = (int)(i % KC);
    const int64_t r = i / KC;
    const int tap = k / CI, ci = k % CI, ky = tap / 3, kx = tap % 3;
    const int b = (int)(r / (HW * HW)), y = (int)(r / HW % HW), x = (int)(r % HW);
    const int yy = y + ky - 1, xx = x + kx - 1;
    const float* X = (const float*)in->x;
    col[i] = yy >= 0 && yy < HW && xx >= 0 && xx < HW ? X[(((int64_t)b * CI + ci) * HW + yy) * HW + xx] : 0.f;
}

// Block c: batch statistics of channel c over the R rows of z (NHWC), then
// xhat, y = ReLU(gamma xhat + beta); mean and variance in two passes.
__device__ __forceinline__ float block_sum(float v, float* red) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    return red[0] + red[1] + red[2] + red[3];
}
__global__ void __launch_bounds__(256) bn5_fwd(const float* __restrict__ z, const float* __restrict__ gam,
                                               const float* __restrict__ bet, float* __restrict__ xhat,
                                               float* __restrict__ y, float* __restrict__ rstd_out, int R) {
    __shared__ float red[4];
    const int c = blockIdx.x;
    float s = 0.f;
    for (int r = threadIdx.x; r < R; r += 256) s += z[(int64_t)r * CO + c];
    const float mu = block_sum(s, red) / R;
    float v = 0.f;
    for (int r = threadIdx.x; r < R; r += 256) {
        const float d = z[(int64_t)r * CO + c] - mu;
        v = fmaf(d, d, v);
    }
    const float rs = 1.f / sqrtf(block_sum(v, red) / R + BN_EPS);
    for (int r = threadIdx.x; r < R; r += 256) {
        const int64_t o = (int64_t)r * CO + c;
        const float xh = (z[o] - mu) * rs;
        xhat[o] = xh;
        y[o] = fmaxf(fmaf(gam[c], xh, bet[c]), 0.f);
    }
    if (threadIdx.x == 0) rstd_out[c] = rs;
}

// 2x2 max pool of y (NHWC [B][8][8][64]) into p ((C, H, W) order, [B][1024]),
// with the window position of the maximum (the first one in row-major order)
__global__ void __launch_bounds__(256) pool5_fwd(const float* __restrict__ y, float* __restrict__ p,
                                                 uint8_t* __restrict__ arg, int B) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= B * NF) return;
    const int b = i / NF, c = i / (HP * HP) % CO, oy = i / HP % HP, ox = i % HP;
    float best = -INFINITY;
    int at = 0;
    for (int w = 0; w < 4; ++w) {
        const int yy = 2 * oy + (w >> 1), xx = 2 * ox + (w & 1);
        const float v = y[(((int64_t)b * HW + yy) * HW + xx) * CO + c];
        if (v > best) {
            best = v;
            at = w;
        }
    }
    p[i] = best;
    arg[i] = (uint8_t)at;
}

// d(batch-norm output) at every pre-pool position: the pooled gradient where
// the position is its window's maximum, times the ReLU mask (y > 0)
__global__ void __launch_bounds__(256) pool5_relu_bwd(const float* __restrict__ dp, const uint8_t* __restrict__ arg,
                                                      const float* __restrict__ y, float* __restrict__ dbn, int B) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)B * HW * HW * CO) return;
    const int c = (int)(i % CO);
    const int64_t r = i / CO;
    const int b = (int)(r / (HW * HW)), yy = (int)(r / HW % HW), xx = (int)(r % HW);
    const int j = ((b * CO + c) * HP + yy / 2) * HP + xx / 2;
    const int w = (yy & 1) * 2 + (xx & 1);
    dbn[i] = arg[j] == w && y[i] > 0.f ? dp[j] : 0.f;
}

// Block c: dgamma = sum dy xhat, dbeta = sum dy, dz = gamma rstd (dy - dbeta/R - xhat dgamma/R)
__global__ void __launch_bounds__(256) bn5_bwd(const float* __restrict__ dy, const float* __restrict__ xhat,
                                               const float* __restrict__ gam, const float* __restrict__ rstd,
                                               float* __restrict__ dz, float* __restrict__ dgam,
                                               float* __restrict__ dbet, int R) {
    __shared__ float red[4];
    const int c = blockIdx.x;
    float sg = 0.f, sb = 0.f;
    for (int r = threadIdx.x; r < R; r += 256) {
        const int64_t o = (int64_t)r * CO + c;
        sg = fmaf(dy[o], xhat[o], sg);
        sb += dy[o];
    }
    const float dg = block_sum(sg, red), db = block_sum(sb, red);
    const float k = gam[c] * rstd[c];
    for (int r = threadIdx.x; r < R; r += 256) {
        const int64_t o = (int64_t)r * CO + c;
        dz[o] = k * (dy[o] - db / R - xhat[o] * dg / R);
    }
    if (threadIdx.x == 0) {
        dgam[c] = dg;
        dbet[c] = db;
    }
}

struct Plan {
    const float *wc, *g, *bb, *w1, *b1, *w2, *b2;
    float *gwc, *gg, *gbb, *gw1, *gb1, *gw2, *gb2;
    float *col, *z, *xhat, *y, *rstd, *p, *f1, *dz, *df1, *dp, *dbn, *dconv, *part, *colws;
    uint8_t* arg;
    size_t part_floats;
};

size_t ws_bytes(const fo_model* m) {
    const size_t B = (size_t)m->max_batch, R = B * HW * HW;
    size_t s = 0;
    auto add = [&](size_t b) { s += (b + 255) & ~size_t(255); };
    add(sizeof(Plan));
    add(4 * R * KC);                       // col
    for (int i = 0; i < 3; ++i) add(4 * R * CO);  // z, xhat, y
    add(4 * CO);                           // rstd
    add(4 * B * NF);                       // p
    add(B * NF);                           // arg
    add(4 * B * F1);                       // f1
    add(4 * B * NCLS);                     // dz
    add(4 * B * F1);                       // df1
    add(4 * B * NF);                       // dp
    add(4 * R * CO);                       // dbn
    add(4 * R * CO);                       // dconv
    add(4 * (size_t)kMaxSlices * CO * KC); // part
    add(4 * colsum_ws_floats((int)B, F1)); // colws
    return s;
}

fo_status init(fo_model* m) {
    Plan* P = new (std::nothrow) Plan();
    if (!P) return FO_ENOMEM;
    m->plan = P;
    const size_t B = (size_t)m->max_batch, R = B * HW * HW;
    const float* p = m->params;
    float* g = m->grads;
    auto take = [&](const float*& w, float*& gw, size_t n) {
        w = p;
        gw = g;
        p += n;
        g += n;
    };
    take(P->wc, P->gwc, (size_t)CO * KC);
    take(P->g, P->gg, CO);
    take(P->bb, P->gbb, CO);
    take(P->w1, P->gw1, (size_t)F1 * NF);
    take(P->b1, P->gb1, F1);
    take(P->w2, P->gw2, (size_t)NCLS * F1);
    take(P->b2, P->gb2, NCLS);
    Arena& a = m->arena;
    a.take<char>(sizeof(Plan));
    P->col = a.take<float>(R * KC);
    P->z = a.take<float>(R * CO);
    P->xhat = a.take<float>(R * CO);
    P->y = a.take<float>(R * CO);
    P->rstd = a.take<float>(CO);
    P->p = a.take<float>(B * NF);
    P->arg = a.take<uint8_t>(B * NF);
    P->f1 = a.take<float>(B * F1);
    P->dz = a.take<float>(B * NCLS);
    P->df1 = a.take<float>(B * F1);
    P->dp = a.take<float>(B * NF);
    P->dbn = a.take<float>(R * CO);
    P->dconv = a.take<float>(R * CO);
    P->part_floats = (size_t)kMaxSlices * CO * KC;
    P->part = a.take<float>(P->part_floats);
    P->colws = a.take<float>(colsum_ws_floats((int)B, F1));
    if (!P->colws) {
        set_error("vgg5: workspace arena too small");
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
    const int B = acts->batch, R = B * HW * HW;
    fo_status st = FO_OK;
    auto gemm = [&](const GemmF32& g) { return launch_gemm_f32(g, P->part, P->part_floats, s); };
#define TRY(x)                      \
    do {                            \
        st = (x);                   \
        if (st != FO_OK) return st; \
    } while (0)
    // forward (Alg. 4: forward pass of M_s)
    hipLaunchKernelGGL(im2col_kernel, dim3(nblk((int64_t)R * KC)), dim3(256), 0, s, m->dev_in, P->col, B);
    FO_LAUNCHED();
    TRY(gemm(prod(P->col, KC, 1, P->wc, KC, 1, P->z, CO, R, CO, KC)));
    hipLaunchKernelGGL(bn5_fwd, dim3(CO), dim3(256), 0, s, P->z, P->g, P->bb, P->xhat, P->y, P->rstd, R);
    hipLaunchKernelGGL(pool5_fwd, dim3(nblk((int64_t)B * NF)), dim3(256), 0, s, P->y, P->p, P->arg, B);
    FO_LAUNCHED();
    GemmF32 g1 = prod(P->p, NF, 1, P->w1, NF, 1, P->f1, F1, B, F1, NF);
    g1.bias = P->b1;
    g1.relu = 1;
    TRY(gemm(g1));
    GemmF32 g2 = prod(P->f1, F1, 1, P->w2, F1, 1, m->logits, NCLS, B, NCLS, F1);
    g2.bias = P->b2;
    TRY(gemm(g2));
    TRY(launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, NCLS, s));
    // backward (Alg. 4: backward pass of M_s)
    TRY(gemm(prod(P->dz, 1, NCLS, P->f1, 1, F1, P->gw2, F1, NCLS, F1, B)));       // dW2 = dz^T f1
    TRY(launch_colsum(P->dz, NCLS, B, nullptr, NCLS, P->gb2, P->colws, s));
    GemmF32 gd = prod(P->dz, NCLS, 1, P->w2, 1, F1, P->df1, F1, B, F1, NCLS);     // df1 = dz W2 * (f1 > 0)
    gd.mask = P->f1;
    gd.ldmask = F1;
    TRY(gemm(gd));
    GemmF32 gw = prod(P->df1, 1, F1, P->p, 1, NF, P->gw1, NF, F1, NF, B);         // dW1 = df1^T p
    TRY(gemm(gw));
    TRY(launch_colsum(P->df1, F1, B, nullptr, F1, P->gb1, P->colws, s));
    TRY(gemm(prod(P->df1, F1, 1, P->w1, 1, NF, P->dp, NF, B, NF, F1)));          // dp = df1 W1
    hipLaunchKernelGGL(pool5_relu_bwd, dim3(nblk((int64_t)R * CO)), dim3(256), 0, s, P->dp, P->arg, P->y, P->dbn, B);
    hipLaunchKernelGGL(bn5_bwd, dim3(CO), dim3(256), 0, s, P->dbn, P->xhat, P->g, P->rstd, P->dconv, P->gg, P->gbb,
                       R);
    FO_LAUNCHED();
    GemmF32 gc = prod(P->dconv, 1, CO, P->col, 1, KC, P->gwc, KC, CO, KC, R);   // dWc = dconv^T col
    gc.S = std::min(kMaxSlices, std::max(1, R / 256));
    TRY(gemm(gc));
#undef TRY
    // SGD (Alg. 4)
    return launch_sgd(m->params, m->grads, nullptr, nullptr, nullptr, m->n_params, m->lr, 0.f, s);
}

void destroy(fo_model* m) {
    delete (Plan*)m->plan;
    m->plan = nullptr;
}

}  // namespace

int64_t vgg5_param_count() { return kParams; }

const Family* family_vgg5() {
    static const Family f = {(int64_t)CI * HW * HW * 4, ws_bytes, init, step, destroy};
    return &f;
}

}  // namespace fo
