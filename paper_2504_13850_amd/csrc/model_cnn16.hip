// Configs 2, 5 (VGG-16 split) and 3 (ResNet-18 split): one training
// iteration of the activation branch of Alg. 4 on bf16 MFMA implicit-GEMM
// convolutions, NHWC activations, fp32 master weights.
//
//   VGG:    10 conv3x3 + bias + ReLU with 4 max pools (16x16 -> 1x1), FC 512-512-10
//   ResNet: stages 2-4 of ResNet-18 (BasicBlocks, training-mode BatchNorm, 1x1
//           stride-2 projection shortcuts), global average pool, FC 512-100,
//           SGD with momentum 0.9
//
// Forward GEMMs are compensated split-bf16 products (high and low parts of the
// activations and weights); backward GEMMs use the high parts.  The input
// gradient of the first server layer is never formed.
#include <vector>

#include "gemm.h"
#include "model.h"

namespace fo {

fo_status launch_nchw_to_nhwc(const StepIn* in, bf16_t* y, int B, int C, int HW, hipStream_t s);
fo_status launch_maxpool_fwd(const bf16_t* xh, const bf16_t* xl, bf16_t* yh, bf16_t* yl, uint8_t* arg, int B, int H,
                             int W, int C, hipStream_t s);
fo_status launch_maxpool_relu_bwd(const float* dy, const uint8_t* arg, const bf16_t* y, float* dxf, bf16_t* dxb, int B,
                                  int H, int W, int C, hipStream_t s);
fo_status launch_gap_fwd(const bf16_t* xh, const bf16_t* xl, float* h, int B, int HW, int C, hipStream_t s);
fo_status launch_gap_relu_bwd(const float* dh, const bf16_t* y, float* dxf, int B, int HW, int C, hipStream_t s);
size_t bn_ws_floats(int rows, int C);
// batch norm (training mode) over rows x C (C % 64 == 0); see k_cnn.hip
// S <= kBnMaxSplits split-K slices
constexpr int kBnMaxSplits = 8;
fo_status launch_bn_fwd_stats(const float* ws, int S, float* z, int rows, int C, float* part, hipStream_t s);
fo_status launch_bn_fwd_apply(const float* z, const float* part, int rows, int C, float eps, const float* g,
                              const float* beta, const float* resf, const bf16_t* resh, const bf16_t* resl, bool relu,
                              float* mean, float* rstd, float* yf, bf16_t* yh, bf16_t* yl, hipStream_t s);
fo_status launch_bn_bwd(const float* gout, const bf16_t* mask, float* dy_out, const float* z, const float* mean,
                        const float* rstd, const float* g, int rows, int C, float* dg, float* db, float* dzf,
                        bf16_t* dzb, float* part, hipStream_t s);
fo_status launch_to_bf16(const float* x, bf16_t* y, int64_t n, hipStream_t s);

namespace {

#define TRY(x)                           \
    do {                                 \
        fo_status st_ = (x);             \
        if (st_ != FO_OK) return st_;    \
    } while (0)

constexpr int kIn = 64, kHW = 16;  // server input: [B][64][16][16]

struct Conv {
    int cin, cout, k, stride, pad, H, W, Ho, Wo;
    int64_t w, b;               // parameter offsets (b < 0: no bias)
    int64_t g, be;              // batch-norm scale / shift offsets (< 0: none)
    int splits;                 // K slices of the weight gradient
    int fsplits, dsplits;       // K slices of the forward and of the input gradient
    // activations
    bf16_t *yh, *yl;            // VGG: post-ReLU output (hi, lo)
    float *z, *mean, *rstd;     // ResNet: pre-norm output and its batch statistics
    float* part;                // ResNet: the norm's per-row-block partial sums
    float *dzf, *dzpart;        // VGG: fp32 gradient of the pre-activation, and the
                                // partial rows of its column sums (the bias gradient)
    float* wgws;                // the weight gradient's own split-K partials (splits > 1)
};

struct Pool {
    int H, W, C;
    bf16_t *yh, *yl;
    uint8_t* arg;
};

struct Block {
    int c1, c2, cd;  // indices into convs (cd < 0: identity shortcut)
    bf16_t *a1h, *a1l, *outh, *outl;
    float* scf;      // projected shortcut after its norm
};

struct Fc {
    int in, out;
    int64_t w, b;
    bf16_t *yh, *yl;  // post-ReLU output (hidden layers)
};

struct Plan {
    bool resnet;
    int B;
    std::vector<Conv> convs;
    std::vector<int> order;   // VGG: op sequence, >= 0 conv index, < 0 pool index -(i+1)
    std::vector<Pool> pools;
    std::vector<Block> blocks;
    std::vector<Fc> fcs;
    bf16_t* xin;              // NHWC input
    float* gap;               // ResNet pooled features fp32 [B][512]
    bf16_t *gaph, *gapl;
    float* dz;                // dlogits [B][classes]
    bf16_t* dzb;
    float *df[3];             // gradient ping-pong (fp32)
    bf16_t *db[2];            // gradient (bf16 GEMM operand)
    float *dsc, *dtmp;        // ResNet shortcut / scratch gradients
    float *splitws, *redws;
    size_t act_max;           // elements of the largest activation
};

// K slices of a conv product: as many as fit one round of two workgroups per
// CU over its output tiles (at most maxs), each at least min_k long.  The deep
// layers have few output tiles (2x2 maps: M = 4 B) and long K (9 Cin up to
// 4608), so without slices most CUs would sit idle.  Measured at batch 64:
// up to 32 slices of at least 256 (VGG) or 128 (ResNet) beat the earlier 8 of
// at least 256 by 7% (VGG) and 3.5% (ResNet) per step; 1024 slots, or 4 or 2
// slices at most, were slower.
constexpr int kMaxSplits = 32;
int split_for(int M, int N, int K, int min_k, int maxs = kMaxSplits) {
    int tiles = (int)(cdiv(M, 128) * cdiv(N, 128));
    int s = std::max(1, std::min(maxs, 512 / std::max(tiles, 1)));
    while (s > 1 && (int64_t)K / s < min_k) --s;
    return s;
}

// Builds the layer list and parameter offsets (the library layout).
void build(Plan& P, int cid, int B) {
    P.resnet = cid == 3;
    P.B = B;
    int64_t o = 0;
    auto conv = [&](int cin, int cout, int k, int stride, int pad, int H, bool bias, bool bn) {
        Conv c{};
        c.cin = cin; c.cout = cout; c.k = k; c.stride = stride; c.pad = pad;
        c.H = H; c.W = H;
        c.Ho = (H + 2 * pad - k) / stride + 1;
        c.Wo = c.Ho;
        c.w = o; o += (int64_t)cout * k * k * cin;
        c.b = -1; c.g = -1; c.be = -1;
        if (bias) { c.b = o; o += cout; }
        if (bn) { c.g = o; o += cout; c.be = o; o += cout; }
        // (the ResNet forward's partials go to its norm's statistics kernel,
        // which sums at most kBnMaxSplits slices)
        const int min_k = P.resnet ? 128 : 256;
        c.splits = split_for(cout, k * k * cin, B * c.Ho * c.Wo, min_k);
        c.fsplits = split_for(B * c.Ho * c.Wo, cout, 3 * (int)cdiv(k * k * cin, 64) * 64, min_k,
                              P.resnet ? kBnMaxSplits : kMaxSplits);
        c.dsplits = split_for(B * H * H, cin, k * k * cout, min_k);
        P.convs.push_back(c);
        return (int)P.convs.size() - 1;
    };
    if (!P.resnet) {
        const int plan[] = {128, 128, 0, 256, 256, 256, 0, 512, 512, 512, 0, 512, 512, 512, 0};
        int cin = kIn, H = kHW;
        for (int v : plan) {
            if (v == 0) {
                Pool p{};
                p.H = H; p.W = H; p.C = cin;
                P.pools.push_back(p);
                P.order.push_back(-(int)P.pools.size());
                H /= 2;
            } else {
                P.order.push_back(conv(cin, v, 3, 1, 1, H, true, false));
                cin = v;
            }
        }
        const int dims[4] = {512, 512, 512, 10};
        for (int i = 0; i < 3; ++i) {
            Fc f{};
            f.in = dims[i]; f.out = dims[i + 1];
            f.w = o; o += (int64_t)f.out * f.in;
            f.b = o; o += f.out;
            P.fcs.push_back(f);
        }
    } else {
        int cin = kIn, H = kHW;
        const int chans[3] = {128, 256, 512};
        for (int st = 0; st < 3; ++st) {
            const int c = chans[st];
            for (int bi = 0; bi < 2; ++bi) {
                Block b{};
                const int stride = bi == 0 ? 2 : 1;
                b.c1 = conv(bi == 0 ? cin : c, c, 3, stride, 1, H, false, true);
                const int Ho = P.convs[b.c1].Ho;
                b.c2 = conv(c, c, 3, 1, 1, Ho, false, true);
                b.cd = bi == 0 ? conv(cin, c, 1, 2, 0, H, false, true) : -1;
                P.blocks.push_back(b);
                H = Ho;
            }
            cin = c;
        }
        Fc f{};
        f.in = 512; f.out = 100;
        f.w = o; o += (int64_t)f.out * f.in;
        f.b = o; o += f.out;
        P.fcs.push_back(f);
    }
}

int64_t count_params(int cid) {
    Plan P;
    build(P, cid, 1);
    int64_t n = 0;
    for (const Conv& c : P.convs) {
        n += (int64_t)c.cout * c.k * c.k * c.cin;
        if (c.b >= 0) n += c.cout;
        if (c.g >= 0) n += 2 * c.cout;
    }
    for (const Fc& f : P.fcs) n += (int64_t)f.out * f.in + f.out;
    return n;
}

size_t ws_bytes(const fo_model* m) {
    Plan P;
    const int B = m->max_batch;
    build(P, m->cid, B);
    size_t s = 0;
    auto add = [&](size_t b) { s += (b + 255) & ~size_t(255); };
    add(sizeof(Plan) + 4096);
    size_t amax = (size_t)B * kHW * kHW * kIn, sw = 0, red = 0;
    add(2 * amax);  // xin
    for (const Conv& c : P.convs) {
        const size_t n = (size_t)B * c.Ho * c.Wo * c.cout;
        amax = std::max(amax, n);
        if (P.resnet) { add(4 * n); add(4 * c.cout); add(4 * c.cout); add(4 * bn_ws_floats(B * c.Ho * c.Wo, c.cout)); }
        else { add(2 * n); add(2 * n); add(4 * n); add(4 * colsum_ws_floats(B * c.Ho * c.Wo, c.cout)); }
        if (P.resnet) add(gemm_ws_bytes(c.cout, c.k * c.k * c.cin, c.splits));  // wgws
        sw = std::max(sw, gemm_ws_bytes(c.cout, c.k * c.k * c.cin, c.splits));
        sw = std::max(sw, gemm_ws_bytes(B * c.Ho * c.Wo, c.cout, c.fsplits));
        sw = std::max(sw, gemm_ws_bytes(B * c.H * c.W, c.cin, c.dsplits));
        red = std::max(red, bn_ws_floats(B * c.Ho * c.Wo, c.cout));
        red = std::max(red, colsum_ws_floats(B * c.Ho * c.Wo, c.cout));
    }
    for (const Pool& p : P.pools) {
        const size_t n = (size_t)B * (p.H / 2) * (p.W / 2) * p.C;
        add(2 * n); add(2 * n); add(n);
    }
    for (const Block& b : P.blocks) {
        const Conv& c = P.convs[b.c2];
        const size_t n = (size_t)B * c.Ho * c.Wo * c.cout;
        add(2 * n); add(2 * n); add(2 * n); add(2 * n);
        if (b.cd >= 0) add(4 * n);
    }
    for (const Fc& f : P.fcs) {
        add(2 * (size_t)B * f.out); add(2 * (size_t)B * f.out);
        red = std::max(red, colsum_ws_floats(B, f.out));
        red = std::max(red, 3 * colsum_ws_floats(B, 512));  // VGG: the classifier's three bias sums together
    }
    add(4 * (size_t)B * 512); add(2 * (size_t)B * 512); add(2 * (size_t)B * 512);
    add(4 * (size_t)B * 128); add(2 * (size_t)B * 128);
    for (int i = 0; i < 3; ++i) add(4 * amax);
    for (int i = 0; i < 2; ++i) add(2 * amax);
    add(4 * amax); add(4 * amax);
    add(sw + 256);
    add(4 * red + 256);
    return s;
}

fo_status init(fo_model* m) {
    Plan* P = new (std::nothrow) Plan();
    if (!P) return FO_ENOMEM;
    m->plan = P;
    const int B = m->max_batch;
    build(*P, m->cid, B);
    Arena& a = m->arena;
    a.take<char>(sizeof(Plan) + 4096);
    size_t amax = (size_t)B * kHW * kHW * kIn, sw = 0, red = 0;
    P->xin = a.take<bf16_t>(amax);
    for (Conv& c : P->convs) {
        const size_t n = (size_t)B * c.Ho * c.Wo * c.cout;
        amax = std::max(amax, n);
        if (P->resnet) {
            c.z = a.take<float>(n);
            c.mean = a.take<float>(c.cout);
            c.rstd = a.take<float>(c.cout);
            c.part = a.take<float>(bn_ws_floats(B * c.Ho * c.Wo, c.cout));
            c.dzf = c.dzpart = nullptr;
        } else {
            c.yh = a.take<bf16_t>(n);
            c.yl = a.take<bf16_t>(n);
            c.dzf = a.take<float>(n);
            c.dzpart = a.take<float>(colsum_ws_floats(B * c.Ho * c.Wo, c.cout));
        }
        c.wgws = P->resnet && c.splits > 1 ? a.take<float>(gemm_ws_bytes(c.cout, c.k * c.k * c.cin, c.splits) / 4)
                                           : nullptr;
        sw = std::max(sw, gemm_ws_bytes(c.cout, c.k * c.k * c.cin, c.splits));
        sw = std::max(sw, gemm_ws_bytes(B * c.Ho * c.Wo, c.cout, c.fsplits));
        sw = std::max(sw, gemm_ws_bytes(B * c.H * c.W, c.cin, c.dsplits));
        red = std::max(red, bn_ws_floats(B * c.Ho * c.Wo, c.cout));
        red = std::max(red, colsum_ws_floats(B * c.Ho * c.Wo, c.cout));
    }
    for (Pool& p : P->pools) {
        const size_t n = (size_t)B * (p.H / 2) * (p.W / 2) * p.C;
        p.yh = a.take<bf16_t>(n);
        p.yl = a.take<bf16_t>(n);
        p.arg = a.take<uint8_t>(n);
    }
    for (Block& b : P->blocks) {
        const Conv& c = P->convs[b.c2];
        const size_t n = (size_t)B * c.Ho * c.Wo * c.cout;
        b.a1h = a.take<bf16_t>(n);
        b.a1l = a.take<bf16_t>(n);
        b.outh = a.take<bf16_t>(n);
        b.outl = a.take<bf16_t>(n);
        b.scf = b.cd >= 0 ? a.take<float>(n) : nullptr;
    }
    for (Fc& f : P->fcs) {
        f.yh = a.take<bf16_t>((size_t)B * f.out);
        f.yl = a.take<bf16_t>((size_t)B * f.out);
        red = std::max(red, colsum_ws_floats(B, f.out));
        red = std::max(red, 3 * colsum_ws_floats(B, 512));  // VGG: the classifier's three bias sums together
    }
    P->gap = a.take<float>((size_t)B * 512);
    P->gaph = a.take<bf16_t>((size_t)B * 512);
    P->gapl = a.take<bf16_t>((size_t)B * 512);
    P->dz = a.take<float>((size_t)B * 128);
    P->dzb = a.take<bf16_t>((size_t)B * 128);
    for (int i = 0; i < 3; ++i) P->df[i] = a.take<float>(amax);
    for (int i = 0; i < 2; ++i) P->db[i] = a.take<bf16_t>(amax);
    P->dsc = a.take<float>(amax);
    P->dtmp = a.take<float>(amax);
    P->splitws = a.take<float>(sw / 4 + 64);
    P->redws = a.take<float>(red + 64);
    P->act_max = amax;
    if (!P->redws) {
        set_error("cnn16: workspace arena too small");
        return FO_ENOMEM;
    }
    return FO_OK;
}

// ------------------------------------------------------------------ GEMM wrappers
ConvGeom geom(const Conv& c, int B) {
    ConvGeom g;
    g.Bn = B; g.H = c.H; g.W = c.W; g.Ci = c.cin;
    g.Ho = c.Ho; g.Wo = c.Wo; g.Co = c.cout;
    g.kh = c.k; g.kw = c.k; g.stride = c.stride; g.pad = c.pad;
    return g;
}

// forward of a convolution as a compensated implicit GEMM
GemmDesc conv_fwd_desc(const fo_model* m, const Conv& c, int B, const bf16_t* xh, const bf16_t* xl) {
    GemmDesc d;
    d.M = B * c.Ho * c.Wo; d.N = c.cout; d.K = c.k * c.k * c.cin;
    d.amode = OP_CONV_FWD; d.A = xh; d.A2 = xl;
    d.bmode = OP_RK; d.B = m->w16 + c.w; d.B2 = m->w16lo + c.w; d.ldb = d.K;
    d.nseg = xl ? 3 : 2;
    d.g = geom(c, B);
    d.splits = c.fsplits; d.ws = static_cast<const Plan*>(m->plan)->splitws;
    return d;
}

// Weight gradient.  Nothing reads it before the update, so with `sums` its
// split slices stay in the conv's own workspace and join the set that the step
// adds up in one launch at the end of the backward (ResNet: 1.029 -> 0.981 ms
// per step); without, the slices are summed right away (VGG, whose larger
// partial sets are cheaper to sum while they are still in cache: 1.070 ms
// against 1.080 deferred).
fo_status conv_wgrad(fo_model* m, const Plan* P, const Conv& c, int B, const bf16_t* dzb, const bf16_t* xh,
                     SplitJobs* sums) {
    GemmDesc d;
    d.M = c.cout; d.N = c.k * c.k * c.cin; d.K = B * c.Ho * c.Wo;
    d.amode = OP_KR; d.A = dzb; d.lda = c.cout;
    d.bmode = OP_CONV_DWX; d.B = xh;
    d.g = geom(c, B);
    d.Cf = m->grads + c.w; d.ldcf = d.N;
    d.splits = c.splits;
    d.ws = sums ? c.wgws : P->splitws;
    if (sums && c.splits > 1) {
        FO_CHECK(sums->n < kSplitJobsMax, "cnn16: more than %d deferred weight-gradient sums", kSplitJobsMax);
        d.defer_reduce = true;
        SplitJob& j = sums->j[sums->n++];
        j.ws = c.wgws; j.C = d.Cf; j.ldc = d.ldcf; j.S = c.splits; j.M = d.M; j.N = d.N;
    }
    return gemm(d, m->stream);
}

// input gradient: dx = conv^T(dz); optional ReLU mask (the input's own values),
// optional residual gradient added; fp32 and/or bf16 outputs
fo_status conv_dgrad(fo_model* m, const Conv& c, int B, const bf16_t* dzb, const bf16_t* mask, const float* resid,
                     float* outf, bf16_t* outb) {
    GemmDesc d;
    d.M = B * c.H * c.W; d.N = c.cin; d.K = c.k * c.k * c.cout;
    d.amode = OP_CONV_DX; d.A = dzb;
    d.bmode = OP_CONV_DXW; d.B = m->w16 + c.w;
    d.g = geom(c, B);
    d.mask = mask; d.ldm = c.cin;
    d.resid = resid; d.ldr = c.cin;
    d.Cf = outf; d.ldcf = c.cin;
    d.Cb = outb; d.ldcb = c.cin;
    d.splits = c.dsplits; d.ws = static_cast<const Plan*>(m->plan)->splitws;
    return gemm(d, m->stream);
}

// fully connected layer forward (compensated), hidden layers with ReLU
fo_status fc_fwd(fo_model* m, const Fc& f, int B, const bf16_t* xh, const bf16_t* xl, bool relu, float* outf,
                 bf16_t* outh, bf16_t* outl) {
    GemmDesc d;
    d.M = B; d.N = f.out; d.K = f.in;
    d.amode = OP_RK; d.A = xh; d.A2 = xl; d.lda = f.in;
    d.bmode = OP_RK; d.B = m->w16 + f.w; d.B2 = m->w16lo + f.w; d.ldb = f.in;
    d.nseg = xl ? 3 : 2;
    d.bias = m->params + f.b;
    d.act = relu ? ACT_RELU : ACT_NONE;
    d.Cf = outf; d.ldcf = f.out;
    d.Cb = outh; d.Cb2 = outl; d.ldcb = f.out;
    return gemm(d, m->stream);
}

// fully connected backward: weight and bias gradients, then the input gradient
// (the bias gradient's column sums join `sums` when given, else run here)
fo_status fc_bwd(fo_model* m, Plan* P, const Fc& f, int B, const float* dyf, const bf16_t* dyb, const bf16_t* xh,
                 const bf16_t* mask, float* dxf, bf16_t* dxb, ColSums* sums = nullptr, float* sum_part = nullptr) {
    GemmDesc w;
    w.M = f.out; w.N = f.in; w.K = B;
    w.amode = OP_KR; w.A = dyb; w.lda = f.out;
    w.bmode = OP_KR; w.B = xh; w.ldb = f.in;
    w.Cf = m->grads + f.w; w.ldcf = f.in;
    TRY(gemm(w, m->stream));
    if (sums)
        sums->add(dyf, f.out, B, f.out, sum_part, m->grads + f.b);
    else
        TRY(launch_colsum(dyf, f.out, B, nullptr, f.out, m->grads + f.b, P->redws, m->stream));
    if (dxf || dxb) {
        GemmDesc d;
        d.M = B; d.N = f.in; d.K = f.out;
        d.amode = OP_RK; d.A = dyb; d.lda = f.out;
        d.bmode = OP_KR; d.B = m->w16 + f.w; d.ldb = f.in;
        d.mask = mask; d.ldm = f.in;
        d.Cf = dxf; d.ldcf = f.in;
        d.Cb = dxb; d.ldcb = f.in;
        TRY(gemm(d, m->stream));
    }
    return FO_OK;
}

// ------------------------------------------------------------------ VGG
fo_status step_vgg(fo_model* m, Plan* P, int B, const int32_t* labels) {
    hipStream_t s = m->stream;
    const bf16_t *xh = P->xin, *xl = nullptr;
    // forward
    for (int op : P->order) {
        if (op >= 0) {
            Conv& c = P->convs[op];
            GemmDesc d = conv_fwd_desc(m, c, B, xh, xl);
            d.bias = m->params + c.b;
            d.act = ACT_RELU;
            d.Cb = c.yh; d.Cb2 = c.yl; d.ldcb = c.cout;
            TRY(gemm(d, s));
            xh = c.yh; xl = c.yl;
        } else {
            Pool& p = P->pools[-op - 1];
            TRY(launch_maxpool_fwd(xh, xl, p.yh, p.yl, p.arg, B, p.H, p.W, p.C, s));
            xh = p.yh; xl = p.yl;
        }
    }
    Fc &f0 = P->fcs[0], &f1 = P->fcs[1], &f2 = P->fcs[2];
    TRY(fc_fwd(m, f0, B, xh, xl, true, nullptr, f0.yh, f0.yl));
    TRY(fc_fwd(m, f1, B, f0.yh, f0.yl, true, nullptr, f1.yh, f1.yl));
    TRY(fc_fwd(m, f2, B, f1.yh, f1.yl, false, m->logits, nullptr, nullptr));
    TRY(launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, f2.out, s));
    // backward through the classifier (its bias sums join the convs' pass at
    // the end; dz, df[0] and df[1] stay intact until then)
    ColSums bias_sums;
    const size_t fcpart = colsum_ws_floats(B, 512);
    TRY(launch_to_bf16(P->dz, P->dzb, (int64_t)B * f2.out, s));
    TRY(fc_bwd(m, P, f2, B, P->dz, P->dzb, f1.yh, f1.yh, P->df[0], P->db[0], &bias_sums, P->redws));
    TRY(fc_bwd(m, P, f1, B, P->df[0], P->db[0], f0.yh, f0.yh, P->df[1], P->db[1], &bias_sums, P->redws + fcpart));
    const Pool& last = P->pools.back();
    TRY(fc_bwd(m, P, f0, B, P->df[1], P->db[1], last.yh, nullptr, P->df[2], nullptr, &bias_sums,
               P->redws + 2 * fcpart));
    // Backward through the convolutions.  db[0] and db[1] alternate as the bf16
    // gradient of a conv's pre-activation (the GEMMs' operand); its fp32 copy
    // goes to the conv's own dzf, whose column sums (the bias gradients) run
    // for all convs in one pass at the end.  df[2] holds the gradient of a
    // pool's output.
    const bf16_t* gb = nullptr;
    int pf = 0;
    for (int idx = (int)P->order.size() - 1; idx >= 0; --idx) {
        const int op = P->order[idx];
        if (op < 0) {
            // pool: route to the window winner, mask with the producing conv's ReLU
            const Pool& p = P->pools[-op - 1];
            const Conv& prod = P->convs[P->order[idx - 1]];
            TRY(launch_maxpool_relu_bwd(P->df[2], p.arg, prod.yh, prod.dzf, P->db[pf], B, p.H, p.W, p.C, s));
            gb = P->db[pf];
            pf ^= 1;
            continue;
        }
        const Conv& c = P->convs[op];
        bias_sums.add(c.dzf, c.cout, B * c.Ho * c.Wo, c.cout, c.dzpart, m->grads + c.b);
        const int prev = idx > 0 ? P->order[idx - 1] : 0;
        const bf16_t* in = idx == 0 ? P->xin : (prev >= 0 ? P->convs[prev].yh : P->pools[-prev - 1].yh);
        TRY(conv_wgrad(m, P, c, B, gb, in, nullptr));
        if (idx == 0) break;  // the first server layer: no input gradient
        if (prev >= 0) {
            // the input is a conv's ReLU output: mask in the epilogue
            const Conv& pc = P->convs[prev];
            TRY(conv_dgrad(m, c, B, gb, pc.yh, nullptr, pc.dzf, P->db[pf]));
            gb = P->db[pf];
            pf ^= 1;
        } else {
            TRY(conv_dgrad(m, c, B, gb, nullptr, nullptr, P->df[2], nullptr));
            gb = nullptr;
        }
    }
    TRY(launch_colsums(bias_sums, s));
    return launch_sgd(m->params, m->grads, nullptr, m->w16, m->w16lo, m->n_params, m->lr, 0.f, s);
}

// ------------------------------------------------------------------ ResNet
fo_status step_resnet(fo_model* m, Plan* P, int B, const int32_t* labels) {
    hipStream_t s = m->stream;
    const float eps = 1e-5f;
    const bf16_t *xh = P->xin, *xl = nullptr;
    for (Block& b : P->blocks) {
        Conv &c1 = P->convs[b.c1], &c2 = P->convs[b.c2];
        const int rows = B * c2.Ho * c2.Wo;
        // Each convolution leaves its split-K partials to the statistics kernel of
        // its norm, which sums them into z.
        auto conv_bn_stats = [&](Conv& c, const bf16_t* inh, const bf16_t* inl) -> fo_status {
            GemmDesc d = conv_fwd_desc(m, c, B, inh, inl);
            d.Cf = c.z; d.ldcf = c.cout;
            d.defer_reduce = true;
            TRY(gemm(d, s));
            return launch_bn_fwd_stats(P->splitws, d.splits, c.z, rows, c.cout, c.part, s);
        };
        auto bn_apply = [&](Conv& c, const float* resf, const bf16_t* resh, const bf16_t* resl, bool relu, float* yf,
                            bf16_t* yh, bf16_t* yl) {
            return launch_bn_fwd_apply(c.z, c.part, rows, c.cout, eps, m->params + c.g, m->params + c.be, resf, resh,
                                       resl, relu, c.mean, c.rstd, yf, yh, yl, s);
        };
        TRY(conv_bn_stats(c1, xh, xl));
        TRY(bn_apply(c1, nullptr, nullptr, nullptr, true, nullptr, b.a1h, b.a1l));
        TRY(conv_bn_stats(c2, b.a1h, b.a1l));
        if (b.cd >= 0) {
            Conv& cd = P->convs[b.cd];
            TRY(conv_bn_stats(cd, xh, xl));
            TRY(bn_apply(cd, nullptr, nullptr, nullptr, false, b.scf, nullptr, nullptr));
            TRY(bn_apply(c2, b.scf, nullptr, nullptr, true, nullptr, b.outh, b.outl));
        } else {
            TRY(bn_apply(c2, nullptr, xh, xl, true, nullptr, b.outh, b.outl));
        }
        xh = b.outh; xl = b.outl;
    }
    const Block& lastb = P->blocks.back();
    const Conv& lastc = P->convs[lastb.c2];
    const int hw = lastc.Ho * lastc.Wo;
    TRY(launch_gap_fwd(xh, xl, P->gap, B, hw, 512, s));
    TRY(launch_cast_bf16(P->gap, P->gaph, P->gapl, (int64_t)B * 512, s));
    Fc& fc = P->fcs[0];
    TRY(fc_fwd(m, fc, B, P->gaph, P->gapl, false, m->logits, nullptr, nullptr));
    TRY(launch_xent(m->logits, m->dev_in, P->dz, m->loss, B, fc.out, s));
    TRY(launch_to_bf16(P->dz, P->dzb, (int64_t)B * fc.out, s));
    TRY(fc_bwd(m, P, fc, B, P->dz, P->dzb, P->gaph, nullptr, P->df[1], nullptr));
    // gradient of the last block's output (through the average pool and its ReLU)
    float* gout = P->df[0];
    TRY(launch_gap_relu_bwd(P->df[1], lastb.outh, gout, B, hw, 512, s));
    SplitJobs wsums;
    for (int bi = (int)P->blocks.size() - 1; bi >= 0; --bi) {
        Block& b = P->blocks[bi];
        Conv &c1 = P->convs[b.c1], &c2 = P->convs[b.c2];
        const int rows = B * c2.Ho * c2.Wo;
        float* g = P->df[1];  // gradient of the pre-ReLU sum (stored by the first norm backward)
        // main branch: second conv + norm (its input gradient is gout through the block's ReLU)
        TRY(launch_bn_bwd(gout, b.outh, g, c2.z, c2.mean, c2.rstd, m->params + c2.g, rows, c2.cout, m->grads + c2.g,
                          m->grads + c2.be, nullptr, P->db[0], c2.part, s));
        TRY(conv_wgrad(m, P, c2, B, P->db[0], b.a1h, &wsums));
        TRY(conv_dgrad(m, c2, B, P->db[0], b.a1h, nullptr, P->dtmp, nullptr));
        TRY(launch_bn_bwd(P->dtmp, nullptr, nullptr, c1.z, c1.mean, c1.rstd, m->params + c1.g, rows, c1.cout,
                          m->grads + c1.g, m->grads + c1.be, nullptr, P->db[1], c1.part, s));
        const bf16_t* xin_h = bi == 0 ? P->xin : P->blocks[bi - 1].outh;
        TRY(conv_wgrad(m, P, c1, B, P->db[1], xin_h, &wsums));
        const bool need_dx = bi > 0;
        float* gnext = P->df[2];
        // shortcut branch
        const float* sc_grad = g;
        if (b.cd >= 0) {
            Conv& cd = P->convs[b.cd];
            TRY(launch_bn_bwd(g, nullptr, nullptr, cd.z, cd.mean, cd.rstd, m->params + cd.g, rows, cd.cout,
                              m->grads + cd.g, m->grads + cd.be, nullptr, P->db[0], cd.part, s));
            TRY(conv_wgrad(m, P, cd, B, P->db[0], xin_h, &wsums));
            if (need_dx) TRY(conv_dgrad(m, cd, B, P->db[0], nullptr, nullptr, P->dsc, nullptr));
            sc_grad = P->dsc;
        }
        if (need_dx) {
            TRY(conv_dgrad(m, c1, B, P->db[1], nullptr, sc_grad, gnext, nullptr));
            // the block input is the previous block's output: next iteration masks it
            std::swap(P->df[0], P->df[2]);
            gout = P->df[0];
        }
    }
    if (wsums.n) TRY(launch_splitk_sum_multi(wsums, s));
    return launch_sgd(m->params, m->grads, m->mom, m->w16, m->w16lo, m->n_params, m->lr, m->momentum, s);
}

fo_status step(fo_model* m, const fo_acts* acts, const int32_t* labels) {
    Plan* P = (Plan*)m->plan;
    const int B = acts->batch;
    TRY(launch_nchw_to_nhwc(m->dev_in, P->xin, B, kIn, kHW * kHW, m->stream));
    return P->resnet ? step_resnet(m, P, B, labels) : step_vgg(m, P, B, labels);
}

void destroy(fo_model* m) {
    delete (Plan*)m->plan;
    m->plan = nullptr;
}

}  // namespace

int64_t cnn16_param_count(int32_t cid) { return count_params(cid); }

const Family* family_cnn16() {
    static const Family f = {(int64_t)kIn * kHW * kHW * 2, ws_bytes, init, step, destroy};
    return &f;
}

}  // namespace fo
