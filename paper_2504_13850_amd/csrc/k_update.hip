// Bandwidth kernels of the hot path: the staleness-weighted aggregation
// (Alg. 4, aggregation branch) and the fused SGD update (Alg. 4, last step of
// the activation branch).  Both are single streaming passes with 16-byte
// vector accesses; the grid is sized to a few waves per CU and strides over
// the vector, so every CU of every XCD streams a contiguous share.
#include "kernels.h"

namespace fo {

// ------------------------------------------------------------------ aggregation
// g <- g + w (l - g), one FMA per element after the difference, so w = 0 and
// l == g leave g bit for bit.
__global__ void __launch_bounds__(256) agg_lerp_kernel(float* __restrict__ g, const float* __restrict__ l,
                                                       int64_t n4, int64_t n, float w) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    f32x4* g4 = reinterpret_cast<f32x4*>(g);
    const f32x4* l4 = reinterpret_cast<const f32x4*>(l);
    for (; i < n4; i += stride) {
        f32x4 a = g4[i];
        f32x4 b = __builtin_nontemporal_load(&l4[i]);
        a.x = __builtin_fmaf(w, b.x - a.x, a.x);
        a.y = __builtin_fmaf(w, b.y - a.y, a.y);
        a.z = __builtin_fmaf(w, b.z - a.z, a.z);
        a.w = __builtin_fmaf(w, b.w - a.w, a.w);
        g4[i] = a;
    }
    // tail (n not a multiple of 4): handled by the first threads
    int64_t t = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n) g[t] = __builtin_fmaf(w, l[t] - g[t], g[t]);
}

// Several arrivals applied in order to each element while it sits in a register.
__global__ void __launch_bounds__(256) agg_lerp_multi_kernel(float* __restrict__ g, AggTable tab, int64_t n4,
                                                             int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    f32x4* g4 = reinterpret_cast<f32x4*>(g);
    for (; i < n4; i += stride) {
        f32x4 a = g4[i];
        for (int m = 0; m < tab.count; ++m) {
            const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(tab.local[m]) + i);
            const float w = tab.w[m];
            a.x = __builtin_fmaf(w, b.x - a.x, a.x);
            a.y = __builtin_fmaf(w, b.y - a.y, a.y);
            a.z = __builtin_fmaf(w, b.z - a.z, a.z);
            a.w = __builtin_fmaf(w, b.w - a.w, a.w);
        }
        g4[i] = a;
    }
    int64_t t = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n) {
        float a = g[t];
        for (int m = 0; m < tab.count; ++m) a = __builtin_fmaf(tab.w[m], tab.local[m][t] - a, a);
        g[t] = a;
    }
}

static int stream_grid(int64_t n4) {
    // 256 CUs x 8 blocks of 256 threads saturate HBM; small vectors use fewer.
    int64_t blocks = cdiv(n4 > 0 ? n4 : 1, 256);
    if (blocks > 2048) blocks = 2048;
    return (int)blocks;
}

fo_status launch_agg_lerp(float* g, const float* l, int64_t n, float w, hipStream_t s) {
    if (n == 0) return FO_OK;
    int64_t n4 = n / 4;
    int grid = stream_grid(n4);
    int tail = (int)(n - n4 * 4);
    if (grid * 256 < tail) grid = 1;
    hipLaunchKernelGGL(agg_lerp_kernel, dim3(grid), dim3(256), 0, s, g, l, n4, n, w);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_agg_lerp_multi(float* g, const AggTable& tab, int64_t n, hipStream_t s) {
    if (n == 0 || tab.count == 0) return FO_OK;
    int64_t n4 = n / 4;
    int grid = stream_grid(n4);
    hipLaunchKernelGGL(agg_lerp_multi_kernel, dim3(grid), dim3(256), 0, s, g, tab, n4, n);
    FO_LAUNCHED();
    return FO_OK;
}

// ------------------------------------------------------------------ SGD
// theta <- theta - lr * g; optional momentum v <- mu v + g, theta <- theta - lr v;
// optional bf16 shadow of theta for the MFMA GEMM operands.
template <bool MOM, bool SHADOW>
__global__ void __launch_bounds__(256) sgd_kernel(float* __restrict__ p, const float* __restrict__ g,
                                                  float* __restrict__ v, bf16_t* __restrict__ w16,
                                                  bf16_t* __restrict__ w16lo, int64_t n4, int64_t n, float lr,
                                                  float mu) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n4; i += stride) {
        float4 a = reinterpret_cast<float4*>(p)[i];
        float4 d = reinterpret_cast<const float4*>(g)[i];
        if (MOM) {
            float4 m = reinterpret_cast<float4*>(v)[i];
            m.x = __builtin_fmaf(mu, m.x, d.x);
            m.y = __builtin_fmaf(mu, m.y, d.y);
            m.z = __builtin_fmaf(mu, m.z, d.z);
            m.w = __builtin_fmaf(mu, m.w, d.w);
            reinterpret_cast<float4*>(v)[i] = m;
            d = m;
        }
        a.x = __builtin_fmaf(-lr, d.x, a.x);
        a.y = __builtin_fmaf(-lr, d.y, a.y);
        a.z = __builtin_fmaf(-lr, d.z, a.z);
        a.w = __builtin_fmaf(-lr, d.w, a.w);
        reinterpret_cast<float4*>(p)[i] = a;
        if (SHADOW) {
            const bf16_t hx = f2bf(a.x), hy = f2bf(a.y), hz = f2bf(a.z), hw = f2bf(a.w);
            uint2 h;
            h.x = (uint32_t)hx | ((uint32_t)hy << 16);
            h.y = (uint32_t)hz | ((uint32_t)hw << 16);
            reinterpret_cast<uint2*>(w16)[i] = h;
            uint2 lo;
            lo.x = (uint32_t)f2bf(a.x - bf2f(hx)) | ((uint32_t)f2bf(a.y - bf2f(hy)) << 16);
            lo.y = (uint32_t)f2bf(a.z - bf2f(hz)) | ((uint32_t)f2bf(a.w - bf2f(hw)) << 16);
            reinterpret_cast<uint2*>(w16lo)[i] = lo;
        }
    }
    int64_t t = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n) {
        float d = g[t];
        if (MOM) {
            d = __builtin_fmaf(mu, v[t], d);
            v[t] = d;
        }
        float a = __builtin_fmaf(-lr, d, p[t]);
        p[t] = a;
        if (SHADOW) {
            const bf16_t h = f2bf(a);
            w16[t] = h;
            w16lo[t] = f2bf(a - bf2f(h));
        }
    }
}

fo_status launch_sgd(float* p, const float* g, float* v, bf16_t* w16, bf16_t* w16lo, int64_t n, float lr, float mu,
                     hipStream_t s) {
    if (n == 0) return FO_OK;
    FO_CHECK(!w16 == !w16lo, "sgd: the bf16 shadow needs both parts");
    int64_t n4 = n / 4;
    int grid = stream_grid(n4);
    if (v && w16)
        hipLaunchKernelGGL((sgd_kernel<true, true>), dim3(grid), dim3(256), 0, s, p, g, v, w16, w16lo, n4, n, lr, mu);
    else if (v)
        hipLaunchKernelGGL((sgd_kernel<true, false>), dim3(grid), dim3(256), 0, s, p, g, v, w16, w16lo, n4, n, lr, mu);
    else if (w16)
        hipLaunchKernelGGL((sgd_kernel<false, true>), dim3(grid), dim3(256), 0, s, p, g, v, w16, w16lo, n4, n, lr, mu);
    else
        hipLaunchKernelGGL((sgd_kernel<false, false>), dim3(grid), dim3(256), 0, s, p, g, v, w16, w16lo, n4, n, lr,
                           mu);
    FO_LAUNCHED();
    return FO_OK;
}

// fp32 -> (bf16 high part, bf16 low part) of the master weights.
__global__ void cast_bf16_kernel(const float* __restrict__ x, bf16_t* __restrict__ y, bf16_t* __restrict__ ylo,
                                 int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) {
        const bf16_t h = f2bf(x[i]);
        y[i] = h;
        if (ylo) ylo[i] = f2bf(x[i] - bf2f(h));
    }
}

fo_status launch_cast_bf16(const float* x, bf16_t* y, bf16_t* ylo, int64_t n, hipStream_t s) {
    if (n == 0) return FO_OK;
    hipLaunchKernelGGL(cast_bf16_kernel, dim3(stream_grid(n)), dim3(256), 0, s, x, y, ylo, n);
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
