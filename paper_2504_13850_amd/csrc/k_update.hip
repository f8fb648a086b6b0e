// Bandwidth kernels of the hot path: the staleness-weighted aggregation
// (Alg. 4, aggregation branch) and the fused SGD update (Alg. 4, last step of
// the activation branch).  Both are single streaming passes with 16-byte
// vector accesses; the grid is sized to a few waves per CU and strides over
// the vector, so every CU of every XCD streams a contiguous share.
#include "kernels.h"

namespace fo {

// Streaming shape shared by the kernels below: a block pass covers SCHUNK
// 16-byte vectors (SU per thread, 256 apart, so each load instruction of a
// wave reads 1 KiB contiguous); every load of a pass is issued before the
// first use, and full passes carry no per-lane bounds test.
constexpr int SU = 4;
constexpr int64_t SCHUNK = 256 * SU;

__device__ __forceinline__ f32x4 lerp4(f32x4 a, f32x4 b, float w) {
    a.x = __builtin_fmaf(w, b.x - a.x, a.x);
    a.y = __builtin_fmaf(w, b.y - a.y, a.y);
    a.z = __builtin_fmaf(w, b.z - a.z, a.z);
    a.w = __builtin_fmaf(w, b.w - a.w, a.w);
    return a;
}

// ------------------------------------------------------------------ aggregation
// g <- g + w (l - g), one FMA per element after the difference, so w = 0 and
// l == g leave g bit for bit.
__global__ void __launch_bounds__(256) agg_lerp_kernel(float* __restrict__ g, const float* __restrict__ l,
                                                       int64_t n4, int64_t n, float w) {
    f32x4* g4 = reinterpret_cast<f32x4*>(g);
    const f32x4* l4 = reinterpret_cast<const f32x4*>(l);
    const int tid = threadIdx.x;
    const int64_t step = (int64_t)gridDim.x * SCHUNK;
    int64_t base = (int64_t)blockIdx.x * SCHUNK;
    for (; base + SCHUNK <= n4; base += step) {
        f32x4 a[SU], b[SU];
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            a[u] = __builtin_nontemporal_load(&g4[base + 256 * u + tid]);
            b[u] = __builtin_nontemporal_load(&l4[base + 256 * u + tid]);
        }
#pragma unroll
        for (int u = 0; u < SU; ++u) __builtin_nontemporal_store(lerp4(a[u], b[u], w), &g4[base + 256 * u + tid]);
    }
    if (base < n4) {  // the partial last pass
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            const int64_t i = base + 256 * u + tid;
            if (i < n4) g4[i] = lerp4(g4[i], l4[i], w);
        }
    }
    // tail (n not a multiple of 4): handled by the first threads
    int64_t t = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n) g[t] = __builtin_fmaf(w, l[t] - g[t], g[t]);
}

// Several arrivals applied in order to each element while it sits in a
// register.  The vectors of the next AP arrivals are in flight while the
// current one is applied: each element's arrivals form a chain of dependent
// updates, so with a small model (a few hundred blocks at most) the chain's
// load latency, not HBM bandwidth, sets the time.
constexpr int MU = 1;
constexpr int AP = 32;

__global__ void __launch_bounds__(256) agg_lerp_multi_kernel(float* __restrict__ g, AggTable tab, int64_t n4,
                                                             int64_t n) {
    f32x4* g4 = reinterpret_cast<f32x4*>(g);
    const int tid = threadIdx.x;
    const int64_t chunk = 256 * MU;
    const int cnt = tab.count;
    for (int64_t base = (int64_t)blockIdx.x * chunk; base < n4; base += (int64_t)gridDim.x * chunk) {
        int64_t idx[MU];
        bool ok[MU];
        f32x4 a[MU], ring[AP][MU];
#pragma unroll
        for (int u = 0; u < MU; ++u) {
            idx[u] = base + 256 * u + tid;
            ok[u] = idx[u] < n4;
            if (!ok[u]) idx[u] = 0;  // in range; the result is not stored
            a[u] = g4[idx[u]];
        }
#pragma unroll
        for (int p = 0; p < AP; ++p)
            if (p < cnt)
#pragma unroll
                for (int u = 0; u < MU; ++u)
                    ring[p][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(tab.local[p]) + idx[u]);
        for (int m0 = 0; m0 < cnt; m0 += AP) {
#pragma unroll
            for (int p = 0; p < AP; ++p) {
                const int m = m0 + p;
                if (m < cnt) {
                    const float w = tab.w[m];
#pragma unroll
                    for (int u = 0; u < MU; ++u) a[u] = lerp4(a[u], ring[p][u], w);
                    if (m + AP < cnt)
#pragma unroll
                        for (int u = 0; u < MU; ++u)
                            ring[p][u] = __builtin_nontemporal_load(
                                reinterpret_cast<const f32x4*>(tab.local[m + AP]) + idx[u]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < MU; ++u)
            if (ok[u]) g4[idx[u]] = a[u];
    }
    int64_t t = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n) {
        float a = g[t];
        for (int m = 0; m < tab.count; ++m) a = __builtin_fmaf(tab.w[m], tab.local[m][t] - a, a);
        g[t] = a;
    }
}

static int stream_grid(int64_t n4, int64_t chunk, int64_t cap = 2048) {
    // 256 CUs x 8 blocks of 256 threads keep HBM busy; small vectors use fewer.
    int64_t blocks = cdiv(n4 > 0 ? n4 : 1, chunk);
    if (blocks > cap) blocks = cap;
    return (int)blocks;
}
static int stream_grid(int64_t n4) { return stream_grid(n4, SCHUNK); }
// The aggregation's 2:1 read-write stream: 16384 blocks (each pass of a block
// 16 KiB of either vector) measured 6.1 TB/s on 1 GiB vectors against 5.8 TB/s
// with 2048 blocks (read-only streams reach 7.1 TB/s, write-only 4.9).
constexpr int64_t kAggGridCap = 16384;

// ------------------------------------------------------------------ pool arrival
// Copies n16 16-byte chunks in the streaming shape above: full passes with
// every load of the pass issued before the first store and no per-lane test
// (with a test on each unrolled load the compiler waits after every load:
// 19.5 us against 7 us for a 6 MiB batch), then one guarded partial pass.
__device__ __forceinline__ void stream_copy16(const uint4* __restrict__ xs, uint4* __restrict__ xd, int64_t n16) {
    const int tid = threadIdx.x;
    const int64_t step = (int64_t)gridDim.x * SCHUNK;
    int64_t base = (int64_t)blockIdx.x * SCHUNK;
    for (; base + SCHUNK <= n16; base += step) {
        uint4 v[SU];
#pragma unroll
        for (int u = 0; u < SU; ++u) v[u] = xs[base + 256 * u + tid];
#pragma unroll
        for (int u = 0; u < SU; ++u) xd[base + 256 * u + tid] = v[u];
    }
    if (base < n16) {
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            const int64_t i = base + 256 * u + tid;
            if (i < n16) xd[i] = xs[i];
        }
    }
}

// One admitted activation batch into its pool slot: the activations (n16
// 16-byte chunks) and the int32 labels and lengths (batch each, lengths
// optional) in one launch.  The first block also copies labels and lengths.
__global__ void __launch_bounds__(256) pool_put_kernel(const uint4* __restrict__ xs, uint4* __restrict__ xd,
                                                       int64_t n16, const int32_t* __restrict__ ls,
                                                       int32_t* __restrict__ ld, const int32_t* __restrict__ ns,
                                                       int32_t* __restrict__ nd, int batch) {
    stream_copy16(xs, xd, n16);
    if (blockIdx.x == 0)
        for (int b = threadIdx.x; b < batch; b += 256) {
            ld[b] = ls[b];
            if (nd) nd[b] = ns[b];
        }
}

fo_status launch_pool_put(const void* x_src, void* x_dst, int64_t bytes, const int32_t* lab_src, int32_t* lab_dst,
                          const int32_t* len_src, int32_t* len_dst, int batch, hipStream_t s) {
    FO_CHECK(bytes % 16 == 0 && ((uintptr_t)x_src & 15) == 0 && ((uintptr_t)x_dst & 15) == 0,
             "pool put: the activations must be whole, 16-byte aligned chunks");
    const int64_t n16 = bytes / 16;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(cdiv(n16, 256 * SU), 1024));
    hipLaunchKernelGGL(pool_put_kernel, dim3(grid), dim3(256), 0, s, (const uint4*)x_src, (uint4*)x_dst, n16, lab_src,
                       lab_dst, len_src, len_dst, batch);
    FO_LAUNCHED();
    return FO_OK;
}

// Up to kPutMaxBatches admitted batches in one launch: blockIdx.y = the batch,
// blocks along x stride over its activations; block (0, y) copies its labels
// and lengths.
__global__ void __launch_bounds__(256) pool_put_gather_kernel(const PutTable t, int64_t n16, int batch) {
    const int e = blockIdx.y;
    const uint4* __restrict__ xs = t.xs[e];
    uint4* __restrict__ xd = t.xd[e];
    stream_copy16(xs, xd, n16);
    if (blockIdx.x == 0)
        for (int b = threadIdx.x; b < batch; b += 256) {
            t.ld[e][b] = t.ls[e][b];
            if (t.nd[e]) t.nd[e][b] = t.ns[e][b];
        }
}

fo_status launch_pool_put_gather(const PutTable& t, int64_t bytes, int batch, hipStream_t s) {
    FO_CHECK(t.count >= 1 && t.count <= kPutMaxBatches, "pool put: %d batches in one launch", t.count);
    FO_CHECK(bytes % 16 == 0, "pool put: slot bytes not a multiple of 16");
    for (int i = 0; i < t.count; ++i)
        FO_CHECK(((uintptr_t)t.xs[i] & 15) == 0 && ((uintptr_t)t.xd[i] & 15) == 0,
                 "pool put: activations of batch %d not 16-byte aligned", i);
    const int64_t n16 = bytes / 16;
    const int gx = (int)std::max<int64_t>(1, std::min<int64_t>(cdiv(n16, 256 * SU), 128));
    hipLaunchKernelGGL(pool_put_gather_kernel, dim3(gx, t.count), dim3(256), 0, s, t, n16, batch);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_agg_lerp(float* g, const float* l, int64_t n, float w, hipStream_t s) {
    if (n == 0) return FO_OK;
    int64_t n4 = n / 4;
    int grid = stream_grid(n4, SCHUNK, kAggGridCap);
    int tail = (int)(n - n4 * 4);
    if (grid * 256 < tail) grid = 1;
    hipLaunchKernelGGL(agg_lerp_kernel, dim3(grid), dim3(256), 0, s, g, l, n4, n, w);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_agg_lerp_multi(float* g, const AggTable& tab, int64_t n, hipStream_t s) {
    if (n == 0 || tab.count == 0) return FO_OK;
    int64_t n4 = n / 4;
    int grid = stream_grid(n4, 256 * MU, kAggGridCap);
    hipLaunchKernelGGL(agg_lerp_multi_kernel, dim3(grid), dim3(256), 0, s, g, tab, n4, n);
    FO_LAUNCHED();
    return FO_OK;
}

// ------------------------------------------------------------------ SGD
// theta <- theta - lr * g; optional momentum v <- mu v + g, theta <- theta - lr v;
// optional bf16 shadow of theta for the MFMA GEMM operands.
template <bool MOM, bool SHADOW>
__device__ __forceinline__ void sgd_store(float* p, float* v, bf16_t* w16, bf16_t* w16lo, int64_t i, f32x4 a,
                                          f32x4 d, f32x4 m, float lr, float mu) {
    if (MOM) {
        m.x = __builtin_fmaf(mu, m.x, d.x);
        m.y = __builtin_fmaf(mu, m.y, d.y);
        m.z = __builtin_fmaf(mu, m.z, d.z);
        m.w = __builtin_fmaf(mu, m.w, d.w);
        __builtin_nontemporal_store(m, reinterpret_cast<f32x4*>(v) + i);
        d = m;
    }
    a.x = __builtin_fmaf(-lr, d.x, a.x);
    a.y = __builtin_fmaf(-lr, d.y, a.y);
    a.z = __builtin_fmaf(-lr, d.z, a.z);
    a.w = __builtin_fmaf(-lr, d.w, a.w);
    __builtin_nontemporal_store(a, reinterpret_cast<f32x4*>(p) + i);
    if (SHADOW) {
        const bf16_t hx = f2bf(a.x), hy = f2bf(a.y), hz = f2bf(a.z), hw = f2bf(a.w);
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        u32x2 h, lo;
        h.x = (uint32_t)hx | ((uint32_t)hy << 16);
        h.y = (uint32_t)hz | ((uint32_t)hw << 16);
        lo.x = (uint32_t)f2bf(a.x - bf2f(hx)) | ((uint32_t)f2bf(a.y - bf2f(hy)) << 16);
        lo.y = (uint32_t)f2bf(a.z - bf2f(hz)) | ((uint32_t)f2bf(a.w - bf2f(hw)) << 16);
        __builtin_nontemporal_store(h, reinterpret_cast<u32x2*>(w16) + i);
        __builtin_nontemporal_store(lo, reinterpret_cast<u32x2*>(w16lo) + i);
    }
}

// ------------------------------------------------------------------ SGD
// theta <- theta - lr * g; optional momentum v <- mu v + g, theta <- theta - lr v;
// optional bf16 shadow (high and low parts) of theta for the MFMA GEMM operands.
template <bool MOM, bool SHADOW>
__global__ void __launch_bounds__(256) sgd_kernel(float* __restrict__ p, const float* __restrict__ g,
                                                  float* __restrict__ v, bf16_t* __restrict__ w16,
                                                  bf16_t* __restrict__ w16lo, int64_t n4, int64_t n, float lr,
                                                  float mu) {
    const f32x4* p4 = reinterpret_cast<const f32x4*>(p);
    const f32x4* g4 = reinterpret_cast<const f32x4*>(g);
    const f32x4* v4 = reinterpret_cast<const f32x4*>(v);
    const int tid = threadIdx.x;
    const int64_t step = (int64_t)gridDim.x * SCHUNK;
    int64_t base = (int64_t)blockIdx.x * SCHUNK;
    for (; base + SCHUNK <= n4; base += step) {
        f32x4 a[SU], d[SU], m[SU];
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            const int64_t i = base + 256 * u + tid;
            a[u] = __builtin_nontemporal_load(p4 + i);
            d[u] = __builtin_nontemporal_load(g4 + i);
            if (MOM) m[u] = __builtin_nontemporal_load(v4 + i);
        }
#pragma unroll
        for (int u = 0; u < SU; ++u)
            sgd_store<MOM, SHADOW>(p, v, w16, w16lo, base + 256 * u + tid, a[u], d[u], m[u], lr, mu);
    }
    if (base < n4) {  // the partial last pass
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            const int64_t i = base + 256 * u + tid;
            if (i < n4) sgd_store<MOM, SHADOW>(p, v, w16, w16lo, i, p4[i], g4[i], MOM ? v4[i] : f32x4{}, lr, mu);
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

// The same plain update (no momentum) restricted to a list of parameter ranges:
// block b updates elements [chunks[2b], chunks[2b] + chunks[2b + 1]) with the
// arithmetic of sgd_kernel; used for the parameters whose update is not fused
// into their weight-gradient product.
__global__ void __launch_bounds__(256) sgd_chunks_kernel(float* __restrict__ p, const float* __restrict__ g,
                                                         bf16_t* __restrict__ w16, bf16_t* __restrict__ w16lo,
                                                         const int64_t* __restrict__ chunks, float lr) {
    const int64_t off = chunks[2 * blockIdx.x], len = chunks[2 * blockIdx.x + 1];
    for (int64_t i = threadIdx.x; i < len; i += blockDim.x) {
        const int64_t t = off + i;
        const float a = __builtin_fmaf(-lr, g[t], p[t]);
        p[t] = a;
        if (w16) {
            const bf16_t h = f2bf(a);
            w16[t] = h;
            w16lo[t] = f2bf(a - bf2f(h));
        }
    }
}

fo_status launch_sgd_chunks(float* p, const float* g, bf16_t* w16, bf16_t* w16lo, const int64_t* chunks,
                            int nchunks, float lr, hipStream_t s) {
    if (nchunks == 0) return FO_OK;
    FO_CHECK(!w16 == !w16lo, "sgd: the bf16 shadow needs both parts");
    hipLaunchKernelGGL(sgd_chunks_kernel, dim3(nchunks), dim3(256), 0, s, p, g, w16, w16lo, chunks, lr);
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
