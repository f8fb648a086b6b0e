// fp32 products for the small fp32 models (the paper's Transformer-6/12 and
// VGG-5 server parts): C[m][n] = epilogue(sum_k A(m, k) B(n, k)) over strided
// operands, as LDS-tiled FMA with the next K chunk's loads in flight, and an
// optional deterministic split over K (slices summed in order afterwards).
#include "kernels.h"

namespace fo {
namespace {

constexpr int GT = 64, GK = 32;
// automatic K split (GemmF32::auto_split): products with fewer than kAutoTiles
// output tiles take min(16, kAutoSlots / tiles, K / kAutoMinK) slices
constexpr int64_t kAutoTiles = 128, kAutoSlots = 512, kAutoMinK = 64;
// workgroups of 64-row tiles below which a product runs on 32-row tiles, of
// 32-row tiles below which it runs on 16-row tiles, and of 16 x 64 tiles below
// which it runs on 16 x 32 (for the 32-row step, thresholds of 256, 512, 1024
// or always gave the same step times)
constexpr int64_t kRows32Below = 512;

__device__ __forceinline__ float epi(const GemmF32& g, const float* add, int m, int n, float v) {
    if (g.bias) v += g.bias[n];
    if (add) v += add[(int64_t)m * g.ldadd + n];
    if (g.relu) v = fmaxf(v, 0.f);
    if (g.mask && !(g.mask[(int64_t)m * g.ldmask + n] > 0.f)) v = 0.f;
    return v;
}

// One operand's share of an RT x 32 chunk (RT = 64, 32 or 16 rows): value v of
// thread t is element e = t + 256 v; with K contiguous (KF) the 32 k of a row
// are consecutive threads, else the RT rows are.
template <bool KF, int RT>
__device__ __forceinline__ void chunk_rc(int e, int& r, int& k) {
    r = KF ? e >> 5 : e % RT;
    k = KF ? e & 31 : e / RT;
}
// Every load reads a valid element (row and k clamped into the operand, R and
// ke >= 1) and the values outside the chunk are zeroed when stored: with
// "in range ? load : 0" the compiler selects right after each load, so each
// load waits for the previous one and the chunk in flight is not in flight.
template <bool KF, int RT, int NV>
__device__ __forceinline__ void load_chunk(const float* P, int64_t sr, int64_t sk, int r0, int R, int k0, int ke,
                                           float (&v)[NV]) {
    static_assert(NV * 256 == RT * GK, "chunk share");
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        int r, k;
        chunk_rc<KF, RT>(threadIdx.x + 256 * i, r, k);
        const int gr = min(r0 + r, R - 1), gk = min(k0 + k, ke - 1);
        v[i] = P[(int64_t)gr * sr + (KF ? (int64_t)gk : (int64_t)gk * sk)];
    }
}
template <bool KF, int RT, int NV>
__device__ __forceinline__ void store_chunk(float (*T)[RT + 4], const float (&v)[NV], int r0, int R, int k0,
                                            int ke) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        int r, k;
        chunk_rc<KF, RT>(threadIdx.x + 256 * i, r, k);
        T[k][r] = r0 + r < R && k0 + k < ke ? v[i] : 0.f;
    }
}

// TM x 16 = 64, 32 or 16 rows by 64 columns of output per workgroup, TM x 4
// per thread; K in chunks of 32, the next chunk's loads in flight (registers)
// while this one is computed from LDS, two LDS buffers (one barrier per
// chunk).  The 32-row form doubles the workgroups of a product with few
// tiles, whose time is otherwise the latency of each workgroup's K walk.
template <bool AKF, bool BKF, int TM, int TN>
__global__ void __launch_bounds__(256) gemm_f32(const GemmF32 g) {
    constexpr int BMt = 16 * TM, BNt = 16 * TN, NA = BMt * GK / 256, NB = BNt * GK / 256;
    __shared__ float As[2][GK][BMt + 4], Bs[2][GK][BNt + 4];
    const float* A = g.inA ? (const float*)g.inA->x : g.A;
    const float* Bp = g.inB ? (const float*)g.inB->x : g.B;
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int n0 = blockIdx.x * BNt, m0 = blockIdx.y * BMt, z = blockIdx.z;
    const int kc = ((g.K + g.S - 1) / g.S + GK - 1) / GK * GK;
    const int kb = z * kc, ke = min(g.K, kb + kc);
    const int nch = ke > kb ? (ke - kb + GK - 1) / GK : 0;
    float acc[TM][TN] = {};
    float ra[NA], rb[NB];
    if (nch > 0) {
        load_chunk<AKF, BMt>(A, g.am, g.ak, m0, g.M, kb, ke, ra);
        load_chunk<BKF, BNt>(Bp, g.bn, g.bk, n0, g.N, kb, ke, rb);
        store_chunk<AKF, BMt>(As[0], ra, m0, g.M, kb, ke);
        store_chunk<BKF, BNt>(Bs[0], rb, n0, g.N, kb, ke);
    }
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
        const int u = c & 1;
        if (c + 1 < nch) {  // next chunk in flight during this chunk's FMAs
            load_chunk<AKF, BMt>(A, g.am, g.ak, m0, g.M, kb + (c + 1) * GK, ke, ra);
            load_chunk<BKF, BNt>(Bp, g.bn, g.bk, n0, g.N, kb + (c + 1) * GK, ke, rb);
        }
#pragma unroll
        for (int k = 0; k < GK; ++k) {
            float a[TM];
            if constexpr (TM == 4) {
                const float4 a4 = *reinterpret_cast<const float4*>(&As[u][k][ty * 4]);
                a[0] = a4.x; a[1] = a4.y; a[2] = a4.z; a[3] = a4.w;
            } else if constexpr (TM == 2) {
                const float2 a2 = *reinterpret_cast<const float2*>(&As[u][k][ty * TM]);
                a[0] = a2.x; a[1] = a2.y;
            } else {
                a[0] = As[u][k][ty];
            }
            float b[TN];
            if constexpr (TN == 4) {
                const float4 b4 = *reinterpret_cast<const float4*>(&Bs[u][k][tx * 4]);
                b[0] = b4.x; b[1] = b4.y; b[2] = b4.z; b[3] = b4.w;
            } else {
                const float2 b2 = *reinterpret_cast<const float2*>(&Bs[u][k][tx * 2]);
                b[0] = b2.x; b[1] = b2.y;
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        if (c + 1 < nch) {
            store_chunk<AKF, BMt>(As[u ^ 1], ra, m0, g.M, kb + (c + 1) * GK, ke);
            store_chunk<BKF, BNt>(Bs[u ^ 1], rb, n0, g.N, kb + (c + 1) * GK, ke);
        }
        __syncthreads();
    }
    if (g.S > 1) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int m = m0 + ty * TM + i;
            if (m >= g.M) continue;
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int n = n0 + tx * TN + j;
                if (n < g.N) g.part[((int64_t)z * g.M + m) * g.N + n] = acc[i][j];
            }
        }
        return;
    }
    // the epilogue's operands of all 16 elements first (indices clamped into
    // the product, so every load is valid), then the guarded stores
    const float* add = g.inAdd ? (const float*)g.inAdd->x : g.add;
    int mi[TM], nj[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) mi[i] = min(m0 + ty * TM + i, g.M - 1);
#pragma unroll
    for (int j = 0; j < TN; ++j) nj[j] = min(n0 + tx * TN + j, g.N - 1);
    float bv[TN] = {}, av[TM][TN] = {}, mv[TM][TN];
    if (g.bias) {
#pragma unroll
        for (int j = 0; j < TN; ++j) bv[j] = g.bias[nj[j]];
    }
    if (add) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) av[i][j] = add[(int64_t)mi[i] * g.ldadd + nj[j]];
    }
    if (g.mask) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) mv[i][j] = g.mask[(int64_t)mi[i] * g.ldmask + nj[j]];
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int m = m0 + ty * TM + i;
        if (m >= g.M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + tx * TN + j;
            if (n >= g.N) continue;
            float v = acc[i][j] + bv[j] + av[i][j];
            if (g.relu) v = fmaxf(v, 0.f);
            if (g.mask && !(mv[i][j] > 0.f)) v = 0.f;
            g.C[(int64_t)m * g.ldc + n] = v;
        }
    }
}

__global__ void __launch_bounds__(256) gemm_f32_reduce(const GemmF32 g) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)g.M * g.N) return;
    const int m = (int)(i / g.N), n = (int)(i % g.N);
    float v = 0.f;
    for (int z = 0; z < g.S; ++z) v += g.part[(int64_t)z * g.M * g.N + i];
    const float* add = g.inAdd ? (const float*)g.inAdd->x : g.add;
    g.C[(int64_t)m * g.ldc + n] = epi(g, add, m, n, v);
}


}  // namespace

fo_status launch_gemm_f32(GemmF32 g, float* part, size_t part_floats, hipStream_t s) {
    FO_CHECK(g.M >= 1 && g.N >= 1 && g.K >= 1, "fp32 product: M=%d N=%d K=%d", g.M, g.N, g.K);
    FO_CHECK(!g.defer || (!g.bias && !g.add && !g.inAdd && !g.mask && !g.relu &&
                          (g.S <= 1 || (part && (size_t)g.S * g.M * g.N <= part_floats))),
             "fp32 product: deferred slices need a plain epilogue and room for all of them");
    if (g.auto_split && g.S == 1 && !g.defer) {
        // few 64 x 64 tiles over a long K leave most CUs idle while each
        // workgroup walks K chunk by chunk: split K so that about kAutoSlots
        // workgroups run, each slice at least kAutoMinK long
        const int64_t tiles = cdiv(g.N, GT) * cdiv(g.M, GT);
        if (tiles < kAutoTiles)
            g.S = (int)std::max<int64_t>(1, std::min<int64_t>({16, kAutoSlots / tiles, g.K / kAutoMinK}));
    }
    if (g.S > 1) {
        const size_t per = (size_t)g.M * g.N;
        if (!part || (size_t)g.S * per > part_floats) g.S = part ? (int)(part_floats / per) : 1;
    }
    if (g.S < 1) g.S = 1;
    g.part = part;
    // 32-row tiles when 64-row ones would not give every CU two workgroups,
    // 16-row tiles when 32-row ones would not either, then 32-column tiles
    const bool rows32 = cdiv(g.N, GT) * cdiv(g.M, GT) * g.S < kRows32Below;
    const bool rows16 = rows32 && cdiv(g.N, GT) * cdiv(g.M, 32) * g.S < kRows32Below;
    const bool cols32 = rows16 && cdiv(g.N, GT) * cdiv(g.M, 16) * g.S < kRows32Below;
    const dim3 grid((int)cdiv(g.N, cols32 ? 32 : GT), (int)cdiv(g.M, rows16 ? 16 : rows32 ? 32 : GT), g.S);
    const bool akf = g.ak == 1, bkf = g.bk == 1;
#define FO_GEMM_F32(AK, BK)                                                       \
    do {                                                                         \
        if (cols32)                                                                 \
            hipLaunchKernelGGL((gemm_f32<AK, BK, 1, 2>), grid, dim3(256), 0, s, g); \
        else if (rows16)                                                            \
            hipLaunchKernelGGL((gemm_f32<AK, BK, 1, 4>), grid, dim3(256), 0, s, g); \
        else if (rows32)                                                            \
            hipLaunchKernelGGL((gemm_f32<AK, BK, 2, 4>), grid, dim3(256), 0, s, g); \
        else                                                                        \
            hipLaunchKernelGGL((gemm_f32<AK, BK, 4, 4>), grid, dim3(256), 0, s, g); \
    } while (0)
    if (akf && bkf)
        FO_GEMM_F32(true, true);
    else if (akf)
        FO_GEMM_F32(true, false);
    else if (bkf)
        FO_GEMM_F32(false, true);
    else
        FO_GEMM_F32(false, false);
#undef FO_GEMM_F32
    FO_LAUNCHED();
    if (g.S > 1 && !g.defer) {
        hipLaunchKernelGGL(gemm_f32_reduce, dim3((int)cdiv((int64_t)g.M * g.N, 256)), dim3(256), 0, s, g);
        FO_LAUNCHED();
    }
    return FO_OK;
}

}  // namespace fo
