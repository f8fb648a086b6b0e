// Small kernels shared by the model executors: the loss f_s (mean softmax
// cross-entropy and its gradient), column sums (bias and norm-parameter
// gradients), fills, and small fp32 linear layers for the classifier heads.
#include "kernels.h"

namespace fo {
namespace {

// Mean softmax cross-entropy over the batch and dz = (softmax - onehot) / B.
// Labels outside [0, C) are clamped into range.
__global__ void __launch_bounds__(256) xent_kernel(const float* __restrict__ z, const int32_t* __restrict__ labels,
                                                   float* __restrict__ dz, float* __restrict__ loss, int B, int C) {
    __shared__ float part[256];
    float mine = 0.f;
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        const float* zr = z + (int64_t)b * C;
        float m = zr[0];
        for (int c = 1; c < C; ++c) m = fmaxf(m, zr[c]);
        float s = 0.f;
        for (int c = 0; c < C; ++c) s += expf(zr[c] - m);
        float lse = m + logf(s);
        int y = labels[b];
        y = y < 0 ? 0 : (y >= C ? C - 1 : y);
        mine += lse - zr[y];
        for (int c = 0; c < C; ++c) dz[(int64_t)b * C + c] = (expf(zr[c] - lse) - (c == y ? 1.f : 0.f)) / (float)B;
    }
    part[threadIdx.x] = mine;
    __syncthreads();
    for (int s = blockDim.x / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) loss[0] = part[0] / (float)B;
}

// Column sums of a [rows][N] matrix in two passes: blocks of (256 columns x
// 64 rows) write partial sums, then one thread per column adds them.
constexpr int CS_ROWS = 64;

template <typename T>
__device__ __forceinline__ float ld_as_f(const T* p);
template <> __device__ __forceinline__ float ld_as_f<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_as_f<bf16_t>(const bf16_t* p) { return bf2f(*p); }

template <typename T>
__global__ void __launch_bounds__(256) colsum_partial(const T* __restrict__ X, int64_t ld, int rows,
                                                      const int* __restrict__ rows_dev, int N,
                                                      float* __restrict__ part) {
    const int R = rows_dev ? min(rows, *rows_dev) : rows;
    const int col = blockIdx.x * 256 + threadIdx.x;
    const int r0 = blockIdx.y * CS_ROWS;
    if (col >= N) return;
    float s = 0.f;
    const int r1 = min(R, r0 + CS_ROWS);
    for (int r = r0; r < r1; ++r) s += ld_as_f<T>(X + (int64_t)r * ld + col);
    part[(int64_t)blockIdx.y * N + col] = s;
}

__global__ void __launch_bounds__(256) colsum_finish(const float* __restrict__ part, int chunks, int N,
                                                     float* __restrict__ out) {
    const int col = blockIdx.x * 256 + threadIdx.x;
    if (col >= N) return;
    float s = 0.f;
    for (int c = 0; c < chunks; ++c) s += part[(int64_t)c * N + col];
    out[col] = s;
}

__global__ void __launch_bounds__(256) fill_kernel(float* __restrict__ p, int64_t n, float v) {
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

// y[b][o] = act(bias[o] + sum_i x[b][i] w[o][i]); one wave per output o, lanes
// stride over i (coalesced rows of w), every b handled by the same wave.
template <int ACT>
__global__ void __launch_bounds__(256) small_linear_fwd_kernel(const float* __restrict__ x, const float* __restrict__ w,
                                                               const float* __restrict__ bias, float* __restrict__ y,
                                                               int B, int I, int O) {
    const int lane = threadIdx.x & 63;
    const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (o >= O) return;
    const float* wr = w + (int64_t)o * I;
    for (int b = 0; b < B; ++b) {
        const float* xr = x + (int64_t)b * I;
        float s = 0.f;
        for (int i = lane; i < I; i += 64) s = fmaf(xr[i], wr[i], s);
        for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
        if (lane == 0) {
            float v = s + bias[o];
            y[(int64_t)b * O + o] = ACT == 1 ? tanhf(v) : v;
        }
    }
}

// gw[o][i] = sum_b dy[b][o] x[b][i]; gb[o] = sum_b dy[b][o]
__global__ void __launch_bounds__(256) small_linear_wgrad_kernel(const float* __restrict__ dy,
                                                                 const float* __restrict__ x, float* __restrict__ gw,
                                                                 float* __restrict__ gb, int B, int I, int O) {
    int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx < (int64_t)O * I) {
        int o = (int)(idx / I), i = (int)(idx % I);
        float s = 0.f;
        for (int b = 0; b < B; ++b) s = fmaf(dy[(int64_t)b * O + o], x[(int64_t)b * I + i], s);
        gw[idx] = s;
    }
    if (idx < O) {
        float s = 0.f;
        for (int b = 0; b < B; ++b) s += dy[(int64_t)b * O + idx];
        gb[idx] = s;
    }
}

// dx[b][i] = (sum_o dy[b][o] w[o][i]) * (ACT == tanh ? 1 - y[b][i]^2 : 1)   (y = the input's own activation)
template <int ACT>
__global__ void __launch_bounds__(256) small_linear_dgrad_kernel(const float* __restrict__ dy,
                                                                 const float* __restrict__ w,
                                                                 const float* __restrict__ yin,
                                                                 float* __restrict__ dx, int B, int I, int O) {
    int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)B * I) return;
    int b = (int)(idx / I), i = (int)(idx % I);
    float s = 0.f;
    for (int o = 0; o < O; ++o) s = fmaf(dy[(int64_t)b * O + o], w[(int64_t)o * I + i], s);
    if (ACT == 1) {
        float t = yin[idx];
        s *= 1.f - t * t;
    }
    dx[idx] = s;
}

}  // namespace

fo_status launch_xent(const float* z, const int32_t* labels, float* dz, float* loss, int B, int C, hipStream_t s) {
    hipLaunchKernelGGL(xent_kernel, dim3(1), dim3(256), 0, s, z, labels, dz, loss, B, C);
    FO_LAUNCHED();
    return FO_OK;
}

size_t colsum_ws_floats(int rows, int N) { return (size_t)cdiv(rows, CS_ROWS) * N; }

template <typename T>
static fo_status colsum_impl(const T* X, int64_t ld, int rows, const int* rows_dev, int N, float* out, float* ws,
                             hipStream_t s) {
    int chunks = (int)cdiv(rows, CS_ROWS);
    hipLaunchKernelGGL((colsum_partial<T>), dim3(cdiv(N, 256), chunks), dim3(256), 0, s, X, ld, rows, rows_dev, N,
                       ws);
    hipLaunchKernelGGL(colsum_finish, dim3(cdiv(N, 256)), dim3(256), 0, s, ws, chunks, N, out);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_colsum(const float* X, int64_t ld, int rows, const int* rows_dev, int N, float* out, float* ws,
                        hipStream_t s) {
    return colsum_impl<float>(X, ld, rows, rows_dev, N, out, ws, s);
}
fo_status launch_colsum(const bf16_t* X, int64_t ld, int rows, const int* rows_dev, int N, float* out, float* ws,
                        hipStream_t s) {
    return colsum_impl<bf16_t>(X, ld, rows, rows_dev, N, out, ws, s);
}

fo_status launch_fill(float* p, int64_t n, float v, hipStream_t s) {
    if (n == 0) return FO_OK;
    int grid = (int)std::min<int64_t>(cdiv(n, 256), 4096);
    hipLaunchKernelGGL(fill_kernel, dim3(grid), dim3(256), 0, s, p, n, v);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_small_linear_fwd(const float* x, const float* w, const float* bias, float* y, int B, int I, int O,
                                  bool tanh_act, hipStream_t s) {
    dim3 grid((unsigned)cdiv(O, 4));
    if (tanh_act)
        hipLaunchKernelGGL((small_linear_fwd_kernel<1>), grid, dim3(256), 0, s, x, w, bias, y, B, I, O);
    else
        hipLaunchKernelGGL((small_linear_fwd_kernel<0>), grid, dim3(256), 0, s, x, w, bias, y, B, I, O);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_small_linear_bwd(const float* dy, const float* x, const float* w, const float* xin_tanh, float* gw,
                                  float* gb, float* dx, int B, int I, int O, hipStream_t s) {
    int64_t nw = std::max<int64_t>((int64_t)O * I, O);
    hipLaunchKernelGGL(small_linear_wgrad_kernel, dim3(cdiv(nw, 256)), dim3(256), 0, s, dy, x, gw, gb, B, I, O);
    if (dx) {
        if (xin_tanh)
            hipLaunchKernelGGL((small_linear_dgrad_kernel<1>), dim3(cdiv((int64_t)B * I, 256)), dim3(256), 0, s, dy,
                               w, xin_tanh, dx, B, I, O);
        else
            hipLaunchKernelGGL((small_linear_dgrad_kernel<0>), dim3(cdiv((int64_t)B * I, 256)), dim3(256), 0, s, dy,
                               w, xin_tanh, dx, B, I, O);
    }
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
