// Small kernels shared by the model executors: the loss f_s (mean softmax
// cross-entropy and its gradient), column sums (bias and norm-parameter
// gradients), fills, and small fp32 linear layers for the classifier heads.
#include "kernels.h"

namespace fo {
namespace {

// Mean softmax cross-entropy over the batch and dz = (softmax - onehot) / B.
// Labels outside [0, C) are clamped into range.
// Mean softmax cross-entropy of z [B][C] and dz = (softmax - onehot) / B.
// One wave per sample (lanes over the classes, 64 at a time; the block's 16
// waves take samples w, w + 16, ...), max and sum by wave reductions; the
// loss adds each wave's samples in order, then the waves in order.
constexpr int XENT_WAVES = 16;
__device__ __forceinline__ float xent_wave_max(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
    return v;
}
__device__ __forceinline__ float xent_wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}
__global__ void __launch_bounds__(64 * XENT_WAVES) xent_kernel(const float* __restrict__ z,
                                                               const StepIn* __restrict__ in,
                                                               float* __restrict__ dz, float* __restrict__ loss, int B,
                                                               int C) {
    __shared__ float part[XENT_WAVES];
    const int32_t* __restrict__ labels = in->labels;
    __shared__ int bad_w[XENT_WAVES];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    float mine = 0.f;
    int bad = 0;
    for (int b = w; b < B; b += XENT_WAVES) {
        const float* zr = z + (int64_t)b * C;
        float m = -INFINITY;
        for (int c = lane; c < C; c += 64) m = fmaxf(m, zr[c]);
        m = xent_wave_max(m);
        float s = 0.f;
        for (int c = lane; c < C; c += 64) s += expf(zr[c] - m);
        const float lse = m + logf(xent_wave_sum(s));
        int y = labels[b];
        if (y < 0 || y >= C) {  // counted into loss[1]; clamped so that every access stays in bounds
            bad++;
            y = y < 0 ? 0 : C - 1;
        }
        mine += lse - zr[y];
        for (int c = lane; c < C; c += 64) dz[(int64_t)b * C + c] = (expf(zr[c] - lse) - (c == y ? 1.f : 0.f)) / (float)B;
    }
    if (lane == 0) {
        part[w] = mine;
        bad_w[w] = bad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        int nb = 0;
        for (int k = 0; k < XENT_WAVES; ++k) {
            t += part[k];
            nb += bad_w[k];
        }
        loss[0] = t / (float)B;
        loss[1] = (float)nb;
    }
}

// Column sums of a [rows][N] matrix in two passes.  colsum_partial: a block
// covers 64 columns (one per lane) and CS_ROWS rows, its four waves take
// interleaved rows with eight loads in flight per lane, and the block writes
// one partial row.  colsum_finish adds the partial rows that cover valid rows,
// in chunk order (the result does not depend on scheduling).
constexpr int CS_ROWS = 128;

template <typename T>
__device__ __forceinline__ float ld_as_f(const T* p);
template <> __device__ __forceinline__ float ld_as_f<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_as_f<bf16_t>(const bf16_t* p) { return bf2f(*p); }

template <typename T>
__global__ void __launch_bounds__(256) colsum_partial(const T* __restrict__ X, int64_t ld, int rows,
                                                      const int* __restrict__ rows_dev, int N,
                                                      float* __restrict__ part) {
    __shared__ float red[4][64];
    const int R = rows_dev ? min(rows, *rows_dev) : rows;
    const int r0 = blockIdx.y * CS_ROWS;
    if (r0 >= R) return;  // uniform: this chunk holds no valid row
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = blockIdx.x * 64 + lane;
    const int r1 = min(R, r0 + CS_ROWS);
    float s = 0.f;
    if (col < N) {
        int r = r0 + wave;
        for (; r + 28 < r1; r += 32) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = ld_as_f<T>(X + (int64_t)(r + 4 * u) * ld + col);
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; r < r1; r += 4) s += ld_as_f<T>(X + (int64_t)r * ld + col);
    }
    red[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && col < N)
        part[(int64_t)blockIdx.y * N + col] = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

// colsum_partial over several matrices: blocks are dealt to the jobs in order,
// job i taking ceil(N_i / 64) x ceil(rows_i / CS_ROWS) of them (column blocks
// fastest); the arithmetic per column is colsum_partial's.
__global__ void __launch_bounds__(256) colsum_partial_multi(const ColPartJobs jobs) {
    __shared__ float red[4][64];
    int bid = blockIdx.x, ji = 0;
    for (; ji < jobs.n - 1; ++ji) {
        const int nb = ((jobs.j[ji].N + 63) / 64) * ((jobs.j[ji].rows + CS_ROWS - 1) / CS_ROWS);
        if (bid < nb) break;
        bid -= nb;
    }
    const ColPartJob& J = jobs.j[ji];
    const int ncb = (J.N + 63) / 64;
    const int by = bid / ncb, bx = bid - by * ncb;
    const int r0 = by * CS_ROWS;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = bx * 64 + lane;
    const int r1 = min(J.rows, r0 + CS_ROWS);
    float s = 0.f;
    if (col < J.N) {
        int r = r0 + wave;
        for (; r + 28 < r1; r += 32) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = J.X[(int64_t)(r + 4 * u) * J.ld + col];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; r < r1; r += 4) s += J.X[(int64_t)r * J.ld + col];
    }
    red[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && col < J.N)
        J.part[(int64_t)by * J.N + col] = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

// part[p][N] for p < ceil(min(rows, *rows_dev) / rows_per_part); column col
// goes to out.p[col / out.seg][col % out.seg].
__global__ void __launch_bounds__(256) colsum_finish(const float* __restrict__ part, int rows,
                                                     const int* __restrict__ rows_dev, int rows_per_part, int N,
                                                     ColOut out) {
    __shared__ float red[4][64];
    const int R = rows_dev ? min(rows, *rows_dev) : rows;
    const int nparts = (R + rows_per_part - 1) / rows_per_part;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = blockIdx.x * 64 + lane;
    float s = 0.f;
    if (col < N) {
        int p = wave;
        for (; p + 28 < nparts; p += 32) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(p + 4 * u) * N + col];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; p < nparts; p += 4) s += part[(int64_t)p * N + col];
    }
    red[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && col < N) {
        const int j = col / out.seg;
        out.p[j][col - j * out.seg] = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
    }
}

// colsum_finish over several jobs: blocks are dealt to the jobs in order, each
// job taking ceil(N / 64) of them.  W waves take interleaved partial rows (eight
// loads in flight per lane) and are added in wave order: with hundreds of
// partial rows per column (the LayerNorm partials, one per four rows) the
// 16-wave form keeps a wave's chain of dependent loads short.
template <int W>
__global__ void __launch_bounds__(64 * W) colsum_finish_multi(const ColJobs jobs) {
    __shared__ float red[W][64];
    int bid = blockIdx.x, ji = 0;
    while (ji < jobs.n - 1 && bid >= (jobs.j[ji].N + 63) / 64) {
        bid -= (jobs.j[ji].N + 63) / 64;
        ++ji;
    }
    const ColJob& J = jobs.j[ji];
    const int R = J.rows_dev ? min(J.rows, *J.rows_dev) : J.rows;
    const int nparts = (R + J.rows_per_part - 1) / J.rows_per_part;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = bid * 64 + lane;
    float s = 0.f;
    if (col < J.N) {
        int p = wave;
        for (; p + 7 * W < nparts; p += 8 * W) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = J.part[(int64_t)(p + W * u) * J.N + col];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; p < nparts; p += W) s += J.part[(int64_t)p * J.N + col];
    }
    red[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && col < J.N) {
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < W; w += 4) t += (red[w][lane] + red[w + 1][lane]) + (red[w + 2][lane] + red[w + 3][lane]);
        const int j = col / J.out.seg;
        J.out.p[j][col - j * J.out.seg] = t;
    }
}

__global__ void __launch_bounds__(256) fill_kernel(float* __restrict__ p, int64_t n, float v) {
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

// y[b][o] = act(bias[o] + sum_i x[b][i] w[o][i]) for I <= 64 * SL_PER.  One
// block per output o holds row o of w in registers (lanes over i); its four
// waves take the batch rows two at a time.
constexpr int SL_PER = 12;

__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

template <int ACT>
__global__ void __launch_bounds__(256) small_linear_fwd_kernel(const float* __restrict__ x, const float* __restrict__ w,
                                                               const float* __restrict__ bias, float* __restrict__ y,
                                                               int B, int I, int O) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int o = blockIdx.x;
    const float* wr = w + (int64_t)o * I;
    float wv[SL_PER];
#pragma unroll
    for (int k = 0; k < SL_PER; ++k) {
        const int i = lane + 64 * k;
        wv[k] = i < I ? wr[i] : 0.f;
    }
    const float bo = bias[o];
    // wave w takes batch rows w, w + 4, ...; eight rows at a time with all
    // their loads issued before the first product
    constexpr int RB = 8;
    for (int b0 = wave; b0 < B; b0 += 4 * RB) {
        float s[RB];
#pragma unroll
        for (int u = 0; u < RB; ++u) {
            const int b = min(b0 + 4 * u, B - 1);  // rows past B repeat row B - 1 and are not stored
            const float* xr = x + (int64_t)b * I;
            float xv[SL_PER];
#pragma unroll
            for (int k = 0; k < SL_PER; ++k) {
                const int i = lane + 64 * k;
                xv[k] = i < I ? xr[i] : 0.f;
            }
            float a = 0.f;
#pragma unroll
            for (int k = 0; k < SL_PER; ++k) a = fmaf(xv[k], wv[k], a);
            s[u] = a;
        }
#pragma unroll
        for (int u = 0; u < RB; ++u) s[u] = wave_sum64(s[u]);
        if (lane == 0) {
#pragma unroll
            for (int u = 0; u < RB; ++u) {
                const int b = b0 + 4 * u;
                if (b < B) {
                    const float v = s[u] + bo;
                    y[(int64_t)b * O + o] = ACT == 1 ? tanhf(v) : v;
                }
            }
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
        // batch rows eight at a time, their loads issued together; one running sum
        float s = 0.f;
        int b = 0;
        for (; b + 8 <= B; b += 8) {
            float dv[8], xv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                dv[u] = dy[(int64_t)(b + u) * O + o];
                xv[u] = x[(int64_t)(b + u) * I + i];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) s = fmaf(dv[u], xv[u], s);
        }
        for (; b < B; ++b) s = fmaf(dy[(int64_t)b * O + o], x[(int64_t)b * I + i], s);
        gw[idx] = s;
    }
    if (idx < O) {
        float s = 0.f;
        for (int b = 0; b < B; ++b) s += dy[(int64_t)b * O + idx];
        gb[idx] = s;
    }
}

// Input gradient of a small linear layer, dx[b][i] = sum_o dy[b][o] w[o][i],
// as partial sums over chunks of SD_K outputs: block (i-tile, o-chunk, b-group)
// stages w[o-chunk][i-tile] and dy[b-group][o-chunk] in LDS and writes
// part[o-chunk][b][i]; small_linear_dgrad_finish adds the chunks in order and
// applies the derivative of the input's tanh when given.
constexpr int SD_K = 64, SD_I = 64, SD_B = 32;

__global__ void __launch_bounds__(256) small_linear_dgrad_partial(const float* __restrict__ dy,
                                                                  const float* __restrict__ w, float* __restrict__ part,
                                                                  int B, int I, int O) {
    __shared__ float ws[SD_K][SD_I];
    __shared__ float ds[SD_B][SD_K + 1];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int i0 = blockIdx.x * SD_I, o0 = blockIdx.y * SD_K, b0 = blockIdx.z * SD_B;
    for (int e = tid; e < SD_K * SD_I; e += 256) {
        const int ok = e / SD_I, ii = e % SD_I;
        ws[ok][ii] = (o0 + ok < O && i0 + ii < I) ? w[(int64_t)(o0 + ok) * I + i0 + ii] : 0.f;
    }
    for (int e = tid; e < SD_B * SD_K; e += 256) {
        const int bb = e / SD_K, ok = e % SD_K;
        ds[bb][ok] = (b0 + bb < B && o0 + ok < O) ? dy[(int64_t)(b0 + bb) * O + o0 + ok] : 0.f;
    }
    __syncthreads();
    // lane: column i0 + lane; wave: batch rows b0 + wave + 4 j
    float acc[SD_B / 4];
#pragma unroll
    for (int j = 0; j < SD_B / 4; ++j) acc[j] = 0.f;
#pragma unroll 8
    for (int k = 0; k < SD_K; ++k) {
        const float wk = ws[k][lane];
#pragma unroll
        for (int j = 0; j < SD_B / 4; ++j) acc[j] = fmaf(ds[wave + 4 * j][k], wk, acc[j]);
    }
    const int i = i0 + lane;
    if (i < I) {
#pragma unroll
        for (int j = 0; j < SD_B / 4; ++j) {
            const int b = b0 + wave + 4 * j;
            if (b < B) part[((int64_t)blockIdx.y * B + b) * I + i] = acc[j];
        }
    }
}

__global__ void __launch_bounds__(256) small_linear_dgrad_finish(const float* __restrict__ part, int chunks,
                                                                 const float* __restrict__ yin,
                                                                 float* __restrict__ dx, int64_t n) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= n) return;
    float s = 0.f;
    int c = 0;
    for (; c + 3 < chunks; c += 4) {
        const float v0 = part[(int64_t)c * n + idx], v1 = part[(int64_t)(c + 1) * n + idx];
        const float v2 = part[(int64_t)(c + 2) * n + idx], v3 = part[(int64_t)(c + 3) * n + idx];
        s += (v0 + v1) + (v2 + v3);
    }
    for (; c < chunks; ++c) s += part[(int64_t)c * n + idx];
    if (yin) {
        const float t = yin[idx];
        s *= 1.f - t * t;
    }
    dx[idx] = s;
}

}  // namespace

fo_status launch_xent(const float* z, const StepIn* in, float* dz, float* loss, int B, int C, hipStream_t s) {
    hipLaunchKernelGGL(xent_kernel, dim3(1), dim3(64 * XENT_WAVES), 0, s, z, in, dz, loss, B, C);
    FO_LAUNCHED();
    return FO_OK;
}

size_t colsum_ws_floats(int rows, int N) { return (size_t)cdiv(rows, CS_ROWS) * N; }

fo_status launch_colsum_finish(const float* part, int rows, const int* rows_dev, int rows_per_part, int N,
                               const ColOut& out, hipStream_t s) {
    FO_CHECK(out.seg > 0 && cdiv(N, out.seg) <= 3, "colsum: %d columns in segments of %d", N, out.seg);
    hipLaunchKernelGGL(colsum_finish, dim3(cdiv(N, 64)), dim3(256), 0, s, part, rows, rows_dev, rows_per_part, N,
                       out);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_colsum_partial_multi(const ColPartJobs& jobs, hipStream_t s) {
    FO_CHECK(jobs.n >= 1 && jobs.n <= kColJobsMax, "colsum: %d jobs", jobs.n);
    int64_t blocks = 0;
    for (int i = 0; i < jobs.n; ++i) {
        const ColPartJob& J = jobs.j[i];
        FO_CHECK(J.X && J.part && J.N > 0 && J.rows > 0 && J.ld >= J.N, "colsum: bad partial job %d", i);
        blocks += cdiv(J.N, 64) * cdiv(J.rows, CS_ROWS);
    }
    hipLaunchKernelGGL(colsum_partial_multi, dim3((unsigned)blocks), dim3(256), 0, s, jobs);
    FO_LAUNCHED();
    return FO_OK;
}

void ColSums::add(const float* X, int64_t ld, int rows, int N, float* part, float* out) {
    if (parts.n >= kColJobsMax) {  // launch_colsums refuses the set
        parts.n = kColJobsMax + 1;
        return;
    }
    ColPartJob& p = parts.j[parts.n++];
    p.X = X; p.ld = ld; p.rows = rows; p.N = N; p.part = part;
    ColJob& f = fin.j[fin.n++];
    f.part = part; f.rows = rows; f.rows_per_part = CS_ROWS; f.N = N;
    f.out.p[0] = out; f.out.seg = N;
}

fo_status launch_colsums(const ColSums& c, hipStream_t s) {
    FO_CHECK(c.parts.n <= kColJobsMax, "colsum: more than %d matrices in one pass", kColJobsMax);
    if (c.parts.n == 0) return FO_OK;
    fo_status st = launch_colsum_partial_multi(c.parts, s);
    return st != FO_OK ? st : launch_colsum_finish_multi(c.fin, s);
}

// partial rows per column above which the finish runs 16 waves per block
constexpr int kFinishWide = 64;

fo_status launch_colsum_finish_multi(const ColJobs& jobs, hipStream_t s) {
    FO_CHECK(jobs.n >= 1 && jobs.n <= kColJobsMax, "colsum: %d jobs", jobs.n);
    int blocks = 0, most = 0;
    for (int i = 0; i < jobs.n; ++i) {
        const ColJob& J = jobs.j[i];
        FO_CHECK(J.part && J.N > 0 && J.rows_per_part > 0 && J.out.seg > 0 && cdiv(J.N, J.out.seg) <= 3,
                 "colsum: bad job %d", i);
        blocks += (int)cdiv(J.N, 64);
        most = std::max(most, (int)cdiv(J.rows, J.rows_per_part));
    }
    if (most > kFinishWide)
        hipLaunchKernelGGL(colsum_finish_multi<16>, dim3(blocks), dim3(1024), 0, s, jobs);
    else
        hipLaunchKernelGGL(colsum_finish_multi<4>, dim3(blocks), dim3(256), 0, s, jobs);
    FO_LAUNCHED();
    return FO_OK;
}

int colsum_rows_per_part() { return CS_ROWS; }

fo_status launch_colsum_partial(const bf16_t* X, int64_t ld, int rows, const int* rows_dev, int N, float* ws,
                                hipStream_t s) {
    if (rows <= 0 || N <= 0) return FO_OK;
    hipLaunchKernelGGL((colsum_partial<bf16_t>), dim3(cdiv(N, 64), cdiv(rows, CS_ROWS)), dim3(256), 0, s, X, ld,
                       rows, rows_dev, N, ws);
    FO_LAUNCHED();
    return FO_OK;
}

template <typename T>
static fo_status colsum_impl(const T* X, int64_t ld, int rows, const int* rows_dev, int N, float* out, float* ws,
                             hipStream_t s) {
    if (rows <= 0 || N <= 0) return FO_OK;
    // one chunk of rows: its partial row is the sum, written straight to out
    const bool one = !rows_dev && rows <= CS_ROWS;
    hipLaunchKernelGGL((colsum_partial<T>), dim3(cdiv(N, 64), cdiv(rows, CS_ROWS)), dim3(256), 0, s, X, ld, rows,
                       rows_dev, N, one ? out : ws);
    FO_LAUNCHED();
    if (one) return FO_OK;
    ColOut o;
    o.p[0] = out;
    o.seg = N;
    return launch_colsum_finish(ws, rows, rows_dev, CS_ROWS, N, o, s);
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
    FO_CHECK(I <= 64 * SL_PER, "small linear: %d inputs (at most %d)", I, 64 * SL_PER);
    if (B <= 0 || O <= 0) return FO_OK;
    if (tanh_act)
        hipLaunchKernelGGL((small_linear_fwd_kernel<1>), dim3(O), dim3(256), 0, s, x, w, bias, y, B, I, O);
    else
        hipLaunchKernelGGL((small_linear_fwd_kernel<0>), dim3(O), dim3(256), 0, s, x, w, bias, y, B, I, O);
    FO_LAUNCHED();
    return FO_OK;
}

size_t small_linear_ws_floats(int B, int I, int O) { return (size_t)cdiv(O, SD_K) * B * I; }

fo_status launch_small_linear_bwd(const float* dy, const float* x, const float* w, const float* xin_tanh, float* gw,
                                  float* gb, float* dx, int B, int I, int O, float* ws, hipStream_t s) {
    int64_t nw = std::max<int64_t>((int64_t)O * I, O);
    hipLaunchKernelGGL(small_linear_wgrad_kernel, dim3(cdiv(nw, 256)), dim3(256), 0, s, dy, x, gw, gb, B, I, O);
    if (dx) {
        const int chunks = (int)cdiv(O, SD_K);
        hipLaunchKernelGGL(small_linear_dgrad_partial, dim3(cdiv(I, SD_I), chunks, cdiv(B, SD_B)), dim3(256), 0, s,
                           dy, w, ws, B, I, O);
        const int64_t n = (int64_t)B * I;
        hipLaunchKernelGGL(small_linear_dgrad_finish, dim3(cdiv(n, 256)), dim3(256), 0, s, ws, chunks, xin_tanh, dx,
                           n);
    }
    FO_LAUNCHED();
    return FO_OK;
}

}  // namespace fo
