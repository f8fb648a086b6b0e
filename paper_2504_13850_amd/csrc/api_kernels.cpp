// Kernel-level C entry points (fedoptima_kernels.h): argument checks, then
// one descriptor for the MFMA GEMM.
#include <mutex>

#include "../../include/fedoptima_kernels.h"
#include "gemm.h"

using namespace fo;

// Split-K partials of fo_gemm_bf16_noalloc.  The array is part of the code
// object: every GPU the library is loaded on holds its own copy from module
// load until the process ends, and no call allocates.  In host code the name
// `scratch` is only a host-side handle; kernels get the device address that
// hipGetSymbolAddress returns for the current device.
constexpr int64_t kNoAllocScratchFloats = int64_t(4) << 20;  // 16 MiB
static __device__ __align__(256) float scratch[kNoAllocScratchFloats];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxScratchDevices] = {};  // per device, set on the first call there

// The device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept; the stream must belong to it.
fo_status scratch_ptr(hipStream_t stream, float** out) {
    int dev = -1;
    FO_HIP(hipGetDevice(&dev));
    FO_CHECK(dev >= 0 && dev < kMaxScratchDevices, "fo_gemm_bf16_noalloc: device %d beyond %d", dev,
             kMaxScratchDevices);
    if (stream) {
        int sdev = -1;
        FO_HIP(hipStreamGetDevice(stream, &sdev));
        FO_CHECK(sdev == dev, "fo_gemm_bf16_noalloc: the stream belongs to device %d, the current device is %d",
                 sdev, dev);
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        FO_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        FO_CHECK(p != nullptr, "fo_gemm_bf16_noalloc: no device address for the scratch array");
        g_scratch_ptr[dev] = (float*)p;
    }
    *out = g_scratch_ptr[dev];
    return FO_OK;
}
}  // namespace

extern "C" fo_status fo_gemm_bf16(int32_t M, int32_t N, int32_t K, int32_t a_layout, const uint16_t* A,
                                  const uint16_t* A_lo, int64_t lda, int32_t b_layout, const uint16_t* B,
                                  const uint16_t* B_lo, int64_t ldb, float* C, int64_t ldc, int32_t splits,
                                  float* workspace, void* hip_stream) {
    FO_CHECK(M >= 1 && N >= 1 && K >= 1, "fo_gemm_bf16: sizes %d x %d x %d", M, N, K);
    FO_CHECK(A && B && C, "fo_gemm_bf16: NULL operand");
    FO_CHECK(a_layout == FO_LAYOUT_ROW_K || a_layout == FO_LAYOUT_K_ROW, "fo_gemm_bf16: bad A layout");
    FO_CHECK(b_layout == FO_LAYOUT_ROW_K || b_layout == FO_LAYOUT_K_ROW, "fo_gemm_bf16: bad B layout");
    FO_CHECK(lda >= (a_layout == FO_LAYOUT_ROW_K ? K : M), "fo_gemm_bf16: lda too small");
    FO_CHECK(ldb >= (b_layout == FO_LAYOUT_ROW_K ? K : N), "fo_gemm_bf16: ldb too small");
    FO_CHECK(ldc >= N, "fo_gemm_bf16: ldc too small");
    FO_CHECK(splits >= 1 && (splits == 1 || workspace), "fo_gemm_bf16: split-K needs a workspace");
    FO_CHECK(!A_lo || B_lo, "fo_gemm_bf16: A_lo needs B_lo");
    GemmDesc d;
    d.M = M; d.N = N; d.K = K;
    d.amode = a_layout == FO_LAYOUT_ROW_K ? OP_RK : OP_KR;
    d.bmode = b_layout == FO_LAYOUT_ROW_K ? OP_RK : OP_KR;
    d.A = A; d.lda = lda; d.A2 = A_lo;
    d.B = B; d.ldb = ldb; d.B2 = B_lo;
    d.nseg = B_lo ? (A_lo ? 3 : 2) : 1;
    d.Cf = C; d.ldcf = ldc;
    d.splits = splits; d.ws = workspace;
    return gemm(d, (hipStream_t)hip_stream);
}

extern "C" fo_status fo_gemm_bf16_noalloc(int32_t M, int32_t N, int32_t K, int32_t a_layout, const uint16_t* A,
                                          const uint16_t* A_lo, int64_t lda, int32_t b_layout, const uint16_t* B,
                                          const uint16_t* B_lo, int64_t ldb, float* C, int64_t ldc, int32_t splits,
                                          void* hip_stream) {
    FO_CHECK(splits >= 1, "fo_gemm_bf16_noalloc: splits=%d", splits);
    FO_CHECK(M >= 1 && N >= 1 && K >= 1, "fo_gemm_bf16_noalloc: sizes %d x %d x %d", M, N, K);
    float* ws = nullptr;
    if (splits > 1) {
        const int64_t need = (int64_t)splits * M * N;
        FO_CHECK(need <= kNoAllocScratchFloats,
                 "fo_gemm_bf16_noalloc: %d slices of a %d x %d product need %lld floats of scratch, the limit is "
                 "%lld (16 MiB)", splits, M, N, (long long)need, (long long)kNoAllocScratchFloats);
        fo_status st = scratch_ptr((hipStream_t)hip_stream, &ws);
        if (st != FO_OK) return st;
    }
    return fo_gemm_bf16(M, N, K, a_layout, A, A_lo, lda, b_layout, B, B_lo, ldb, C, ldc, splits, ws, hip_stream);
}

extern "C" fo_status fo_conv2d_bf16(int32_t pass, int32_t Bn, int32_t H, int32_t W, int32_t Ci, int32_t Co,
                                    int32_t k, int32_t stride, int32_t pad, const uint16_t* in,
                                    const uint16_t* in_lo, const uint16_t* in2, const uint16_t* w,
                                    const uint16_t* w_lo, float* out, int32_t splits, float* workspace,
                                    void* hip_stream) {
    FO_CHECK(pass >= 0 && pass <= 2, "fo_conv2d_bf16: pass=%d", pass);
    FO_CHECK(Bn >= 1 && H >= 1 && W >= 1 && Ci >= 1 && Co >= 1 && k >= 1 && stride >= 1 && pad >= 0,
             "fo_conv2d_bf16: bad geometry");
    FO_CHECK(H + 2 * pad >= k && W + 2 * pad >= k, "fo_conv2d_bf16: kernel larger than the padded input");
    FO_CHECK(in && out && (pass == 2 ? in2 != nullptr : w != nullptr), "fo_conv2d_bf16: NULL operand");
    FO_CHECK(Ci % 8 == 0 && (pass != 0 || Ci % 64 == 0) && (pass != 1 || Co % 64 == 0),
             "fo_conv2d_bf16: channel counts not supported (Ci=%d, Co=%d)", Ci, Co);
    FO_CHECK(!in_lo || w_lo, "fo_conv2d_bf16: in_lo needs w_lo");
    FO_CHECK(splits >= 1 && (splits == 1 || workspace), "fo_conv2d_bf16: split-K needs a workspace");
    ConvGeom g;
    g.Bn = Bn; g.H = H; g.W = W; g.Ci = Ci;
    g.Ho = (H + 2 * pad - k) / stride + 1;
    g.Wo = (W + 2 * pad - k) / stride + 1;
    g.Co = Co; g.kh = k; g.kw = k; g.stride = stride; g.pad = pad;
    GemmDesc d;
    d.g = g;
    d.Cf = out;
    d.splits = splits; d.ws = workspace;
    if (pass == 0) {
        d.M = Bn * g.Ho * g.Wo; d.N = Co; d.K = k * k * Ci;
        d.amode = OP_CONV_FWD; d.A = in; d.A2 = in_lo;
        d.bmode = OP_RK; d.B = w; d.B2 = w_lo; d.ldb = d.K;
        d.nseg = w_lo ? (in_lo ? 3 : 2) : 1;
        d.ldcf = Co;
    } else if (pass == 1) {
        d.M = Bn * H * W; d.N = Ci; d.K = k * k * Co;
        d.amode = OP_CONV_DX; d.A = in;
        d.bmode = OP_CONV_DXW; d.B = w;
        d.ldcf = Ci;
    } else {
        d.M = Co; d.N = k * k * Ci; d.K = Bn * g.Ho * g.Wo;
        d.amode = OP_KR; d.A = in; d.lda = Co;
        d.bmode = OP_CONV_DWX; d.B = in2;
        d.ldcf = d.N;
    }
    return gemm(d, (hipStream_t)hip_stream);
}
