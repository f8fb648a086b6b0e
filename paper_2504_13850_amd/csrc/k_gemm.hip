// bf16 MFMA GEMM / implicit-GEMM convolution for gfx950 (CDNA4).
//
// Tiling: a 256-thread workgroup (4 waves of 64) computes a 128x128 tile of C;
// each wave owns a 64x64 sub-tile = 2x2 v_mfma_f32_32x32x16_bf16 accumulators
// (64 fp32 per lane).  Four kernels share the tile, its XCD-aware order and its
// fused epilogue:
//  - gemm_kernel: the general form (any operand layout, unaligned sizes,
//    implicit-GEMM convolution operands).  K advances in tiles of 64 through
//    two LDS buffers, staged through registers; LDS tiles hold 128 rows x 64 k
//    with an XOR swizzle of the 16-byte chunks.  Operands whose rows are
//    contiguous in memory are either transposed on their way into LDS (k
//    pairs packed into 32-bit stores) or stored [k][row] and read back with
//    the LDS transpose read.
//  - gemm_comp_dma_kernel: compensated products of row-major operands
//    (A.B + A.B_lo + A_lo.B in one pass over K), tiles copied straight into
//    LDS by global_load_lds in a two-stage ring.
//  - gemm_wgrad_dma_kernel: groups of products of two k-major operands
//    (weight gradients), tiles copied into LDS in the [k][row] layout and read
//    by transpose reads, four-stage ring; gemm_wgrad_tall_kernel, the same on
//    256 x 128 tiles (128 x 64 per wave) for groups that share the GPU.
//  - gemm_rk_krt_dma_kernel: row-major A times k-major B (input gradients),
//    the same copies and ring.
#include <algorithm>
#include <type_traits>

#include <hip/hip_ext.h>

#include "gemm.h"
#include "kernels.h"
#include "prof.h"

namespace fo {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64, NT = 256;
// Rings of the kernels with copies into LDS: weight gradients in 32-deep K
// tiles, four stages; input gradients four stages (64 KB of LDS each, two
// workgroups per CU: deeper rings at one workgroup per CU starve the
// concurrent input-gradient chain of LDS).
constexpr int kWgradKT = 32, kWgradNST = 4, kDgradKT = 32, kDgradNST = 4;
constexpr int NV = BM * BK / 8 / NT;  // 16-byte vectors per thread per operand per K tile (4)

// LDS tiles are 128 rows x 64 k with rows padded to 72 elements (144 B = 36
// banks): 8 consecutive rows start 4 banks apart, so the 128-bit operand reads
// (8 rows, one 16-byte chunk each) and the row-contiguous stores are bank
// conflict free, and every read of a lane is its own base plus a constant.
constexpr int LDR = BK + 8;
__device__ __forceinline__ int lds_idx(int row, int k) { return row * LDR + k; }

__device__ __forceinline__ uint16_t half_of(const uint4& v, int e) {
    uint32_t w = e < 2 ? v.x : e < 4 ? v.y : e < 6 ? v.z : v.w;
    return (e & 1) ? (uint16_t)(w >> 16) : (uint16_t)(w & 0xFFFFu);
}

__device__ __forceinline__ uint4 load8(const bf16_t* p) { return *reinterpret_cast<const uint4*>(p); }

// Sixteen zero bytes in device memory (never written): the source of the
// chunks of an aligned tile that lie outside the operand.
__device__ __attribute__((aligned(16))) bf16_t kZero8[8];

__device__ __forceinline__ uint4 load8_guarded(const bf16_t* p, int n_ok) {
    // first n_ok (0..8) elements from p, rest zero
    uint16_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = e < n_ok ? p[e] : (uint16_t)0;
    uint4 v;
    v.x = h[0] | ((uint32_t)h[1] << 16);
    v.y = h[2] | ((uint32_t)h[3] << 16);
    v.z = h[4] | ((uint32_t)h[5] << 16);
    v.w = h[6] | ((uint32_t)h[7] << 16);
    return v;
}

// ------------------------------------------------------------------ loaders
// A loader keeps the address state of its thread; load() fills NV registers
// for the K tile starting at kb (operand base P passed per tile, so that
// compensated products can switch between high and low parts), store() puts
// them into an LDS tile.

// Row-major, k contiguous: rows (tid/8) + 32 v, k chunk (tid % 8) * 8.
struct LdRK {
    int64_t off[NV];  // row offsets, -1 past the last row
    int kc;
    bool vec;   // 16-byte aligned rows
    bool full;  // all 128 rows of the tile exist (uniform over the workgroup)
    __device__ void init(const bf16_t* P, int64_t ld, int r0, int R, int tid) {
        kc = (tid & 7) * 8;
        vec = (ld % 8 == 0) && (((uintptr_t)P & 15) == 0);
        full = r0 + BM <= R;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int gr = r0 + (tid >> 3) + 32 * v;
            off[v] = gr < R ? (int64_t)gr * ld : -1;
        }
    }
    __device__ void load(const bf16_t* P, int kb, int kend, uint4* r) const {
        const int k = kb + kc;
        if (vec && full && kb + BK <= kend) {  // interior tile: no checks (a uniform branch)
#pragma unroll
            for (int v = 0; v < NV; ++v) r[v] = load8(P + off[v] + k);
            return;
        }
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            if (off[v] < 0 || k >= kend) r[v] = make_uint4(0, 0, 0, 0);
            else if (vec && k + 8 <= kend) r[v] = load8(P + off[v] + k);
            else r[v] = load8_guarded(P + off[v] + k, kend - k);
        }
    }
    // Aligned operands (16-byte rows, K and kend multiples of 8): every 8-element
    // chunk is wholly inside or wholly outside, so one predicated 16-byte load
    // per chunk covers the edges as well.
    // Every load is issued (an outside chunk reads kZero8), so the number of
    // loads in flight is static and the wait before the LDS store covers only
    // the older register set.
    __device__ void load_al(const bf16_t* P, int kb, int kend, uint4* r) const {
        const int k = kb + kc;
#pragma unroll
        for (int v = 0; v < NV; ++v) r[v] = load8(off[v] >= 0 && k < kend ? P + off[v] + k : kZero8);
    }
    __device__ void store(bf16_t* t, const uint4* r, int tid) const {
#pragma unroll
        for (int v = 0; v < NV; ++v) *reinterpret_cast<uint4*>(&t[lds_idx((tid >> 3) + 32 * v, kc)]) = r[v];
    }
};

// Rows contiguous: per thread the k pair (2 kp, 2 kp + 1), kp = tid % 32, and
// two chunks of 8 rows, rc_q = (tid / 32) * 8 + 64 q.  Register v = 2 q + j holds
// k row 2 kp + j; the store transposes into (k, k+1) dword pairs.
struct LdKRBase {
    int kp, rc;
    __device__ void store(bf16_t* t, const uint4* r, int) const {
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                uint32_t w = (uint32_t)half_of(r[2 * q], e) | ((uint32_t)half_of(r[2 * q + 1], e) << 16);
                *reinterpret_cast<uint32_t*>(&t[lds_idx(rc + 64 * q + e, 2 * kp)]) = w;
            }
    }
};

// Rows contiguous (k-major memory [k][R]): thread = (k quad kq = tid % 16, row
// chunk tid / 16); register j holds k row 4 kq + j at rows rr0 .. rr0 + 7, and the
// store packs the four k values of each row into one 8-byte LDS write (a
// wave's writes of one row offset cover 64 banks without conflict).
struct LdKR {
    int64_t ld;
    int kq, mrow, rr0, R;
    bool vec, full;
    __device__ void init(const bf16_t* P, int64_t ld_, int r0, int R_, int tid) {
        ld = ld_;
        R = R_;
        kq = tid & 15;
        mrow = (tid >> 4) * 8;
        rr0 = r0 + mrow;
        vec = (ld % 8 == 0) && (((uintptr_t)P & 15) == 0);
        full = r0 + BM <= R;
    }
    __device__ void load(const bf16_t* P, int kb, int kend, uint4* r) const {
        if (vec && full && kb + BK <= kend) {  // interior tile: no checks (a uniform branch)
#pragma unroll
            for (int j = 0; j < 4; ++j) r[j] = load8(P + (int64_t)(kb + 4 * kq + j) * ld + rr0);
            return;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = kb + 4 * kq + j;
            if (k >= kend || rr0 >= R) r[j] = make_uint4(0, 0, 0, 0);
            else if (vec && rr0 + 8 <= R) r[j] = load8(P + (int64_t)k * ld + rr0);
            else r[j] = load8_guarded(P + (int64_t)k * ld + rr0, R - rr0);
        }
    }
    // Aligned operands (16-byte rows, R a multiple of 8): predicated 16-byte
    // loads, always issued as in LdRK::load_al.
    __device__ void load_al(const bf16_t* P, int kb, int kend, uint4* r) const {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = kb + 4 * kq + j;
            r[j] = load8(k < kend && rr0 < R ? P + (int64_t)k * ld + rr0 : kZero8);
        }
    }
    __device__ void store(bf16_t* t, const uint4* r, int) const {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            uint2 w;
            w.x = (uint32_t)half_of(r[0], e) | ((uint32_t)half_of(r[1], e) << 16);
            w.y = (uint32_t)half_of(r[2], e) | ((uint32_t)half_of(r[3], e) << 16);
            *reinterpret_cast<uint2*>(&t[lds_idx(mrow + e, 4 * kq)]) = w;
        }
    }
};


// Rows contiguous, aligned (16-byte rows, R a multiple of 8), staged without a
// transpose: the LDS tile is [64 k][128 rows] and the MFMA operand fragments
// come out of it through the LDS transpose read (ds_read_b64_tr_b16).  Thread
// = (row chunk c = tid % 16, k row kr = tid / 16): register j holds k row
// kr + 16 j, rows r0 + 8 c .. + 7, so every 16 lanes load and store one whole
// k row (256 B).  Row segments of 32 elements (64 B) are XOR-swizzled by
// k mod 4: the four k rows that half a wave's transpose read touches then fall
// in distinct 64-byte bank groups.
template <int R = BM>
__device__ __forceinline__ int kr_idx(int k, int r) { return k * R + (r ^ ((k & 3) << 5)); }

struct LdKRt {
    int64_t base;  // element offset of (k row kr, row r0 + 8 c)
    int64_t ld;
    int kr, rc;
    bool rowok, full;
    __device__ void init(const bf16_t* P, int64_t ld_, int r0, int R, int tid) {
        ld = ld_;
        kr = tid >> 4;
        rc = (tid & 15) * 8;
        rowok = r0 + rc < R;
        full = r0 + BM <= R;
        base = (int64_t)kr * ld + r0 + rc;
    }
    // every load is issued (an outside chunk reads kZero8), as in LdRK::load_al
    __device__ void load_al(const bf16_t* P, int kb, int kend, uint4* r) const {
        const bf16_t* p = P + base + (int64_t)kb * ld;
        if (full && kb + BK <= kend) {  // interior tile (uniform)
#pragma unroll
            for (int j = 0; j < 4; ++j) r[j] = load8(p + 16 * j * ld);
            return;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) r[j] = load8(rowok && kb + kr + 16 * j < kend ? p + 16 * j * ld : kZero8);
    }
    __device__ void store(bf16_t* t, const uint4* r, int) const {
#pragma unroll
        for (int j = 0; j < 4; ++j) *reinterpret_cast<uint4*>(&t[kr_idx(kr + 16 * j, rc)]) = r[j];
    }
};

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

// One 32 x 16 MFMA operand fragment (lane l: row l % 32, k = 8 (l / 32) .. + 7)
// from a [k][row] tile: two transpose reads of four k each.  Within a group of
// 16 lanes the read hands lane i element i % 4 of the 8 bytes addressed by lane
// 4 j + i / 4, for j = 0..3; so lane (g = l / 16, s = l % 16) addresses k row
// 8 (g / 2) + s / 4 (+ 4 for the second read), rows 16 (g % 2) + 4 (s % 4)
// .. + 3 of the fragment.  off.x / off.y are those addresses for k block 0
// (the swizzle depends on k mod 4 only, so block kb adds 16 kb rows).
__device__ __forceinline__ bf16x8_t frag_tr(const bf16_t* T, int2 off, int kadd) {
    const s16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(T + off.x + kadd));
    const s16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(T + off.y + kadd));
    const s16x8_t v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8_t, v);
}
template <int R = BM>
__device__ __forceinline__ int2 frag_tr_off(int lane, int row0) {
    const int g = lane >> 4, s = lane & 15;
    const int k = 8 * (g >> 1) + (s >> 2), r = row0 + 16 * (g & 1) + 4 * (s & 3);
    return make_int2(kr_idx<R>(k, r), kr_idx<R>(k + 4, r));
}

// Conv forward A: rows = output pixels (b, oy, ox); k = (ky, kx, ci), Ci % 64 == 0
// so that a K tile lies within one filter tap.
struct LdConvFwd {
    ConvGeom g;
    int kc, b[NV], oy[NV], ox[NV];
    bool ok[NV];
    __device__ void init(const bf16_t*, const ConvGeom& g_, int r0, int R, int tid) {
        g = g_;
        kc = (tid & 7) * 8;
        const int hw = g.Ho * g.Wo;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int gr = r0 + (tid >> 3) + 32 * v;
            ok[v] = gr < R;
            b[v] = gr / hw;
            const int rem = gr - b[v] * hw;
            oy[v] = rem / g.Wo;
            ox[v] = rem - oy[v] * g.Wo;
        }
    }
    __device__ void load(const bf16_t* X, int kb, int kend, uint4* r) const {
        const int tap = kb / g.Ci, ci = kb - tap * g.Ci + kc;
        const int ky = tap / g.kw, kx = tap - ky * g.kw;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int iy = oy[v] * g.stride - g.pad + ky, ix = ox[v] * g.stride - g.pad + kx;
            const bool in = ok[v] && kb + kc < kend && iy >= 0 && iy < g.H && ix >= 0 && ix < g.W;
            r[v] = in ? load8(X + (((int64_t)b[v] * g.H + iy) * g.W + ix) * g.Ci + ci) : make_uint4(0, 0, 0, 0);
        }
    }
    __device__ void store(bf16_t* t, const uint4* r, int tid) const {
#pragma unroll
        for (int v = 0; v < NV; ++v) *reinterpret_cast<uint4*>(&t[lds_idx((tid >> 3) + 32 * v, kc)]) = r[v];
    }
};

// Conv input-gradient A: rows = input pixels (b, iy, ix); k = (ky, kx, co) over dY, Co % 64 == 0.
struct LdConvDx {
    ConvGeom g;
    int kc, b[NV], iy[NV], ix[NV];
    bool ok[NV];
    __device__ void init(const bf16_t*, const ConvGeom& g_, int r0, int R, int tid) {
        g = g_;
        kc = (tid & 7) * 8;
        const int hw = g.H * g.W;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int gr = r0 + (tid >> 3) + 32 * v;
            ok[v] = gr < R;
            b[v] = gr / hw;
            const int rem = gr - b[v] * hw;
            iy[v] = rem / g.W;
            ix[v] = rem - iy[v] * g.W;
        }
    }
    // (every load is issued, zero-filled outside: usable by the aligned kernel)
    __device__ void load_al(const bf16_t* P, int kb, int kend, uint4* r) const { load(P, kb, kend, r); }
    __device__ void load(const bf16_t* DY, int kb, int kend, uint4* r) const {
        const int tap = kb / g.Co, co = kb - tap * g.Co + kc;
        const int ky = tap / g.kw, kx = tap - ky * g.kw;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int ty = iy[v] + g.pad - ky, tx = ix[v] + g.pad - kx;
            bool in = ok[v] && kb + kc < kend && ty >= 0 && tx >= 0;
            int oy = 0, ox = 0;
            if (in) {
                oy = ty / g.stride;
                ox = tx / g.stride;
                in = (oy * g.stride == ty) && (ox * g.stride == tx) && oy < g.Ho && ox < g.Wo;
            }
            r[v] = in ? load8(DY + (((int64_t)b[v] * g.Ho + oy) * g.Wo + ox) * g.Co + co) : make_uint4(0, 0, 0, 0);
        }
    }
    __device__ void store(bf16_t* t, const uint4* r, int tid) const {
#pragma unroll
        for (int v = 0; v < NV; ++v) *reinterpret_cast<uint4*>(&t[lds_idx((tid >> 3) + 32 * v, kc)]) = r[v];
    }
};

// Conv input-gradient B: rows = ci, k = (ky, kx, co): W[co][ky][kx][ci], ci contiguous.
struct LdConvDxW : LdKRBase {
    ConvGeom g;
    int r;
    __device__ void init(const bf16_t*, const ConvGeom& g_, int r0, int R, int tid) {
        g = g_;
        kp = tid & 31;
        rc = (tid >> 5) * 8;
        r = r0 + rc;
        (void)R;
    }
    __device__ void load(const bf16_t* Wt, int kb, int kend, uint4* o) const {
        const int tap = kb / g.Co;
        const int KK = g.kh * g.kw;
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int k = kb + 2 * kp + j, co = k - tap * g.Co, rr = r + 64 * q;
                const bool in = k < kend && rr < g.Ci;
                o[2 * q + j] = in ? load8(Wt + ((int64_t)co * KK + tap) * g.Ci + rr) : make_uint4(0, 0, 0, 0);
            }
    }
};

// The same operand staged untransposed for the LDS transpose read (as LdKRt):
// tile [64 k = co][128 rows = ci] of one filter tap (Co % 64 == 0, Ci % 8 == 0),
// sixteen lanes per k row.
struct LdConvDxWt {
    ConvGeom g;
    int kr, rl, rc;  // k row, row within the tile, operand row (ci)
    bool rowok;
    int64_t ldk;     // elements between consecutive co
    __device__ void init(const bf16_t*, const ConvGeom& g_, int r0, int R, int tid) {
        g = g_;
        kr = tid >> 4;
        rl = (tid & 15) * 8;
        rc = r0 + rl;
        rowok = rc < R;
        ldk = (int64_t)g.kh * g.kw * g.Ci;
    }
    __device__ void load_al(const bf16_t* Wt, int kb, int kend, uint4* o) const {
        const int tap = kb / g.Co, co0 = kb - tap * g.Co;
        const bf16_t* p = Wt + (int64_t)(co0 + kr) * ldk + (int64_t)tap * g.Ci + rc;
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = load8(rowok && kb + kr + 16 * j < kend ? p + 16 * j * ldk : kZero8);
    }
    __device__ void store(bf16_t* t, const uint4* r, int) const {
#pragma unroll
        for (int j = 0; j < 4; ++j) *reinterpret_cast<uint4*>(&t[kr_idx(kr + 16 * j, rl)]) = r[j];
    }
};

// Conv weight-gradient B: rows = (ky, kx, ci), k = output pixel; reads the input NHWC.
struct LdConvDwX : LdKRBase {
    ConvGeom g;
    int ky[2], kx[2], ci[2];
    bool rok[2];
    __device__ void init(const bf16_t*, const ConvGeom& g_, int r0, int R, int tid) {
        g = g_;
        kp = tid & 31;
        rc = (tid >> 5) * 8;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int n = r0 + rc + 64 * q;
            rok[q] = n < R;
            const int tap = n / g.Ci;
            ci[q] = n - tap * g.Ci;
            ky[q] = tap / g.kw;
            kx[q] = tap - ky[q] * g.kw;
        }
    }
    // (every load is issued, zero-filled outside: usable by the aligned kernel)
    __device__ void load_al(const bf16_t* P, int kb, int kend, uint4* r) const { load(P, kb, kend, r); }
    __device__ void load(const bf16_t* X, int kb, int kend, uint4* o) const {
        const int hw = g.Ho * g.Wo;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int pix = kb + 2 * kp + j;
            int b = 0, oy = 0, ox = 0;
            const bool pin = pix < kend;
            if (pin) {
                b = pix / hw;
                const int rem = pix - b * hw;
                oy = rem / g.Wo;
                ox = rem - oy * g.Wo;
            }
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int iy = oy * g.stride - g.pad + ky[q], ix = ox * g.stride - g.pad + kx[q];
                const bool in = pin && rok[q] && iy >= 0 && iy < g.H && ix >= 0 && ix < g.W;
                o[2 * q + j] = in ? load8(X + (((int64_t)b * g.H + iy) * g.W + ix) * g.Ci + ci[q])
                                  : make_uint4(0, 0, 0, 0);
            }
        }
    }
};

// The same operand staged untransposed for the LDS transpose read: tile
// [64 k = output pixels][128 rows = (ky, kx, ci)].  Thread = one pixel (tid / 4)
// and four 8-row chunks 8 (tid % 4 + 4 j), so a thread decomposes one pixel
// per K tile; four lanes read 64 contiguous bytes of one input pixel.
struct LdConvDwXt {
    ConvGeom g;
    int kr, c0;
    int ky[4], kx[4], ci[4];
    bool rok[4];
    __device__ void init(const bf16_t*, const ConvGeom& g_, int r0, int R, int tid) {
        g = g_;
        kr = tid >> 2;
        c0 = (tid & 3) * 8;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = r0 + c0 + 32 * j;
            rok[j] = n < R;
            const int tap = n / g.Ci;
            ci[j] = n - tap * g.Ci;
            ky[j] = tap / g.kw;
            kx[j] = tap - ky[j] * g.kw;
        }
    }
    __device__ void load_al(const bf16_t* X, int kb, int kend, uint4* o) const {
        const int pix = kb + kr, hw = g.Ho * g.Wo;
        const bool pin = pix < kend;
        const int b = pix / hw, rem = pix - b * hw, oy = rem / g.Wo, ox = rem - oy * g.Wo;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int iy = oy * g.stride - g.pad + ky[j], ix = ox * g.stride - g.pad + kx[j];
            const bool in = pin && rok[j] && iy >= 0 && iy < g.H && ix >= 0 && ix < g.W;
            o[j] = load8(in ? X + (((int64_t)b * g.H + iy) * g.W + ix) * g.Ci + ci[j] : kZero8);
        }
    }
    __device__ void store(bf16_t* t, const uint4* r, int) const {
#pragma unroll
        for (int j = 0; j < 4; ++j) *reinterpret_cast<uint4*>(&t[kr_idx(kr, c0 + 32 * j)]) = r[j];
    }
};

template <int MODE>
struct LoaderOf;
template <> struct LoaderOf<OP_RK> { typedef LdRK T; };
template <> struct LoaderOf<OP_KR> { typedef LdKR T; };
template <> struct LoaderOf<OP_CONV_FWD> { typedef LdConvFwd T; };
template <> struct LoaderOf<OP_CONV_DX> { typedef LdConvDx T; };
template <> struct LoaderOf<OP_CONV_DXW> { typedef LdConvDxW T; };
template <> struct LoaderOf<OP_CONV_DWX> { typedef LdConvDwX T; };
constexpr int OP_KRT = 6;  // OP_KR staged untransposed, read through the LDS transpose
template <> struct LoaderOf<OP_KRT> { typedef LdKRt T; };
constexpr int OP_CONV_DXWT = 7;  // OP_CONV_DXW staged untransposed, read through the LDS transpose
template <> struct LoaderOf<OP_CONV_DXWT> { typedef LdConvDxWt T; };
constexpr int OP_CONV_DWXT = 8;  // OP_CONV_DWX staged untransposed, read through the LDS transpose
template <> struct LoaderOf<OP_CONV_DWXT> { typedef LdConvDwXt T; };

template <int MODE>
__device__ __forceinline__ void loader_init(typename LoaderOf<MODE>::T& L, const bf16_t* P, int64_t ld,
                                            const ConvGeom& g, int r0, int R, int tid) {
    if constexpr (MODE == OP_RK || MODE == OP_KR || MODE == OP_KRT)
        L.init(P, ld, r0, R, tid);
    else
        L.init(P, g, r0, R, tid);
}

// ------------------------------------------------------------------ epilogue
// Standard normal CDF without a library erf: Phi(-|x|) = erfc(z) / 2 with
// z = |x| / sqrt(2), and erfc(z) = t exp(-z^2 + P(t)), t = 1 / (1 + z / 2), P
// the degree-9 Chebyshev fit of Numerical Recipes' erfcc (fractional error
// below 1.2e-7 for every z >= 0).  In fp32 the GELU built on it is within
// 4e-7 absolute and 2e-5 relative of the exact one over the whole real line.
__device__ __forceinline__ float norm_cdf(float x) {
    const float z = fabsf(x) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.5f, z, 1.f));
    float p = 0.17087277f;
    p = fmaf(p, t, -0.82215223f);
    p = fmaf(p, t, 1.48851587f);
    p = fmaf(p, t, -1.13520398f);
    p = fmaf(p, t, 0.27886807f);
    p = fmaf(p, t, -0.18628806f);
    p = fmaf(p, t, 0.09678418f);
    p = fmaf(p, t, 0.37409196f);
    p = fmaf(p, t, 1.00002368f);
    p = fmaf(p, t, -1.26551223f);
    const float q = 0.5f * t * __expf(fmaf(-z, z, p));  // Phi(-|x|)
    return x >= 0.f ? 1.f - q : q;
}
__device__ __forceinline__ float gelu_f(float x) { return x * norm_cdf(x); }
// GELU(x) = x Phi(x) and its derivative Phi(x) + x phi(x), sharing Phi(x)
__device__ __forceinline__ float gelu_and_grad(float x, float* grad) {
    const float p = norm_cdf(x);
    *grad = fmaf(x, 0.39894228040143268f * __expf(-0.5f * x * x), p);
    return x * p;
}

// The epilogue in two halves: epi_load fetches the per-element operands
// (residual, ReLU mask, GELU input), epi_store applies activation, mask and
// GELU' and stores, so that a thread can issue the loads of several rows
// before it needs any of them.
// The epilogue's per-element operands, loaded in batches before the first
// use; bf16 operands stay raw bits until used, so that converting them does
// not make each load of a batch wait for the previous one.
struct EpiIn {
    float resid = 0.f, theta = 0.f;
    bf16_t mask = 0x3F80, dact = 0x3F80;  // 1.0
};

__device__ __forceinline__ EpiIn epi_load(const GemmDesc& d, int row, int col) {
    EpiIn e;
    if (d.resid) e.resid = d.resid[(int64_t)row * d.ldr + col];
    if (d.mask) e.mask = d.mask[(int64_t)row * d.ldm + col];
    if (d.dact) e.dact = d.dact[(int64_t)row * d.ldm + col];
    if (d.sgd_theta) e.theta = d.sgd_theta[(int64_t)row * d.ldcf + col];
    return e;
}

// v already holds bias and residual
__device__ __forceinline__ float epi_store(const GemmDesc& d, int row, int col, float v, const EpiIn& e) {
    if (d.act == ACT_GELU) {
        if (d.dact_out) {
            float g;
            v = gelu_and_grad(v, &g);
            d.dact_out[(int64_t)row * d.ldm + col] = f2bf(g);
        } else {
            v = gelu_f(v);
        }
    } else if (d.act == ACT_RELU) {
        v = v > 0.f ? v : 0.f;
    }
    if (d.mask && !(bf2f(e.mask) > 0.f)) v = 0.f;
    if (d.dact) v *= bf2f(e.dact);
    if (d.Cf) d.Cf[(int64_t)row * d.ldcf + col] = v;
    if (d.sgd_theta) {
        const int64_t o = (int64_t)row * d.ldcf + col;
        const float th = __builtin_fmaf(-d.sgd_lr, v, e.theta);
        d.sgd_theta[o] = th;
        const bf16_t h = f2bf(th);
        d.sgd_hi[o] = h;
        d.sgd_lo[o] = f2bf(th - bf2f(h));
    }
    if (d.Cb) {
        const bf16_t hi = f2bf(v);
        d.Cb[(int64_t)row * d.ldcb + col] = hi;
        if (d.Cb2) d.Cb2[(int64_t)row * d.ldcb + col] = f2bf(v - bf2f(hi));
    }
    return v;
}

__device__ __forceinline__ float epilogue(const GemmDesc& d, int row, int col, float v) {
    const EpiIn e = epi_load(d, row, col);
    if (d.bias) v += d.bias[col];
    return epi_store(d, row, col, v + e.resid, e);
}

// The same epilogue on four consecutive columns (col % 4 == 0) with 16-byte
// (fp32) and 8-byte (bf16) accesses, one address computation per operand; used
// when the launcher found every operand aligned for it (vec_epi).
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4 bf4_to_f(u32x2 w) {
    f32x4 f;
    f.x = bf2f((bf16_t)(w.x & 0xFFFFu));
    f.y = bf2f((bf16_t)(w.x >> 16));
    f.z = bf2f((bf16_t)(w.y & 0xFFFFu));
    f.w = bf2f((bf16_t)(w.y >> 16));
    return f;
}
__device__ __forceinline__ u32x2 f_to_bf4(f32x4 v, f32x4* lo) {
    u32x2 w;
    w.x = f2bf2(v.x, v.y);
    w.y = f2bf2(v.z, v.w);
    if (lo) {
        lo->x = v.x - bf2f((bf16_t)(w.x & 0xFFFFu));
        lo->y = v.y - bf2f((bf16_t)(w.x >> 16));
        lo->z = v.z - bf2f((bf16_t)(w.y & 0xFFFFu));
        lo->w = v.w - bf2f((bf16_t)(w.y >> 16));
    }
    return w;
}

struct EpiIn4 {  // as EpiIn, four columns (bf16 operands as raw bits)
    f32x4 resid = {0.f, 0.f, 0.f, 0.f}, theta = {0.f, 0.f, 0.f, 0.f};
    u32x2 mask = {0x3F803F80u, 0x3F803F80u}, dact = {0x3F803F80u, 0x3F803F80u};  // 1.0 x 4
};

__device__ __forceinline__ EpiIn4 epi_load4(const GemmDesc& d, int row, int col) {
    EpiIn4 e;
    if (d.resid) e.resid = *reinterpret_cast<const f32x4*>(d.resid + (int64_t)row * d.ldr + col);
    if (d.mask) e.mask = *reinterpret_cast<const u32x2*>(d.mask + (int64_t)row * d.ldm + col);
    if (d.dact) e.dact = *reinterpret_cast<const u32x2*>(d.dact + (int64_t)row * d.ldm + col);
    if (d.sgd_theta) e.theta = *reinterpret_cast<const f32x4*>(d.sgd_theta + (int64_t)row * d.ldcf + col);
    return e;
}

// The operands of NB rows (clamped into the product by the caller, so every
// load is in bounds): each operand's loads sit in one uniform branch, all of
// them issued before the first use.
template <int NB>
__device__ __forceinline__ void epi_load4_batch(const GemmDesc& d, const int (&row)[NB], int col, EpiIn4 (&e)[NB]) {
    if (d.resid) {
#pragma unroll
        for (int u = 0; u < NB; ++u) e[u].resid = *reinterpret_cast<const f32x4*>(d.resid + (int64_t)row[u] * d.ldr + col);
    }
    if (d.mask) {
#pragma unroll
        for (int u = 0; u < NB; ++u) e[u].mask = *reinterpret_cast<const u32x2*>(d.mask + (int64_t)row[u] * d.ldm + col);
    }
    if (d.dact) {
#pragma unroll
        for (int u = 0; u < NB; ++u) e[u].dact = *reinterpret_cast<const u32x2*>(d.dact + (int64_t)row[u] * d.ldm + col);
    }
    if (d.sgd_theta) {
#pragma unroll
        for (int u = 0; u < NB; ++u)
            e[u].theta = *reinterpret_cast<const f32x4*>(d.sgd_theta + (int64_t)row[u] * d.ldcf + col);
    }
}
template <int NB>
__device__ __forceinline__ void epi_load_batch(const GemmDesc& d, const int (&row)[NB], int col, EpiIn (&e)[NB]) {
    if (d.resid) {
#pragma unroll
        for (int u = 0; u < NB; ++u) e[u].resid = d.resid[(int64_t)row[u] * d.ldr + col];
    }
    if (d.mask) {
#pragma unroll
        for (int u = 0; u < NB; ++u) e[u].mask = d.mask[(int64_t)row[u] * d.ldm + col];
    }
    if (d.dact) {
#pragma unroll
        for (int u = 0; u < NB; ++u) e[u].dact = d.dact[(int64_t)row[u] * d.ldm + col];
    }
    if (d.sgd_theta) {
#pragma unroll
        for (int u = 0; u < NB; ++u) e[u].theta = d.sgd_theta[(int64_t)row[u] * d.ldcf + col];
    }
}

// v already holds bias and residual
__device__ __forceinline__ f32x4 epi_store4(const GemmDesc& d, int row, int col, f32x4 v, const EpiIn4& e) {
    if (d.act == ACT_GELU) {
        if (d.dact_out) {
            f32x4 g;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float gq;
                v[q] = gelu_and_grad(v[q], &gq);
                g[q] = gq;
            }
            *reinterpret_cast<u32x2*>(d.dact_out + (int64_t)row * d.ldm + col) = f_to_bf4(g, nullptr);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = gelu_f(v[q]);
        }
    } else if (d.act == ACT_RELU) {
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = v[q] > 0.f ? v[q] : 0.f;
    }
    if (d.mask) {
        const f32x4 mk = bf4_to_f(e.mask);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (!(mk[q] > 0.f)) v[q] = 0.f;
    }
    if (d.dact) v *= bf4_to_f(e.dact);
    if (d.Cf) *reinterpret_cast<f32x4*>(d.Cf + (int64_t)row * d.ldcf + col) = v;
    if (d.sgd_theta) {
        const int64_t o = (int64_t)row * d.ldcf + col;
        f32x4 th = e.theta, lo;
#pragma unroll
        for (int q = 0; q < 4; ++q) th[q] = __builtin_fmaf(-d.sgd_lr, v[q], th[q]);
        *reinterpret_cast<f32x4*>(d.sgd_theta + o) = th;
        *reinterpret_cast<u32x2*>(d.sgd_hi + o) = f_to_bf4(th, &lo);
        *reinterpret_cast<u32x2*>(d.sgd_lo + o) = f_to_bf4(lo, nullptr);
    }
    if (d.Cb) {
        f32x4 lo;
        const int64_t o = (int64_t)row * d.ldcb + col;
        *reinterpret_cast<u32x2*>(d.Cb + o) = f_to_bf4(v, d.Cb2 ? &lo : nullptr);
        if (d.Cb2) *reinterpret_cast<u32x2*>(d.Cb2 + o) = f_to_bf4(lo, nullptr);
    }
    return v;
}

// ------------------------------------------------------------------ kernel
// The K range over the concatenation of nseg segments (segment s pairs (A, B),
// (A, B2), (A2, B) for s = 0, 1, 2), each padded to a whole number of K tiles
// when nseg > 1 (the loaders zero-fill past K).
__device__ __forceinline__ int gemm_kseg(const GemmDesc& d, int Keff) {
    return d.nseg > 1 ? (d.K + BK - 1) / BK * BK : Keff;
}

// Split-K slices in use.  With a device-side row bound the launch's slice count
// is a maximum: the kernel and the reduction both take as many slices as keep
// two workgroups per CU busy over the active tiles, each at least four K tiles
// long.  With static sizes every launched slice is used.
__device__ __forceinline__ int active_splits(const GemmDesc& d, int M_eff, int ktot) {
    return d.Mdev ? gemm_active_splits(d.splits, M_eff, d.N, ktot) : d.splits;
}

// The output tile and K slice of a workgroup.
struct TileJob {
    int m0, n0, mt, zt, S;
};

// XCD-aware tile order.  Workgroups are handed to the eight XCDs round robin
// by linear id, and each XCD has its own L2: the first W ids (the tiles below
// the effective M, times the slices in use; the rest exit) are renumbered so
// that XCD x owns a contiguous range, walked in groups of GM tile rows (M
// fastest), which keeps the A row blocks and B column blocks it reads few and
// shared.  Returns false when the workgroup has no tile.
template <int BMt = BM, int BNt = BN>
__device__ __forceinline__ bool map_tile(const GemmDesc& d, int M, int ktot_split, TileJob& job) {
    constexpr int GM = 8;
    const int S = active_splits(d, M, ktot_split);
    const int nN = gridDim.x, nMe = (M + BMt - 1) / BMt;
    const int W = nMe * nN * S;
    const int w = blockIdx.x + nN * (blockIdx.y + gridDim.y * blockIdx.z);
    if (w >= W) return false;
    const int xq = W >> 3, xr = W & 7, xc = w & 7;
    const int nid = xc * xq + min(xc, xr) + (w >> 3);
    const int T1 = nMe * nN;
    const int zt = nid / T1, tt = nid - zt * T1;
    const int g = tt / (GM * nN), tg = tt - g * GM * nN;
    const int gr = min(GM, nMe - g * GM);
    job.mt = g * GM + tg % gr;
    job.m0 = job.mt * BMt;
    job.n0 = (tg / gr) * BNt;
    job.zt = zt;
    job.S = S;
    return true;
}

// The 128 x 128 accumulator tile leaves through LDS (Cs, 64 KB): accumulator
// (i, j, r) of a lane holds C[row][col] with row = i*32 + (r/4)*8 +
// (lane/32)*4 + r%4, col = j*32 + lane%32 (wave-relative).  Each thread then
// owns one column and walks 64 rows, so every global store instruction covers
// 64 consecutive columns of one row.  Split slices store fp32 partials; a
// whole product runs the epilogue (and the optional column sums).
// BMt rows by NTt threads (4 waves of 64 x 64 per 128 rows); RP = NTt / 32 rows per
// pass of the four-column path, HP = NTt / 128 row groups of the one-column path.
// drain_tile is the second half: from the tile staged in LDS (Cs[row][BNt]) to
// memory, for rows job.m0 .. job.m0 + BMt - 1, the epilogue's operands of NB
// rows loaded together.
template <int BMt = BM, int NTt = NT, int BNt = BN, int NB = 8>
__device__ __forceinline__ void drain_tile(const GemmDesc& d, float* Cs, const TileJob& job, int M, int tid) {
    // TPR threads per row in the four-column path, RP rows per pass; HP row
    // groups in the one-column path
    constexpr int TPR = BNt / 4, RP = NTt / TPR, HP = NTt / BNt;
    static_assert(HP >= 1, "tile shape");
    if (d.vec_epi) {
        // four columns per thread: rows tid / TPR + RP u, columns n0 + 4 (tid % TPR) .. + 3
        const int m0 = job.m0, c4 = (tid % TPR) * 4, col = job.n0 + c4, rr = tid / TPR;
        f32x4 csum = {0.f, 0.f, 0.f, 0.f};
        if (col < d.N) {
            if (job.S > 1) {
                for (int lr = rr; lr < BMt && m0 + lr < M; lr += RP)
                    *reinterpret_cast<f32x4*>(d.ws + ((int64_t)job.zt * d.M + m0 + lr) * d.N + col) =
                        *reinterpret_cast<const f32x4*>(&Cs[lr * BNt + c4]);
            } else {
                f32x4 bias = {0.f, 0.f, 0.f, 0.f};
                if (d.bias) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) bias[q] = d.bias[col + q];
                }
                for (int lr0 = rr; lr0 < BMt && m0 + lr0 < M; lr0 += NB * RP) {
                    EpiIn4 e[NB];
                    int rows[NB];
#pragma unroll
                    for (int u = 0; u < NB; ++u) rows[u] = min(m0 + lr0 + RP * u, M - 1);
                    epi_load4_batch(d, rows, col, e);
#pragma unroll
                    for (int u = 0; u < NB; ++u) {
                        const int lr = lr0 + RP * u, row = m0 + lr;
                        if (row < M)
                            csum += epi_store4(d, row, col,
                                               *reinterpret_cast<const f32x4*>(&Cs[lr * BNt + c4]) + bias + e[u].resid,
                                               e[u]);
                    }
                }
            }
        }
        if (d.colpart) {  // uniform; the RP row groups of a column meet in LDS
            __syncthreads();
            *reinterpret_cast<f32x4*>(&Cs[rr * BNt + c4]) = csum;
            __syncthreads();
            if (tid < BNt && job.n0 + tid < d.N) {
                float t = 0.f;
#pragma unroll
                for (int g = 0; g < RP; ++g) t += Cs[g * BNt + tid];
                d.colpart[(int64_t)job.mt * d.N + job.n0 + tid] = t;
            }
        }
        return;
    }
    const int m0 = job.m0, c = tid % BNt, col = job.n0 + c;
    float csum = 0.f;
    if (col < d.N) {
        if (job.S > 1) {
            for (int lr = tid / BNt; lr < BMt; lr += HP) {
                const int row = m0 + lr;
                if (row >= M) break;
                d.ws[((int64_t)job.zt * d.M + row) * d.N + col] = Cs[lr * BNt + c];
            }
        } else {
            const float bcol = d.bias ? d.bias[col] : 0.f;
            // NB rows per batch: their operand loads are in flight together
            for (int lr0 = tid / BNt; lr0 < BMt && m0 + lr0 < M; lr0 += NB * HP) {
                EpiIn e[NB];
                int rows[NB];
#pragma unroll
                for (int u = 0; u < NB; ++u) rows[u] = min(m0 + lr0 + HP * u, M - 1);
                epi_load_batch(d, rows, col, e);
#pragma unroll
                for (int u = 0; u < NB; ++u) {
                    const int lr = lr0 + HP * u, row = m0 + lr;
                    if (row < M) csum += epi_store(d, row, col, Cs[lr * BNt + c] + bcol + e[u].resid, e[u]);
                }
            }
        }
    }
    if (d.colpart) {  // uniform; the HP row groups of a column meet in LDS
        __syncthreads();
        if (tid >= BNt) Cs[(tid / BNt) * BNt + c] = csum;
        __syncthreads();
        if (tid < BNt && col < d.N) {
            float t = csum;
#pragma unroll
            for (int g = 1; g < HP; ++g) t += Cs[g * BNt + c];
            d.colpart[(int64_t)job.mt * d.N + col] = t;
        }
    }
}

template <int BMt = BM, int NTt = NT, int BNt = BN, int WNF = 2>
__device__ __forceinline__ void store_tile(const GemmDesc& d, const f32x16 (&acc)[2][WNF], float* Cs,
                                           const TileJob& job, int M, int tid) {
    static_assert(BNt == 32 * 2 * WNF, "tile shape");
    const int lane = tid & 63, wave = tid >> 6, wm = wave >> 1, wn = wave & 1;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < WNF; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int lr = wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                Cs[lr * BNt + wn * 32 * WNF + j * 32 + (lane & 31)] = acc[i][j][r];
            }
    __syncthreads();
    drain_tile<BMt, NTt, BNt>(d, Cs, job, M, tid);
}

// Two K tiles (A and B each 128 x 72 bf16) = 72 KB of LDS; reused for the C tile.
typedef bf16_t GemmSmem[2][2][BM * LDR];

// One 128 x 128 output tile (one K slice of it) of the product d: the K loop
// and the epilogue, shared by the single-product and the grouped kernels.
template <int AM, int BMODE, bool AL>
__device__ __forceinline__ void gemm_tile(const GemmDesc& d, const TileJob& job, int M, int Keff, GemmSmem& smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int kseg = gemm_kseg(d, Keff);
    const int ktot = d.nseg * kseg;
    const int S = job.S, zt = job.zt, m0 = job.m0, n0 = job.n0;
    // this slice's K range (slices are whole K tiles long)
    const int kc = ((ktot + S - 1) / S + BK - 1) / BK * BK;
    const int kbeg = zt * kc;
    const int kstop = min(ktot, kbeg + kc);
    const int nk = kstop > kbeg ? (kstop - kbeg + BK - 1) / BK : 0;

    typename LoaderOf<AM>::T la;
    typename LoaderOf<BMODE>::T lb;
    loader_init<AM>(la, d.A, d.lda, d.g, m0, M, tid);
    loader_init<BMODE>(lb, d.B, d.ldb, d.g, n0, d.N, tid);

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // tile t's loads land in register set t % 2; they are issued two compute
    // phases before the registers are stored to LDS
    uint4 ra0[NV], rb0[NV], ra1[NV], rb1[NV];
    // the (segment, offset) of the next tile to load, advanced without division;
    // segments are whole tiles long, so a tile never straddles two
    int ld_seg = kseg > 0 ? kbeg / kseg : 0, ld_kk = kbeg - ld_seg * kseg;
    int ld_t = 0;  // index (within this slice) of the next tile to load
    auto load_tile = [&](uint4* ra, uint4* rb) {
        if constexpr (AL) {
            // a prefetch past the slice's last tile reads zeros only: its
            // (segment, offset) may name a low part that does not exist
            const int ke = ld_t < nk ? Keff : 0;
            la.load_al(ld_seg == 2 ? d.A2 : d.A, ld_kk, ke, ra);
            lb.load_al(ld_seg == 1 ? d.B2 : d.B, ld_kk, ke, rb);
        } else {
            la.load(ld_seg == 2 ? d.A2 : d.A, ld_kk, Keff, ra);
            lb.load(ld_seg == 1 ? d.B2 : d.B, ld_kk, Keff, rb);
        }
        ++ld_t;
        ld_kk += BK;
        if (ld_kk >= kseg) {
            ld_kk -= kseg;
            ++ld_seg;
        }
    };
    const int lrow = lane & 31, lk = (lane >> 5) * 8;
    const int aoff = lds_idx(wm * 64 + lrow, lk), boff = lds_idx(wn * 64 + lrow, lk);
    const int2 atr0 = frag_tr_off(lane, wm * 64), atr1 = frag_tr_off(lane, wm * 64 + 32);
    const int2 btr0 = frag_tr_off(lane, wn * 64), btr1 = frag_tr_off(lane, wn * 64 + 32);
    auto compute = [&](const bf16_t* As, const bf16_t* Bs) {
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            bf16x8_t a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                a[i] = (AM == OP_KRT || AM == OP_CONV_DXWT || AM == OP_CONV_DWXT) ? frag_tr(As, i ? atr1 : atr0, ks * 16 * BM)
                                    : *reinterpret_cast<const bf16x8_t*>(&As[aoff + i * 32 * LDR + ks * 16]);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                b[j] = (BMODE == OP_KRT || BMODE == OP_CONV_DXWT || BMODE == OP_CONV_DWXT) ? frag_tr(Bs, j ? btr1 : btr0, ks * 16 * BM)
                                       : *reinterpret_cast<const bf16x8_t*>(&Bs[boff + j * 32 * LDR + ks * 16]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    };

    // The aligned variant issues every prefetch, also past the last tile (those
    // read zeros or operand memory and are never stored): with a static number
    // of loads in flight, each wait covers exactly the register set it needs.
    if (AL || nk > 0) load_tile(ra0, rb0);
    if (AL || nk > 1) load_tile(ra1, rb1);
    if (nk > 0) {
        la.store(smem[0][0], ra0, tid);
        lb.store(smem[0][1], rb0, tid);
    }
    __syncthreads();
    // two K tiles per trip and no exit inside the body (an exit between the
    // halves makes the compiler keep the accumulators in two register sets)
    int t = 0;
    for (; t + 1 < nk; t += 2) {
        // even half: compute tile t from buffer 0, stage tile t+1 (set 1) into buffer 1
        if (AL || t + 2 < nk) load_tile(ra0, rb0);
        compute(smem[0][0], smem[0][1]);
        la.store(smem[1][0], ra1, tid);
        lb.store(smem[1][1], rb1, tid);
        __syncthreads();
        // odd half: compute tile t+1 from buffer 1, stage tile t+2 (set 0) into buffer 0
        if (AL || t + 3 < nk) load_tile(ra1, rb1);
        compute(smem[1][0], smem[1][1]);
        if (t + 2 < nk) {
            la.store(smem[0][0], ra0, tid);
            lb.store(smem[0][1], rb0, tid);
        }
        __syncthreads();
    }
    if (t < nk) {  // odd tile count: the last tile is in buffer 0
        compute(smem[0][0], smem[0][1]);
        __syncthreads();
    }

    store_tile(d, acc, reinterpret_cast<float*>(&smem[0][0][0]), job, M, tid);
}

template <int AM, int BMODE, bool AL>
__global__ void __launch_bounds__(NT, 2) gemm_kernel(const GemmDesc d) {
    __shared__ __attribute__((aligned(16))) GemmSmem smem;
    const int M = d.Mdev ? min(d.M, *d.Mdev) : d.M;
    const int Keff = d.Kdev ? min(d.K, *d.Kdev) : d.K;
    if (d.prof_snap && (blockIdx.x | blockIdx.y | blockIdx.z) == 0 && threadIdx.x == 0) {
        d.prof_snap[0] = M;
        d.prof_snap[1] = Keff;
    }
    TileJob job;
    if (!map_tile(d, M, d.nseg * gemm_kseg(d, Keff), job)) return;  // uniform for the whole workgroup
    gemm_tile<AM, BMODE, AL>(d, job, M, Keff, smem);
}

// Several independent products in one launch (each unsplit, over its whole K):
// the grid is the concatenation of their 128 x 128 output tiles.  Workgroup
// ids are renumbered as in map_tile so that each XCD owns a contiguous range
// of the concatenated tiles, and within a product the tiles are walked in
// groups of eight tile rows.  Used for the four weight gradients of an
// encoder layer, which are ready at the same point of the backward.
struct GemmGroupArg {
    GemmDesc d[kGemmGroupMax];
    int n;
    int* prof_snap;  // (M, K) effective per member, when profiling
};

// Calls f(d, job, M, K) for each BMt x 128 tile of a group that this
// workgroup owns.
template <int BMt = BM, class F>
__device__ __forceinline__ void for_group_tiles(const GemmGroupArg& g, F&& f) {
    constexpr int GM = 8;
    int Ms[kGemmGroupMax], Ks[kGemmGroupMax], start[kGemmGroupMax + 1];
    start[0] = 0;
#pragma unroll
    for (int i = 0; i < kGemmGroupMax; ++i) {
        const GemmDesc& d = g.d[i < g.n ? i : 0];
        Ms[i] = d.Mdev ? min(d.M, *d.Mdev) : d.M;
        Ks[i] = d.Kdev ? min(d.K, *d.Kdev) : d.K;
        const int tiles = ((Ms[i] + BMt - 1) / BMt) * ((d.N + BN - 1) / BN);
        start[i + 1] = start[i] + (i < g.n ? tiles : 0);
    }
    if (g.prof_snap && blockIdx.x == 0 && threadIdx.x == 0) {
#pragma unroll
        for (int i = 0; i < kGemmGroupMax; ++i)
            if (i < g.n) {
                g.prof_snap[2 * i] = Ms[i];
                g.prof_snap[2 * i + 1] = Ks[i];
            }
    }
    const int W = start[kGemmGroupMax];
    // A grid smaller than the tile count (a multiple of 8, so that a workgroup
    // stays on its XCD's share) walks the tiles in rounds.
    for (int w = blockIdx.x; w < W; w += gridDim.x) {
        const int xq = W >> 3, xr = W & 7, xc = w & 7;
        const int nid = xc * xq + min(xc, xr) + (w >> 3);
        // the member owning tile nid (selects in registers: no dynamic indexing)
        int m = 0, s0 = 0, Mm = Ms[0], Km = Ks[0];
#pragma unroll
        for (int i = 1; i < kGemmGroupMax; ++i)
            if (nid >= start[i]) {
                m = i;
                s0 = start[i];
                Mm = Ms[i];
                Km = Ks[i];
            }
        const GemmDesc& d = g.d[m];
        const int tt = nid - s0;
        const int nN = (d.N + BN - 1) / BN, nMe = (Mm + BMt - 1) / BMt;
        const int grp = tt / (GM * nN), tg = tt - grp * GM * nN;
        const int gr = min(GM, nMe - grp * GM);
        TileJob job;
        job.mt = grp * GM + tg % gr;
        job.m0 = job.mt * BMt;
        job.n0 = (tg / gr) * BN;
        job.zt = 0;
        job.S = 1;
        f(d, job, Mm, Km);
        __syncthreads();  // the next tile's stores reuse the LDS of this one's C tile
    }
}

// ------------------------------------------------------------------ single-pass compensated product
// C = A.B + A.B_lo + A_lo.B (NSEG = 3) or A.B + A.B_lo (NSEG = 2) for aligned
// row-major operands (K contiguous, K, lda, ldb multiples of 8): every K tile
// stages the high and low parts of both operands once and issues the two or
// three MFMAs of each fragment pair back to back, instead of running the K loop
// once per segment.  Per MFMA that is two thirds of the LDS reads and a third
// of the barriers of the segmented form.
constexpr int CBK = 32;

// The operand tiles go straight from global memory into LDS
// (global_load_lds_dwordx4: lane L of a wave writes 16 bytes at the
// instruction's LDS base + 16 L), so there are no LDS store instructions and no
// staging registers.  A 128 x 32 tile is 128 rows of 64 bytes, the 16-byte chunk c of
// row r at position c ^ ((r / 4) mod 4): one instruction fills 16 rows, and
// the operand reads of any eight consecutive rows hit distinct banks.  Two
// stages in separate arrays (the halves of the unrolled loop name them
// statically); the copy of tile t+1 is issued before the MFMAs of tile t.
#define FO_LDS(p) ((__attribute__((address_space(3))) void*)(p))

struct DmaRKc {  // one 128 x 32 tile; this wave's instructions are q = wave and wave + 4
    int64_t off[2];
    int koff;
    __device__ void init(const GemmDesc& d, bool is_a, int r0, int R, int lane, int wave) {
        init(is_a ? d.lda : d.ldb, r0, R, lane, wave);
    }
    __device__ void init(int64_t ld, int r0, int R, int lane, int wave) {
        koff = 8 * ((lane & 3) ^ ((lane >> 4) & 3));
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const int gr = r0 + 16 * (wave + 4 * v) + (lane >> 2);
            off[v] = gr < R ? (int64_t)gr * ld : -1;
        }
    }
    __device__ void copy(const bf16_t* P, int kb, int kend, bf16_t* tile, int wave) const {
        const int k = kb + koff;
#pragma unroll
        for (int v = 0; v < 2; ++v)
            __builtin_amdgcn_global_load_lds(off[v] >= 0 && k < kend ? P + off[v] + k : kZero8,
                                             FO_LDS(tile + (wave + 4 * v) * 512), 16, 0, 0);
    }
};

// The A operand of a convolution forward (implicit GEMM: rows = output pixels
// (b, oy, ox), k = (ky, kx, ci) over the NHWC input, Ci % 64 == 0 so that a
// 32-wide K tile lies in one filter tap), in the same 128 x 32 LDS tile layout
// as DmaRKc: each lane copies the 16 bytes of channels it owns from the input
// pixel its row reads at the tile's tap, or the zero block in the padding.
struct DmaConvA {
    ConvGeom g;
    int b[2], iy0[2], ix0[2];
    bool ok[2];
    int koff;
    __device__ void init(const GemmDesc& d, bool, int r0, int R, int lane, int wave) {
        g = d.g;
        koff = 8 * ((lane & 3) ^ ((lane >> 4) & 3));
        const int hw = g.Ho * g.Wo;
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const int gr = r0 + 16 * (wave + 4 * v) + (lane >> 2);
            ok[v] = gr < R;
            b[v] = gr / hw;
            const int rem = gr - b[v] * hw, oy = rem / g.Wo, ox = rem - oy * g.Wo;
            iy0[v] = oy * g.stride - g.pad;
            ix0[v] = ox * g.stride - g.pad;
        }
    }
    __device__ void copy(const bf16_t* X, int kb, int kend, bf16_t* tile, int wave) const {
        const int tap = kb / g.Ci, ci = kb - tap * g.Ci + koff;
        const int ky = tap / g.kw, kx = tap - ky * g.kw;
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const int iy = iy0[v] + ky, ix = ix0[v] + kx;
            const bool in = ok[v] && kb < kend && iy >= 0 && iy < g.H && ix >= 0 && ix < g.W;
            __builtin_amdgcn_global_load_lds(in ? X + (((int64_t)b[v] * g.H + iy) * g.W + ix) * g.Ci + ci : kZero8,
                                             FO_LDS(tile + (wave + 4 * v) * 512), 16, 0, 0);
        }
    }
};

// s_waitcnt immediate that waits for at most n vector memory operations in
// flight and does not wait on LDS / scalar memory or exports.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
// The same, and no LDS operation in flight (lgkmcnt(0)): the wait that closes a
// ring step, after which no wave may still be reading the stage the next copy
// overwrites.
constexpr int vmcnt_lds0_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

// Workgroup barrier without the release / acquire fences of __syncthreads:
// with copies into LDS in flight the compiler turns those fences into a wait
// for every outstanding copy (vmcnt(0)) before the barrier, which collapses a
// ring of stages to a single one.  The callers wait explicitly for the copies
// the next step reads; the wavefront-scope fences only keep the compiler from
// moving memory operations across the barrier.
__device__ __forceinline__ void ring_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// NST stages in a ring: the copy of tile t + NST - 1 is issued before the MFMAs
// of tile t.  Every copy is issued, also past the slice's last tile (those read
// kZero8 into a stage that is not read again), so the number of copies in
// flight is static and each wait names exactly the tile it needs.
template <int NSEG, int NST, class LA>
__global__ void __launch_bounds__(NT, NST == 2 ? 2 : 1) gemm_comp_dma_kernel(const GemmDesc d) {
    // NST stages of four unpadded 128 x 32 tiles (A, A_lo, B, B_lo) = 32 KB each;
    // reused for the C tile (64 KB)
    __shared__ __attribute__((aligned(1024))) bf16_t smem[NST][4][BM * CBK];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int M = d.Mdev ? min(d.M, *d.Mdev) : d.M;
    const int K = d.K;
    if (d.prof_snap && (blockIdx.x | blockIdx.y | blockIdx.z) == 0 && tid == 0) {
        d.prof_snap[0] = M;
        d.prof_snap[1] = K;
    }
    TileJob job;
    if (!map_tile(d, M, d.nseg * gemm_kseg(d, K), job)) return;  // uniform for the whole workgroup
    const int S = job.S;
    const int kpad = (K + CBK - 1) / CBK * CBK;
    const int kc = ((kpad + S - 1) / S + CBK - 1) / CBK * CBK;
    const int kbeg = job.zt * kc;
    const int kstop = min(kpad, kbeg + kc);
    const int nk = kstop > kbeg ? (kstop - kbeg) / CBK : 0;

    LA la;
    DmaRKc lb;
    la.init(d, true, job.m0, M, lane, wave);
    lb.init(d, false, job.n0, d.N, lane, wave);

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    constexpr int CPT = NSEG == 3 ? 8 : 6;  // copy instructions per tile and thread
    auto copy_tile = [&](bf16_t (*st)[BM * CBK], int t) {
        const int kb = kbeg + t * CBK, ke = t < nk ? K : 0;
        la.copy(d.A, kb, ke, st[0], wave);
        if (NSEG == 3) la.copy(d.A2, kb, ke, st[1], wave);
        lb.copy(d.B, kb, ke, st[2], wave);
        lb.copy(d.B2, kb, ke, st[3], wave);
    };
    const int lrow = lane & 31, lc = lane >> 5;
    auto frag = [&](const bf16_t* t, int row, int ks) {
        const int C = 2 * ks + lc;
        return *reinterpret_cast<const bf16x8_t*>(&t[row * CBK + 8 * (C ^ ((row >> 2) & 3))]);
    };
    auto compute = [&](bf16_t (*st)[BM * CBK]) {
#pragma unroll
        for (int ks = 0; ks < CBK / 16; ++ks) {
            bf16x8_t a[2], al[2], b[2], bl[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int row = wm * 64 + i * 32 + lrow;
                a[i] = frag(st[0], row, ks);
                if (NSEG == 3) al[i] = frag(st[1], row, ks);
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int row = wn * 64 + j * 32 + lrow;
                b[j] = frag(st[2], row, ks);
                bl[j] = frag(st[3], row, ks);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], bl[j], acc[i][j], 0, 0, 0);
                    if (NSEG == 3)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[i], b[j], acc[i][j], 0, 0, 0);
                }
        }
    };
    // one step: issue the copy NST - 1 tiles ahead, compute tile t, wait until
    // tile t + 1 has landed in every wave
    auto step = [&](int t, int u) {
        copy_tile(smem[(u + NST - 1) % NST], t + NST - 1);
        compute(smem[u]);
        __builtin_amdgcn_s_waitcnt(vmcnt_lds0_imm(CPT * (NST - 2)));
        ring_barrier();
    };

#pragma unroll
    for (int u = 0; u < NST - 1; ++u) copy_tile(smem[u], u);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(CPT * (NST - 2)));  // tile 0 has landed
    ring_barrier();
    int t = 0;
    for (; t + NST <= nk; t += NST) {  // whole rounds: static stage indices
#pragma unroll
        for (int u = 0; u < NST; ++u) step(t + u, u);
    }
    for (int u = 0; t < nk; ++t, ++u) step(t, u);  // the rest of a round (stage index u < NST)
    __builtin_amdgcn_s_waitcnt(0);  // copies past the last tile
    __syncthreads();
    store_tile(d, acc, reinterpret_cast<float*>(&smem[0][0][0]), job, M, tid);
}

// ------------------------------------------------------------------ weight gradients, copies into LDS
// The transpose reads of this kernel are written as inline assembly: with the
// intrinsic, the compiler waits for every copy into LDS still in flight
// (vmcnt(0)) before each read, which would leave one stage of the ring in use.
// The compiler does not track these reads, so their results are used only
// after lgkm_wait_tr, whose operands tie the registers to the wait.
typedef int i32x2_t __attribute__((ext_vector_type(2)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint32_t lds_addr(const bf16_t* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16_t*)p;
}
__device__ __forceinline__ i32x2_t tr_read(uint32_t addr) {
    i32x2_t v;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
    return v;
}
// waits until at most 8 n (n = 0, 1) LDS operations are in flight (the reads
// of the next k block; LDS operations complete in order) and hands r on
__device__ __forceinline__ void lgkm_wait_tr(i32x2_t (&r)[8], int n) {
    if (n)
        asm volatile("s_waitcnt lgkmcnt(8)"
                     : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7]));
    else
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7]));
}
__device__ __forceinline__ bf16x8_t frag_cat(i32x2_t a, i32x2_t b) {
    const i32x4_t v = {a.x, a.y, b.x, b.y};
    return __builtin_bit_cast(bf16x8_t, v);
}

// Both operands k-major (A = [K][M], B = [K][N], the rows of a tile contiguous
// in memory), as in the products of weight gradients.  The tiles (KT k rows of
// RT operand rows) keep the [k][row] layout of the transposed loaders (kr_idx)
// that the transpose reads take their fragments from, but are filled by
// global_load_lds: a k row is RT / 8 16-byte chunks, so instruction i of the
// workgroup writes KPI = 64 / (RT / 8) k rows from KPI i on, lane L its 16-byte
// slot L of them, which under the swizzle is k row k = KPI i + L / (RT / 8) and
// the eight rows 8 ((L mod RT / 8) xor 4 (k mod 4)) .. + 7.  No staging
// registers and no LDS store instructions; the waits name exactly the tile
// the next step reads.
template <int KT, int RT = BM>
struct DmaKRt {
    static constexpr int CPR = RT / 8;     // 16-byte chunks per k row
    static constexpr int KPI = 64 / CPR;   // k rows per copy instruction
    static constexpr int NI = KT / KPI / 4;  // instructions per wave and operand tile
    static_assert((RT == 128 || RT == 256) && KT % (4 * KPI) == 0 && KT <= 64, "tile shape");
    // Instruction v of a wave covers k row kk0 + 4 KPI v; k mod 4, hence the
    // lane's rows, is the same for every v (4 KPI is a multiple of 4).
    int64_t off0;  // element offset of the lane's chunk at k = kk0 (-1 outside the rows)
    int64_t ld;
    int kk0;
    __device__ void init(int64_t ld_, int r0, int R, int lane, int wave) {
        ld = ld_;
        const int sub = lane / CPR, slot = lane % CPR;
        kk0 = KPI * wave + sub;
        const int r = r0 + 8 * (slot ^ (4 * (kk0 & 3)));
        off0 = r < R ? (int64_t)kk0 * ld + r : -1;
    }
    __device__ void copy(const bf16_t* P, int kb, int kend, bf16_t* tile, int wave) const {
        const bf16_t* p = P + off0 + (int64_t)kb * ld;
#pragma unroll
        for (int v = 0; v < NI; ++v)
            __builtin_amdgcn_global_load_lds(off0 >= 0 && kb + kk0 + 4 * KPI * v < kend ? p + (int64_t)4 * KPI * v * ld
                                                                                          : kZero8,
                                             FO_LDS(tile + (wave + 4 * v) * 512), 16, 0, 0);
    }
};

// One 128 x 128 tile of a weight-gradient product over its whole K, NST stages
// of KT-deep tiles in a ring (the copy of tile t + NST - 1 issued before the
// MFMAs of tile t; every copy issued, past the last tile too, so that the
// number in flight is static).  The stages (NST x 2 x KT x 128 bf16) hold the
// fp32 C tile afterwards.
template <int KT, int NST>
__device__ __forceinline__ void wgrad_tile(const GemmDesc& d, const TileJob& job, int M, int K,
                                           bf16_t (*smem)[2][KT * BM]) {
    static_assert(NST * 2 * KT * BM * 2 >= BM * BN * 4, "the C tile lives in the stages");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int nk = (K + KT - 1) / KT;
    DmaKRt<KT> la, lb;
    la.init(d.lda, job.m0, M, lane, wave);
    lb.init(d.ldb, job.n0, d.N, lane, wave);

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    constexpr int CPT = 2 * DmaKRt<KT>::NI;  // copy instructions per tile and thread
    auto copy_tile = [&](int st, int t) {
        const int kb = t * KT, ke = t < nk ? K : 0;
        la.copy(d.A, kb, ke, smem[st][0], wave);
        lb.copy(d.B, kb, ke, smem[st][1], wave);
    };
    // byte addresses in LDS of this lane's transpose reads for k block 0 of
    // stage 0: A fragments i = 0, 1 (first and second four k), then B fragments
    const uint32_t sbase = lds_addr(&smem[0][0][0]);
    uint32_t ra[8];
    {
        const int2 o[4] = {frag_tr_off(lane, wm * 64), frag_tr_off(lane, wm * 64 + 32), frag_tr_off(lane, wn * 64),
                           frag_tr_off(lane, wn * 64 + 32)};
#pragma unroll
        for (int f = 0; f < 4; ++f) {
            const uint32_t op = f < 2 ? 0u : (uint32_t)(KT * BM * 2);
            ra[2 * f] = sbase + op + 2 * o[f].x;
            ra[2 * f + 1] = sbase + op + 2 * o[f].y;
        }
    }
    // k blocks in pairs: the sixteen reads of a pair are issued together, the
    // first block's MFMAs wait for its eight (lgkmcnt counts up to 15)
    auto compute = [&](int st) {
        const uint32_t so = (uint32_t)st * (2 * KT * BM * 2);
#pragma unroll
        for (int kp = 0; kp < KT / 32; ++kp) {
            i32x2_t r[2][8];
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int q = 0; q < 8; ++q) r[h][q] = tr_read(ra[q] + so + (2 * kp + h) * 16 * BM * 2);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                lgkm_wait_tr(r[h], 1 - h);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            frag_cat(r[h][2 * i], r[h][2 * i + 1]), frag_cat(r[h][4 + 2 * j], r[h][5 + 2 * j]),
                            acc[i][j], 0, 0, 0);
            }
        }
    };
    auto step = [&](int t, int u) {
        copy_tile((u + NST - 1) % NST, t + NST - 1);
        compute(u);
        __builtin_amdgcn_s_waitcnt(vmcnt_lds0_imm(CPT * (NST - 2)));  // tile t + 1 has landed
        ring_barrier();
    };
#pragma unroll
    for (int u = 0; u < NST - 1; ++u) copy_tile(u, u);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(CPT * (NST - 2)));  // tile 0 has landed
    ring_barrier();
    int t = 0;
    for (; t + NST <= nk; t += NST) {  // whole rounds: static stage indices
#pragma unroll
        for (int u = 0; u < NST; ++u) step(t + u, u);
    }
    for (int u = 0; t < nk; ++t, ++u) step(t, u);
    __builtin_amdgcn_s_waitcnt(0);  // copies past the last tile
    __syncthreads();
    store_tile(d, acc, reinterpret_cast<float*>(&smem[0][0][0]), job, M, tid);
}

template <int KT, int NST>
__global__ void __launch_bounds__(NT, 2) gemm_wgrad_dma_kernel(const GemmGroupArg g) {
    __shared__ __attribute__((aligned(1024))) bf16_t smem[NST][2][KT * BM];
    for_group_tiles(g, [&](const GemmDesc& d, const TileJob& job, int M, int K) {
        wgrad_tile<KT, NST>(d, job, M, K, smem);
    });
}

// Tall tiles: 256 x 128 per workgroup, 128 x 64 per wave (4 x 2 accumulators),
// for groups that run beside other work with a capped grid.  Per MFMA they
// read a quarter fewer operand bytes than 128 x 128 tiles (A 256 rows, B 128
// rows per k).  Three 24 KB stages of KT = 32 (two workgroups per CU); the C
// tile leaves in two 128-row halves through the stages.
__device__ __forceinline__ void lgkm_wait_tr12(i32x2_t (&r)[12]) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7]),
                   "+v"(r[8]), "+v"(r[9]), "+v"(r[10]), "+v"(r[11]));
}

constexpr int kTallRows = 2 * BM;

template <int KT, int NST>
__device__ __forceinline__ void wgrad_tall_tile(const GemmDesc& d, const TileJob& job, int M, int K,
                                                bf16_t (*smem)[KT * (kTallRows + BN)]) {
    constexpr int RA = kTallRows, RB = BN, SA = KT * RA, SB = KT * RB;
    static_assert(NST * (SA + SB) * 2 >= BM * BN * 4, "a 128-row half of the C tile lives in the stages");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int nk = (K + KT - 1) / KT;
    DmaKRt<KT, RA> la;
    DmaKRt<KT, RB> lb;
    la.init(d.lda, job.m0, M, lane, wave);
    lb.init(d.ldb, job.n0, d.N, lane, wave);

    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    constexpr int CPT = DmaKRt<KT, RA>::NI + DmaKRt<KT, RB>::NI;  // copy instructions per tile and thread
    auto copy_tile = [&](int st, int t) {
        const int kb = t * KT, ke = t < nk ? K : 0;
        la.copy(d.A, kb, ke, smem[st], wave);
        lb.copy(d.B, kb, ke, smem[st] + SA, wave);
    };
    // byte addresses in LDS of this lane's transpose reads for k block 0 of
    // stage 0: A fragments i = 0..3 (rows 128 wm + 32 i), then B fragments
    // j = 0, 1 (rows 64 wn + 32 j); two reads each (first and second four k)
    const uint32_t sbase = lds_addr(&smem[0][0]);
    uint32_t ra[12];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int2 o = frag_tr_off<RA>(lane, wm * 128 + 32 * i);
        ra[2 * i] = sbase + 2 * o.x;
        ra[2 * i + 1] = sbase + 2 * o.y;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int2 o = frag_tr_off<RB>(lane, wn * 64 + 32 * j);
        ra[8 + 2 * j] = sbase + 2 * SA + 2 * o.x;
        ra[9 + 2 * j] = sbase + 2 * SA + 2 * o.y;
    }
    // k blocks of 16: twelve reads, then the block's eight MFMAs (which run
    // while the next block's reads are issued)
    auto compute = [&](int st) {
        const uint32_t so = (uint32_t)st * ((SA + SB) * 2);
#pragma unroll
        for (int kb16 = 0; kb16 < KT / 16; ++kb16) {
            i32x2_t r[12];
            const uint32_t ka = kb16 * 16 * RA * 2, kb = kb16 * 16 * RB * 2;
#pragma unroll
            for (int q = 0; q < 8; ++q) r[q] = tr_read(ra[q] + so + ka);
#pragma unroll
            for (int q = 8; q < 12; ++q) r[q] = tr_read(ra[q] + so + kb);
            lgkm_wait_tr12(r);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        frag_cat(r[2 * i], r[2 * i + 1]), frag_cat(r[8 + 2 * j], r[9 + 2 * j]), acc[i][j], 0, 0, 0);
        }
    };
    auto step = [&](int t, int u) {
        copy_tile((u + NST - 1) % NST, t + NST - 1);
        compute(u);
        __builtin_amdgcn_s_waitcnt(vmcnt_lds0_imm(CPT * (NST - 2)));  // tile t + 1 has landed
        ring_barrier();
    };
#pragma unroll
    for (int u = 0; u < NST - 1; ++u) copy_tile(u, u);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(CPT * (NST - 2)));  // tile 0 has landed
    ring_barrier();
    int t = 0;
    for (; t + NST <= nk; t += NST) {  // whole rounds: static stage indices
#pragma unroll
        for (int u = 0; u < NST; ++u) step(t + u, u);
    }
    for (int u = 0; t < nk; ++t, ++u) step(t, u);
    __builtin_amdgcn_s_waitcnt(0);  // copies past the last tile
    // the two 128-row halves: waves 2h and 2h + 1 stage half h, all drain it
    float* Cs = reinterpret_cast<float*>(&smem[0][0]);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        __syncthreads();  // the stages (h = 0) or the first half (h = 1) are free
        if (wm == h) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int lr = i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                        Cs[lr * BN + wn * 64 + j * 32 + (lane & 31)] = acc[i][j][r];
                    }
        }
        __syncthreads();
        TileJob half = job;
        half.m0 = job.m0 + h * BM;
        drain_tile<BM, NT, BN, 4>(d, Cs, half, M, tid);  // four-row batches: the other half's accumulators stay live
    }
}

template <int KT, int NST>
__global__ void __launch_bounds__(NT, 2) gemm_wgrad_tall_kernel(const GemmGroupArg g) {
    __shared__ __attribute__((aligned(1024))) bf16_t smem[NST][KT * (kTallRows + BN)];
    for_group_tiles<kTallRows>(g, [&](const GemmDesc& d, const TileJob& job, int M, int K) {
        wgrad_tall_tile<KT, NST>(d, job, M, K, smem);
    });
}

// ------------------------------------------------------------------ input gradients, copies into LDS
// C = A B with A row-major (k contiguous) and B k-major ([K][N], the rows of
// the tile contiguous), as in the input gradients dX = dY W: A in the 128 x 32
// tile layout of DmaRKc (its fragments by plain LDS reads), B in the [32 k][128
// row] layout of DmaKRt (its fragments by transpose reads), NST stages in a
// ring as in gemm_comp_dma_kernel; split-K slices and the epilogue as in
// gemm_kernel.
__device__ __forceinline__ void lgkm_wait_tr4(i32x2_t (&r)[4], int n) {
    if (n)
        asm volatile("s_waitcnt lgkmcnt(4)" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]));
    else
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]));
}

template <int KT, int NST>
__global__ void __launch_bounds__(NT, 2) gemm_rk_krt_dma_kernel(const GemmDesc d) {
    // the input-gradient chain is the critical path of the backward: its waves
    // win the issue arbitration against the weight-gradient waves they share
    // SIMDs with (wave priority, not a stream priority)
    __builtin_amdgcn_s_setprio(2);
    // NST stages of an A tile (KT / 32 blocks of 128 x 32) and a B tile (KT x 128);
    // reused for the C tile (64 KB)
    static_assert(KT == 32 || KT == 64, "tile depth");
    constexpr int KA = KT / CBK;  // A blocks per stage
    __shared__ __attribute__((aligned(1024))) bf16_t smem[NST][2][BM * KT];
    static_assert(NST * 2 * KT * BM * 2 >= BM * BN * 4, "the C tile lives in the stages");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int M = d.Mdev ? min(d.M, *d.Mdev) : d.M;
    const int K = d.K;
    if (d.prof_snap && (blockIdx.x | blockIdx.y | blockIdx.z) == 0 && tid == 0) {
        d.prof_snap[0] = M;
        d.prof_snap[1] = K;
    }
    TileJob job;
    if (!map_tile(d, M, K, job)) return;  // uniform for the whole workgroup
    const int S = job.S;
    const int kpad = (K + KT - 1) / KT * KT;
    const int kc = ((kpad + S - 1) / S + KT - 1) / KT * KT;
    const int kbeg = job.zt * kc;
    const int kstop = min(kpad, kbeg + kc);
    const int nk = kstop > kbeg ? (kstop - kbeg) / KT : 0;

    DmaRKc la;
    DmaKRt<KT> lb;
    la.init(d.lda, job.m0, M, lane, wave);
    lb.init(d.ldb, job.n0, d.N, lane, wave);

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    constexpr int CPT = 2 * KA + DmaKRt<KT>::NI;  // copy instructions per tile and thread
    auto copy_tile = [&](int st, int t) {
        const int kb = kbeg + t * KT, ke = t < nk ? K : 0;
#pragma unroll
        for (int a = 0; a < KA; ++a) la.copy(d.A, kb + CBK * a, ke, smem[st][0] + a * BM * CBK, wave);
        lb.copy(d.B, kb, ke, smem[st][1], wave);
    };
    const int lrow = lane & 31, lc = lane >> 5;
    // byte addresses in LDS of this lane's B transpose reads for k block 0 of stage 0
    uint32_t rb[4];
    {
        const uint32_t b0 = lds_addr(&smem[0][1][0]);
        const int2 o0 = frag_tr_off(lane, wn * 64), o1 = frag_tr_off(lane, wn * 64 + 32);
        rb[0] = b0 + 2 * o0.x;
        rb[1] = b0 + 2 * o0.y;
        rb[2] = b0 + 2 * o1.x;
        rb[3] = b0 + 2 * o1.y;
    }
    // k blocks of 16 in pairs (one A block of 32): the pair's eight transpose
    // reads are issued together, the first block's MFMAs wait for its four
    auto compute = [&](int st) {
        const uint32_t so = (uint32_t)st * (2 * KT * BM * 2);
#pragma unroll
        for (int kp = 0; kp < KA; ++kp) {
            const bf16_t* At = smem[st][0] + kp * BM * CBK;
            i32x2_t r[2][4];
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int q = 0; q < 4; ++q) r[h][q] = tr_read(rb[q] + so + (2 * kp + h) * 16 * BM * 2);
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                bf16x8_t a[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int row = wm * 64 + i * 32 + lrow, C = 2 * ks + lc;
                    a[i] = *reinterpret_cast<const bf16x8_t*>(&At[row * CBK + 8 * (C ^ ((row >> 2) & 3))]);
                }
                lgkm_wait_tr4(r[ks], 1 - ks);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            a[i], frag_cat(r[ks][2 * j], r[ks][2 * j + 1]), acc[i][j], 0, 0, 0);
            }
        }
    };
    auto step = [&](int t, int u) {
        copy_tile((u + NST - 1) % NST, t + NST - 1);
        compute(u);
        __builtin_amdgcn_s_waitcnt(vmcnt_lds0_imm(CPT * (NST - 2)));  // tile t + 1 has landed
        ring_barrier();
    };
#pragma unroll
    for (int u = 0; u < NST - 1; ++u) copy_tile(u, u);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(CPT * (NST - 2)));  // tile 0 has landed
    ring_barrier();
    int t = 0;
    for (; t + NST <= nk; t += NST) {
#pragma unroll
        for (int u = 0; u < NST; ++u) step(t + u, u);
    }
    for (int u = 0; t < nk; ++t, ++u) step(t, u);
    __builtin_amdgcn_s_waitcnt(0);  // copies past the last tile
    __syncthreads();
    store_tile(d, acc, reinterpret_cast<float*>(&smem[0][0][0]), job, M, tid);
}

// Sums the split-K partials and runs the epilogue; four columns per thread
// when N % 4 == 0, with the slices loaded four at a time.
__global__ void __launch_bounds__(256) splitk_reduce(const GemmDesc d) {
    const int M = d.Mdev ? min(d.M, *d.Mdev) : d.M;
    const int64_t full = (int64_t)d.M * d.N;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int Keff = d.Kdev ? min(d.K, *d.Kdev) : d.K;
    const int S = active_splits(d, M, d.nseg * gemm_kseg(d, Keff));
    if (S <= 1) return;  // the GEMM ran the epilogue itself
    if ((d.N & 3) == 0) {
        const int64_t total4 = (int64_t)M * d.N / 4;
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total4; i += stride) {
            const float* p = d.ws + 4 * i;
            const int row = (int)(4 * i / d.N), col = (int)(4 * i % d.N);
            // the epilogue's operands are loaded with the slices, before the first sum
            f32x4 bias = {0.f, 0.f, 0.f, 0.f};
            EpiIn4 e;
            if (d.vec_epi) {
                if (d.bias) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) bias[q] = d.bias[col + q];
                }
                e = epi_load4(d, row, col);
            }
            f32x4 v = *reinterpret_cast<const f32x4*>(p);
            int z = 1;
            for (; z + 3 < S; z += 4) {
                const f32x4 a = *reinterpret_cast<const f32x4*>(p + z * full);
                const f32x4 b = *reinterpret_cast<const f32x4*>(p + (z + 1) * full);
                const f32x4 c = *reinterpret_cast<const f32x4*>(p + (z + 2) * full);
                const f32x4 f = *reinterpret_cast<const f32x4*>(p + (z + 3) * full);
                v += (a + b) + (c + f);
            }
            for (; z < S; ++z) v += *reinterpret_cast<const f32x4*>(p + z * full);
            if (d.vec_epi) {
                epi_store4(d, row, col, v + bias + e.resid, e);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) epilogue(d, row, col + e, v[e]);
            }
        }
    } else {
        const int64_t total = (int64_t)M * d.N;
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
            float v = 0.f;
            for (int z = 0; z < S; ++z) v += d.ws[(int64_t)z * full + i];
            epilogue(d, (int)(i / d.N), (int)(i % d.N), v);
        }
    }
}

// launch_splitk_sum_multi: blocks are dealt to the jobs in order, job i
// taking ceil(M_i N_i / 1024) of them; each thread sums four consecutive
// elements (one when N_i % 4 != 0 or C_i is not 16-byte aligned).
__global__ void __launch_bounds__(256) splitk_sum_multi(const SplitJobs jobs) {
    int bid = blockIdx.x, ji = 0;
    for (; ji < jobs.n - 1; ++ji) {
        const int nb = (int)(((int64_t)jobs.j[ji].M * jobs.j[ji].N + 1023) / 1024);
        if (bid < nb) break;
        bid -= nb;
    }
    const SplitJob& J = jobs.j[ji];
    const int64_t full = (int64_t)J.M * J.N;
    const int64_t e0 = (int64_t)bid * 1024 + 4 * threadIdx.x;
    if (e0 >= full) return;
    const bool vec = (J.N & 3) == 0 && (J.ldc & 3) == 0 && ((uintptr_t)J.C & 15) == 0;
    if (vec) {
        const float* p = J.ws + e0;
        f32x4 v = *reinterpret_cast<const f32x4*>(p);
        int z = 1;
        for (; z + 3 < J.S; z += 4) {
            const f32x4 a = *reinterpret_cast<const f32x4*>(p + z * full);
            const f32x4 b = *reinterpret_cast<const f32x4*>(p + (z + 1) * full);
            const f32x4 c = *reinterpret_cast<const f32x4*>(p + (z + 2) * full);
            const f32x4 f = *reinterpret_cast<const f32x4*>(p + (z + 3) * full);
            v += (a + b) + (c + f);
        }
        for (; z < J.S; ++z) v += *reinterpret_cast<const f32x4*>(p + z * full);
        const int64_t row = e0 / J.N, col = e0 - row * J.N;
        *reinterpret_cast<f32x4*>(J.C + row * J.ldc + col) = v;
    } else {
        for (int64_t e = e0; e < min(e0 + 4, full); ++e) {
            float v = 0.f;
            for (int z = 0; z < J.S; ++z) v += J.ws[(int64_t)z * full + e];
            const int64_t row = e / J.N, col = e - row * J.N;
            J.C[row * J.ldc + col] = v;
        }
    }
}

template <int NSEG, class LA = DmaRKc, int NST = 2>
void launch_comp(const GemmDesc& d, hipStream_t s) {
    ProfInfo pi;
    pi.kind = PROF_GEMM;
    pi.M = d.M; pi.N = d.N; pi.K = d.K; pi.nseg = d.nseg;
    pi.Mdev = d.Mdev; pi.Kdev = d.Kdev;
    hipEvent_t ea, eb;
    constexpr bool conv = std::is_same<LA, DmaConvA>::value;
    const char* name = conv ? (NSEG == 3 ? "gemm_comp_dma_kernel<3, conv>" : "gemm_comp_dma_kernel<2, conv>")
                            : (NSEG == 3 ? "gemm_comp_dma_kernel<3>" : "gemm_comp_dma_kernel<2>");
    const int h = prof_begin_ext(name, pi, &ea, &eb);
    GemmDesc dd = d;
    dd.prof_snap = prof_snap(h);
    dim3 grid((d.N + BN - 1) / BN, (d.M + BM - 1) / BM, d.splits);
    hipExtLaunchKernelGGL((gemm_comp_dma_kernel<NSEG, NST, LA>), grid, dim3(NT), 0, s, ea, eb, 0, dd);
    prof_end_ext(h);
}

void launch_rk_krt(const GemmDesc& d, hipStream_t s) {
    ProfInfo pi;
    pi.kind = PROF_GEMM;
    pi.M = d.M; pi.N = d.N; pi.K = d.K; pi.nseg = d.nseg;
    pi.Mdev = d.Mdev; pi.Kdev = d.Kdev;
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("gemm_rk_krt_dma_kernel", pi, &ea, &eb);
    GemmDesc dd = d;
    dd.prof_snap = prof_snap(h);
    dim3 grid((d.N + BN - 1) / BN, (d.M + BM - 1) / BM, d.splits);
    hipExtLaunchKernelGGL((gemm_rk_krt_dma_kernel<kDgradKT, kDgradNST>), grid, dim3(NT), 0, s, ea, eb, 0, dd);
    prof_end_ext(h);
}

template <int AM, int BMODE, bool AL = false>
void launch(const GemmDesc& d, hipStream_t s) {
    // kernel names as the profilers print them
    static const char* names[9][9] = {};
    static char buf[9][9][32];
    if (!names[AM][BMODE]) {
        snprintf(buf[AM][BMODE], sizeof(buf[AM][BMODE]), "gemm_kernel<%d, %d>", AM, BMODE);
        names[AM][BMODE] = buf[AM][BMODE];
    }
    ProfInfo pi;
    pi.kind = PROF_GEMM;
    pi.M = d.M; pi.N = d.N; pi.K = d.K; pi.nseg = d.nseg;
    pi.Mdev = d.Mdev; pi.Kdev = d.Kdev;
    hipEvent_t ea, eb;
    const int h = prof_begin_ext(names[AM][BMODE], pi, &ea, &eb);
    GemmDesc dd = d;
    dd.prof_snap = prof_snap(h);
    dim3 grid((d.N + BN - 1) / BN, (d.M + BM - 1) / BM, d.splits);
    hipExtLaunchKernelGGL((gemm_kernel<AM, BMODE, AL>), grid, dim3(NT), 0, s, ea, eb, 0, dd);
    prof_end_ext(h);
}

}  // namespace


fo_status gemm_group(const GemmDesc* ds, int n, hipStream_t s, int max_wg) {
    FO_CHECK(n >= 1 && n <= kGemmGroupMax, "gemm_group: %d products", n);
    // a group runs in one launch when every member is an unsplit, aligned
    // product of k-major operands (the weight-gradient form); otherwise each
    // member is launched on its own
    auto al16 = [](const void* p) { return p == nullptr || ((uintptr_t)p & 15) == 0; };
    bool one = true;
    for (int i = 0; i < n; ++i) {
        const GemmDesc& d = ds[i];
        one = one && d.amode == OP_KR && d.bmode == OP_KR && d.splits == 1 && d.nseg == 1 && !d.Mdev &&
              !d.colpart && d.lda % 8 == 0 && d.ldb % 8 == 0 && d.M % 8 == 0 && d.N % 8 == 0 && al16(d.A) &&
              al16(d.B);
    }
    if (!one) {
        for (int i = 0; i < n; ++i) {
            fo_status st = gemm(ds[i], s);
            if (st != FO_OK) return st;
        }
        return FO_OK;
    }
    GemmGroupArg g;
    g.n = n;
    int tiles = 0, tall_tiles = 0;
    ProfInfo pi;
    pi.kind = PROF_GEMM;
    pi.ngroup = n;
    for (int i = 0; i < kGemmGroupMax; ++i) {
        const GemmDesc& d = ds[i < n ? i : 0];
        FO_CHECK(d.M > 0 && d.N > 0 && d.K > 0, "gemm_group: empty product %dx%dx%d", d.M, d.N, d.K);
        FO_CHECK(d.Cf || d.Cb, "gemm_group: no output");
        FO_CHECK(!d.sgd_theta || (d.Cf && d.sgd_hi && d.sgd_lo), "gemm_group: the fused SGD needs Cf and both parts");
        g.d[i] = d;
        auto al = [](const void* p, uintptr_t m) { return p == nullptr || ((uintptr_t)p & (m - 1)) == 0; };
        bool v = d.N % 4 == 0 && al(d.Cf, 16) && al(d.resid, 16) && al(d.Cb, 8) && al(d.Cb2, 8) &&
                 al(d.dact_out, 8) && al(d.mask, 8) && al(d.dact, 8) && al(d.sgd_theta, 16) && al(d.sgd_hi, 8) &&
                 al(d.sgd_lo, 8);
        if (d.Cf) v = v && d.ldcf % 4 == 0;
        if (d.resid) v = v && d.ldr % 4 == 0;
        if (d.Cb) v = v && d.ldcb % 4 == 0;
        if (d.dact_out || d.mask || d.dact) v = v && d.ldm % 4 == 0;
        g.d[i].vec_epi = v ? 1 : 0;
        g.d[i].prof_snap = nullptr;
        if (i < n) {
            tiles += (int)(cdiv(d.M, BM) * cdiv(d.N, BN));
            tall_tiles += (int)(cdiv(d.M, kTallRows) * cdiv(d.N, BN));
            pi.gN[i] = d.N;
        }
    }
    // a capped group runs beside other work: 256 x 128 tiles read a quarter
    // fewer operand bytes per MFMA and leave more of the GPU to that work; an
    // uncapped group has the GPU to itself and fills it better with 128 x 128
    const bool tall = max_wg > 0;
    hipEvent_t ea, eb;
    const int h = prof_begin_ext(tall ? "gemm_wgrad_tall_kernel" : "gemm_wgrad_dma_kernel", pi, &ea, &eb);
    g.prof_snap = prof_snap(h);
    int grid = tall ? tall_tiles : tiles;
    if (max_wg > 0 && grid > max_wg) grid = std::max(8, max_wg / 8 * 8);
    if (tall)
        hipExtLaunchKernelGGL((gemm_wgrad_tall_kernel<32, 3>), dim3(grid), dim3(NT), 0, s, ea, eb, 0, g);
    else
        hipExtLaunchKernelGGL((gemm_wgrad_dma_kernel<kWgradKT, kWgradNST>), dim3(grid), dim3(NT), 0, s, ea, eb, 0,
                              g);
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status launch_splitk_sum_multi(const SplitJobs& jobs, hipStream_t s) {
    FO_CHECK(jobs.n >= 1 && jobs.n <= kSplitJobsMax, "split-K sums: %d jobs", jobs.n);
    int64_t blocks = 0;
    for (int i = 0; i < jobs.n; ++i) {
        const SplitJob& J = jobs.j[i];
        FO_CHECK(J.ws && J.C && J.S >= 1 && J.M >= 1 && J.N >= 1 && J.ldc >= J.N, "split-K sums: bad job %d", i);
        blocks += cdiv((int64_t)J.M * J.N, 1024);
    }
    hipEvent_t ea, eb;
    const int h = prof_begin_ext("splitk_sum_multi", ProfInfo(), &ea, &eb);
    hipExtLaunchKernelGGL(splitk_sum_multi, dim3((unsigned)blocks), dim3(256), 0, s, ea, eb, 0, jobs);
    prof_end_ext(h);
    FO_LAUNCHED();
    return FO_OK;
}

fo_status gemm(const GemmDesc& d, hipStream_t s) {
    FO_CHECK(d.M > 0 && d.N > 0 && d.K > 0, "gemm: empty problem %dx%dx%d", d.M, d.N, d.K);
    FO_CHECK(d.splits >= 1 && (d.splits == 1 || d.ws != nullptr), "gemm: split-K needs a workspace");
    FO_CHECK(d.Cf || d.Cb, "gemm: no output");
    FO_CHECK(!d.colpart || d.splits == 1, "gemm: column sums need splits == 1");
    FO_CHECK(!d.sgd_theta || (d.Cf && d.sgd_hi && d.sgd_lo && !d.defer_reduce),
             "gemm: the fused SGD needs Cf, both bf16 parts and a reduction in this call");
    const bool conv = d.amode == OP_CONV_FWD || d.amode == OP_CONV_DX || d.bmode == OP_CONV_DXW ||
                      d.bmode == OP_CONV_DWX;
    if (conv) {
        FO_CHECK(d.g.Ci % BK == 0 || d.amode != OP_CONV_FWD, "gemm: conv forward needs Ci %% %d == 0", BK);
        FO_CHECK(d.g.Co % BK == 0 || d.amode != OP_CONV_DX, "gemm: conv dgrad needs Co %% %d == 0", BK);
        FO_CHECK(d.g.Ci % 8 == 0, "gemm: conv needs Ci %% 8 == 0");
    }
    FO_CHECK(d.nseg >= 1 && d.nseg <= 3, "gemm: nseg=%d must be 1, 2 or 3", d.nseg);
    if (d.nseg > 1) {
        FO_CHECK(d.B2 && (d.nseg == 2 || d.A2), "gemm: compensated product needs its low parts");
        FO_CHECK(!d.Kdev, "gemm: compensated product needs a static K");
    }
    // four-column epilogue: N and every leading dimension multiples of 4, fp32
    // operands 16-byte and bf16 operands 8-byte aligned
    GemmDesc dv = d;
    {
        auto al = [](const void* p, uintptr_t m) { return p == nullptr || ((uintptr_t)p & (m - 1)) == 0; };
        bool v = d.N % 4 == 0 && al(d.ws, 16) && al(d.Cf, 16) && al(d.resid, 16) && al(d.Cb, 8) && al(d.Cb2, 8) &&
                 al(d.dact_out, 8) && al(d.mask, 8) && al(d.dact, 8) && al(d.colpart, 4) && al(d.sgd_theta, 16) &&
                 al(d.sgd_hi, 8) && al(d.sgd_lo, 8);
        if (d.Cf) v = v && d.ldcf % 4 == 0;
        if (d.resid) v = v && d.ldr % 4 == 0;
        if (d.Cb) v = v && d.ldcb % 4 == 0;
        if (d.dact_out || d.mask || d.dact) v = v && d.ldm % 4 == 0;
        dv.vec_epi = v ? 1 : 0;
    }
    const int a = d.amode, b = d.bmode;
    // aligned variant: every contiguous dimension a multiple of 8 and 16-byte rows
    auto al16 = [](const void* p) { return p == nullptr || ((uintptr_t)p & 15) == 0; };
    auto op_aligned = [&](int mode, const bf16_t* P, const bf16_t* P2, int64_t ld, int rows) {
        if (ld % 8 != 0 || !al16(P) || !al16(P2)) return false;
        return mode == OP_RK ? (d.K % 8 == 0 && !d.Kdev) : (rows % 8 == 0);
    };
    // (a k-major A with a device-side row bound may end inside an 8-row chunk)
    const bool al = (a == OP_RK || a == OP_KR) && (b == OP_RK || b == OP_KR) && !(a == OP_KR && d.Mdev) &&
                    op_aligned(a, d.A, d.A2, d.lda, d.M) && op_aligned(b, d.B, d.B2, d.ldb, d.N);
    // a 16-byte aligned operand whose contiguous rows come in whole chunks of 8
    auto conv_al = [&](const bf16_t* P, int rows) { return al16(P) && rows % 8 == 0; };
    // compensated convolution forward, single pass with copies straight into LDS:
    // 16-byte aligned input and weights, Ci % 64 == 0, static sizes
    const bool conv_comp = a == OP_CONV_FWD && b == OP_RK && d.nseg > 1 && !d.Kdev && d.g.Ci % 64 == 0 &&
                           al16(d.A) && al16(d.A2) && op_aligned(OP_RK, d.B, d.B2, d.ldb, d.N);
    // an unsplit aligned product of two k-major operands (a weight gradient)
    // runs as a group of one on the kernel with copies into LDS
    if (a == OP_KR && b == OP_KR && al && d.splits == 1 && d.nseg == 1 && !d.colpart) return gemm_group(&d, 1, s, 0);
    // (two stages and two workgroups per CU beat deeper rings at one per CU, and
    // 256 x 128 tiles with a three-stage ring at one per CU on these products)
    if (a == OP_RK && b == OP_RK && al && d.nseg > 1 && !d.Kdev)
        d.nseg == 3 ? launch_comp<3>(dv, s) : launch_comp<2>(dv, s);
    else if (a == OP_RK && b == OP_RK) al ? launch<OP_RK, OP_RK, true>(dv, s) : launch<OP_RK, OP_RK>(dv, s);
    else if (a == OP_RK && b == OP_KR && al && d.nseg == 1 && !d.Kdev) launch_rk_krt(dv, s);
    else if (a == OP_RK && b == OP_KR) al ? launch<OP_RK, OP_KRT, true>(dv, s) : launch<OP_RK, OP_KR>(dv, s);
    else if (a == OP_KR && b == OP_KR) al ? launch<OP_KRT, OP_KRT, true>(dv, s) : launch<OP_KR, OP_KR>(dv, s);
    else if (a == OP_KR && b == OP_RK) al ? launch<OP_KRT, OP_RK, true>(dv, s) : launch<OP_KR, OP_RK>(dv, s);
    else if (a == OP_CONV_FWD && b == OP_RK && conv_comp)
        d.nseg == 3 ? launch_comp<3, DmaConvA>(dv, s) : launch_comp<2, DmaConvA>(dv, s);
    else if (a == OP_CONV_FWD && b == OP_RK) launch<OP_CONV_FWD, OP_RK>(dv, s);
    else if (a == OP_CONV_DX && b == OP_CONV_DXW && conv_al(d.B, d.g.Ci))
        launch<OP_CONV_DX, OP_CONV_DXWT, true>(dv, s);
    else if (a == OP_CONV_DX && b == OP_CONV_DXW) launch<OP_CONV_DX, OP_CONV_DXW>(dv, s);
    else if (a == OP_KR && b == OP_CONV_DWX && conv_al(d.A, d.M) && d.lda % 8 == 0 && !d.Mdev && !d.Kdev)
        launch<OP_KRT, OP_CONV_DWXT, true>(dv, s);
    else if (a == OP_KR && b == OP_CONV_DWX) launch<OP_KR, OP_CONV_DWX>(dv, s);
    else {
        set_error("gemm: unsupported operand modes %d/%d", a, b);
        return FO_EINVAL;
    }
    FO_LAUNCHED();
    if (d.splits > 1 && !d.defer_reduce) {
        int64_t total = (int64_t)d.M * d.N;
        if (d.N % 4 == 0) total /= 4;
        int grid = (int)std::min<int64_t>(cdiv(total, 256), 4096);
        hipEvent_t ea, eb;
        const int h = prof_begin_ext("splitk_reduce", ProfInfo(), &ea, &eb);
        hipExtLaunchKernelGGL(splitk_reduce, dim3(grid), dim3(256), 0, s, ea, eb, 0, dv);
        prof_end_ext(h);
        FO_LAUNCHED();
    }
    return FO_OK;
}

}  // namespace fo
