// Internal helpers shared by the HIP translation units of libfedoptima.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "../../include/fedoptima.h"

namespace fo {

// ------------------------------------------------------------------ errors
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));

#define FO_HIP(call)                                                                  \
    do {                                                                              \
        hipError_t e_ = (call);                                                       \
        if (e_ != hipSuccess) {                                                       \
            ::fo::set_error("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_),    \
                            __FILE__, __LINE__);                                      \
            return FO_EHIP;                                                           \
        }                                                                             \
    } while (0)

#define FO_CHECK(cond, ...)                                                           \
    do {                                                                              \
        if (!(cond)) {                                                                \
            ::fo::set_error(__VA_ARGS__);                                             \
            return FO_EINVAL;                                                         \
        }                                                                             \
    } while (0)

// Launch check: a failed launch is reported through hipGetLastError.
#define FO_LAUNCHED()                                                                 \
    do {                                                                              \
        hipError_t e_ = hipGetLastError();                                            \
        if (e_ != hipSuccess) {                                                       \
            ::fo::set_error("kernel launch failed: %s (%s:%d)", hipGetErrorString(e_), \
                            __FILE__, __LINE__);                                      \
            return FO_EHIP;                                                           \
        }                                                                             \
    } while (0)

// native vector types (usable with the clang builtins)
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ bf16
typedef uint16_t bf16_t;  // storage type: the upper 16 bits of an IEEE fp32

__host__ __device__ inline float bf2f(bf16_t h) {
    union { uint32_t u; float f; } v;
    v.u = (uint32_t)h << 16;
    return v.f;
}

// fp32 -> bf16, round to nearest even (inputs are finite).  Device code uses
// the gfx950 conversion instruction (v_cvt_pk_bf16_f32, the same rounding);
// host code rounds the bit pattern.
__host__ __device__ inline bf16_t f2bf(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_bit_cast(bf16_t, (__bf16)f);
#else
    union { uint32_t u; float f; } v;
    v.f = f;
    uint32_t u = v.u;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
#endif
}

// Two fp32 -> one packed bf16 pair (a in the low half), round to nearest even.
__device__ inline uint32_t f2bf2(float a, float b) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// The batch of a training step as its kernels read it: a model-owned device
// record that the step's first launch fills with the caller's pointers, so
// that a captured step can be replayed on another batch by changing the
// arguments of that one launch (no copy of the batch).
struct StepIn {
    const void* x;
    const int32_t* labels;
    const int32_t* lengths;
    void* out;  // the device-side step's output activations (NULL for server steps)
};

// Device memory arena: one hipMalloc, bump allocation, 256-byte alignment.
struct Arena {
    char* base = nullptr;
    size_t size = 0, used = 0;
    template <class T>
    T* take(size_t count) {
        size_t bytes = (count * sizeof(T) + 255) & ~size_t(255);
        if (used + bytes > size) return nullptr;
        T* p = (T*)(base + used);
        used += bytes;
        return p;
    }
};

}  // namespace fo
