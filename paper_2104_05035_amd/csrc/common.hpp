// Shared device/host helpers of librat3d (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "rat3d.h"

namespace rat3d {

typedef uint16_t bf16;  // bfloat16 storage (upper half of a float32)

// bfloat16 <-> float32.  Rounding is to nearest, ties to even, on the float32
// bit pattern; NaN stays a quiet NaN.
__device__ __forceinline__ float bf2f(bf16 h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ bf16 f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16)(u >> 16);
}

// Storage-type traits: load as float, store from float.
template <typename T> struct Elt;
template <> struct Elt<float> {
    static constexpr rat3d_dtype dtype = RAT3D_F32;
    __device__ __forceinline__ static float ld(const float* p) { return *p; }
    __device__ __forceinline__ static float cvt(float v) { return v; }
    __device__ __forceinline__ static void st(float* p, float v) { *p = v; }
    __device__ __forceinline__ static float from_bits(float v) { return v; }
    __device__ __forceinline__ static float to_bits(float v) { return v; }
};
template <> struct Elt<bf16> {
    static constexpr rat3d_dtype dtype = RAT3D_BF16;
    __device__ __forceinline__ static float ld(const bf16* p) { return bf2f(*p); }
    __device__ __forceinline__ static float cvt(bf16 v) { return bf2f(v); }
    __device__ __forceinline__ static void st(bf16* p, float v) { *p = f2bf(v); }
    __device__ __forceinline__ static float from_bits(bf16 v) { return bf2f(v); }
    __device__ __forceinline__ static bf16 to_bits(float v) { return f2bf(v); }
};

// MFMA operand / accumulator vector types.
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

// Workgroup ids are dealt round-robin over the 8 XCDs; remap them so that
// XCD x runs the contiguous ids [x * q, (x + 1) * q) of a balanced split
// (a ragged tail keeps its place).  Neighbouring tiles then share an L2.
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
    const int q = nb >> 3;
    if (q == 0 || bid >= q * 8) return bid;
    return (bid & 7) * q + (bid >> 3);
}

__host__ __device__ __forceinline__ int64_t ceil_div(int64_t a, int64_t b) {
    return (a + b - 1) / b;
}

inline int out_dim(int in, int k, int s, int p) { return (in + 2 * p - k) / s + 1; }

// Launch-error check used by host launchers: returns RAT3D_EHIP from the
// enclosing function after recording the message.
void set_error(const char* fmt, ...);
#define RAT3D_LAUNCH_CHECK()                                                          \
    do {                                                                              \
        hipError_t e_ = hipGetLastError();                                            \
        if (e_ != hipSuccess) {                                                       \
            ::rat3d::set_error("HIP launch failed: %s (%s:%d)", hipGetErrorString(e_), \
                               __FILE__, __LINE__);                                   \
            return RAT3D_EHIP;                                                        \
        }                                                                             \
    } while (0)

}  // namespace rat3d
