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
    // v_cvt_pk_bf16_f32: round to nearest even, NaN stays a quiet NaN
    return __builtin_bit_cast(bf16, (__bf16)f);
}

// Two floats to packed bfloat16 (lo in bits 0-15), one instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
// The soft mask's sigmoid: one definition for every kernel that forms it, so
// that a mask recomputed elsewhere has the same bits.
__device__ __forceinline__ float sigmoidf(float z) { return 1.f / (1.f + expf(-z)); }

// Storage-type traits: load as float, store from float.
template <typename T> struct Elt;
template <> struct Elt<float> {
    static constexpr rat3d_dtype dtype = RAT3D_F32;
    __device__ __forceinline__ static float ld(const float* p) { return *p; }
    __device__ __forceinline__ static float cvt(float v) { return v; }
    __device__ __forceinline__ static void st(float* p, float v) { *p = v; }
    __device__ __forceinline__ static float from_bits(float v) { return v; }
    __device__ __forceinline__ static float to_bits(float v) { return v; }
    // the value a store of v holds
    __device__ __forceinline__ static float round(float v) { return v; }
};
template <> struct Elt<bf16> {
    static constexpr rat3d_dtype dtype = RAT3D_BF16;
    __device__ __forceinline__ static float ld(const bf16* p) { return bf2f(*p); }
    __device__ __forceinline__ static float cvt(bf16 v) { return bf2f(v); }
    __device__ __forceinline__ static void st(bf16* p, float v) { *p = f2bf(v); }
    __device__ __forceinline__ static float from_bits(bf16 v) { return bf2f(v); }
    __device__ __forceinline__ static bf16 to_bits(float v) { return f2bf(v); }
    __device__ __forceinline__ static float round(float v) { return bf2f(f2bf(v)); }
};

// MFMA operand / accumulator vector types.
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

// Raw buffer loads: a 128-bit resource in SGPRs (base, byte size) plus a
// per-lane byte offset (VGPR) and a wave-uniform byte offset (SGPR), so the
// address arithmetic of the hot loops stays off the vector ALU.  Callers keep
// every offset inside the buffer.
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}
// The same resource for a base and size that are wave-uniform but that the
// compiler may hold in vector registers: each word is taken from the first
// lane, so the resource stays in scalar registers (no per-lane loop around
// the accesses that use it).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc_u(const void* p, uint32_t bytes) {
    const uint64_t a = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return buf_rsrc((const void*)(((uint64_t)hi << 32) | lo), __builtin_amdgcn_readfirstlane(bytes));
}
__device__ __forceinline__ uint4 buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                          uint32_t soff) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 buf_ld8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    return make_uint2(v.x, v.y);
}
__device__ __forceinline__ uint32_t buf_ld2(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                            uint32_t soff) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}
__device__ __forceinline__ void buf_st8(__amdgpu_buffer_rsrc_t r, uint2 v, uint32_t voff,
                                        uint32_t soff) {
    const u32x2 w = {v.x, v.y};
    __builtin_amdgcn_raw_buffer_store_b64(w, r, voff, soff, 0);
}
__device__ __forceinline__ void buf_st16(__amdgpu_buffer_rsrc_t r, uint4 v, uint32_t voff,
                                         uint32_t soff) {
    const u32x4 w = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, voff, soff, 0);
}

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

// Compute units of the current device (queried once per device; 256 on MI355X).
int device_cus();
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
