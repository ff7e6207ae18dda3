// 16-byte vector loads/stores of float32 or bfloat16 tensors as float lanes.
#pragma once

#include "common.hpp"

namespace rat3d {

// VEC elements starting at p (p aligned to VEC * sizeof(T)).
template <typename T, int VEC>
__device__ __forceinline__ void vload(const T* __restrict__ p, float (&o)[VEC]) {
    if constexpr (VEC == 1) {
        o[0] = Elt<T>::ld(p);
    } else if constexpr (sizeof(T) == 2 && VEC == 8) {
        const uint4 u = *reinterpret_cast<const uint4*>(p);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[2 * i] = __uint_as_float(w[i] << 16);
            o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    } else if constexpr (sizeof(T) == 4 && VEC == 4) {
        const float4 u = *reinterpret_cast<const float4*>(p);
        o[0] = u.x; o[1] = u.y; o[2] = u.z; o[3] = u.w;
    } else {
        static_assert(VEC == 1, "unsupported vector width");
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void vstore(T* __restrict__ p, const float (&o)[VEC]) {
    if constexpr (VEC == 1) {
        Elt<T>::st(p, o[0]);
    } else if constexpr (sizeof(T) == 2 && VEC == 8) {
        uint4 u;
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = pack_bf16x2(o[2 * i], o[2 * i + 1]);
        u.x = w[0]; u.y = w[1]; u.z = w[2]; u.w = w[3];
        *reinterpret_cast<uint4*>(p) = u;
    } else if constexpr (sizeof(T) == 4 && VEC == 4) {
        *reinterpret_cast<float4*>(p) = make_float4(o[0], o[1], o[2], o[3]);
    } else {
        static_assert(VEC == 1, "unsupported vector width");
    }
}

// Natural 16-byte vector width of T.
template <typename T> constexpr int vec16() { return 16 / (int)sizeof(T); }

}  // namespace rat3d
