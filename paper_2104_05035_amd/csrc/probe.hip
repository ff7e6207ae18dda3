// Achievable-peak probes for the measurement report: a pure bf16 MFMA stream
// (the ceiling the convolution kernels are compared with, next to the
// datasheet's 2.5 PFLOP/s) and a streaming 16-byte copy (the ceiling of the
// bandwidth-bound kernels, next to the datasheet's 8 TB/s).  Neither touches
// the training data.
#include "kernels.hpp"

namespace rat3d {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kChains = 4;  // independent accumulators per wave

// Each wave issues kChains independent v_mfma_f32_16x16x32_bf16 per iteration
// (16 x 16 x 32 x 2 flops each); the sums are stored so nothing is removed.
__global__ __launch_bounds__(kProbeThreads) void probe_mfma_k(int iters, float* __restrict__ sink) {
    const int lane = threadIdx.x & 63;
    bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(0.001f * (float)(lane + i));
        b[i] = (__bf16)(0.002f * (float)(63 - lane + i));
    }
    // named accumulators with distinct starting values (an array, or equal
    // starts, let the compiler shuffle registers between the MFMAs)
    const float l = (float)lane;
    f32x4 c0 = {l, 0.f, 0.f, 0.f}, c1 = {0.f, l, 0.f, 0.f}, c2 = {0.f, 0.f, l, 0.f},
          c3 = {0.f, 0.f, 0.f, l};
    for (int it = 0; it < iters; it += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            c0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c3, 0, 0, 0);
        }
    }
    const f32x4 t = c0 + c1 + c2 + c3;
    const float s = t[0] + t[1] + t[2] + t[3];
    sink[(int64_t)blockIdx.x * kProbeThreads + threadIdx.x] = s;
}

// Each workgroup copies 4 x 256 16-byte vectors: four loads in flight per
// thread, every load instruction covering 1 KiB contiguous per wave; the grid
// covers the buffer once (the shape of the fast elementwise passes).
__global__ __launch_bounds__(kProbeThreads) void probe_copy_k(const uint4* __restrict__ src,
                                                              uint4* __restrict__ dst,
                                                              int64_t n) {
    const int64_t base = (int64_t)blockIdx.x * kProbeThreads * 4 + threadIdx.x;
    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t i = base + j * kProbeThreads;
        if (i < n) v[j] = src[i];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t i = base + j * kProbeThreads;
        if (i < n) dst[i] = v[j];
    }
}

}  // namespace
}  // namespace rat3d

using namespace rat3d;

extern "C" {

double rat3d_probe_mfma_flops(int blocks, int iters) {
    iters = (iters + 7) / 8 * 8;  // the loop runs whole groups of 8 iterations
    return (double)blocks * (kProbeThreads / 64) * (double)iters * kChains * 16.0 * 16.0 * 32.0 *
           2.0;
}

rat3d_status rat3d_probe_mfma(int blocks, int iters, float* sink, void* stream) {
    if (blocks < 1 || iters < 1 || !sink) {
        set_error("rat3d_probe_mfma: blocks, iters >= 1 and a sink of blocks * 256 floats");
        return RAT3D_EINVAL;
    }
    probe_mfma_k<<<blocks, kProbeThreads, 0, (hipStream_t)stream>>>(iters, sink);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status rat3d_probe_copy(const void* src, void* dst, size_t bytes, void* stream) {
    if (!src || !dst || bytes % 16 != 0 || ((uintptr_t)src & 15u) || ((uintptr_t)dst & 15u)) {
        set_error("rat3d_probe_copy: 16-byte aligned buffers and a multiple of 16 bytes");
        return RAT3D_EINVAL;
    }
    const int64_t n = (int64_t)(bytes / 16);
    const int64_t blocks = ceil_div(n, (int64_t)kProbeThreads * 4);
    probe_copy_k<<<(unsigned)blocks, kProbeThreads, 0, (hipStream_t)stream>>>(
        (const uint4*)src, (uint4*)dst, n);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // extern "C"
