// Soft-mask branch kernels of the residual attention module: max pooling
// down (with a uint8 argmax), trilinear resampling up, and the sigmoid fuse
// out = (1 + sigmoid(z)) * T.  All are HBM-bound elementwise/stencil kernels;
// every backward is written in gather form (one thread per destination
// element, no atomics), so results are deterministic.
#include "common.hpp"
#include "kernels.hpp"
#include "vec.hpp"
#include "prof.hpp"
#include "bn_coef.hpp"

namespace rat3d {

constexpr int kEwThreads = 256;

// ---------------------------------------------------------------- max pool
template <typename T>
__global__ __launch_bounds__(kEwThreads) void pool_fwd_k(const T* __restrict__ x, int NC, int D,
                                                         int H, int W, int k, int s, int p,
                                                         int Do, int Ho, int Wo,
                                                         T* __restrict__ y,
                                                         uint8_t* __restrict__ am) {
    const int64_t o = (int64_t)blockIdx.x * kEwThreads + threadIdx.x;
    const int64_t total = (int64_t)NC * Do * Ho * Wo;
    if (o >= total) return;
    const int ow = (int)(o % Wo);
    const int oh = (int)((o / Wo) % Ho);
    const int od = (int)((o / ((int64_t)Wo * Ho)) % Do);
    const int64_t nc = o / ((int64_t)Wo * Ho * Do);
    const T* xp = x + nc * D * H * W;
    float best = 0.f;
    int arg = -1;
    for (int kd = 0; kd < k; ++kd) {
        const int id = od * s - p + kd;
        if ((unsigned)id >= (unsigned)D) continue;
        for (int kh = 0; kh < k; ++kh) {
            const int ih = oh * s - p + kh;
            if ((unsigned)ih >= (unsigned)H) continue;
            for (int kw = 0; kw < k; ++kw) {
                const int iw = ow * s - p + kw;
                if ((unsigned)iw >= (unsigned)W) continue;
                const float v = Elt<T>::ld(xp + ((int64_t)id * H + ih) * W + iw);
                if (arg < 0 || v > best) {  // first maximum in scan order
                    best = v;
                    arg = (kd * k + kh) * k + kw;
                }
            }
        }
    }
    Elt<T>::st(y + o, best);
    am[o] = (uint8_t)arg;
}

// Gather form: input voxel i collects dy of every window whose argmax is i.
template <typename T>
__global__ __launch_bounds__(kEwThreads) void pool_bwd_k(const T* __restrict__ dy,
                                                         const uint8_t* __restrict__ am, int NC,
                                                         int D, int H, int W, int k, int s,
                                                         int p, int Do, int Ho, int Wo,
                                                         T* __restrict__ dx, int accumulate) {
    const int64_t i = (int64_t)blockIdx.x * kEwThreads + threadIdx.x;
    const int64_t total = (int64_t)NC * D * H * W;
    if (i >= total) return;
    const int iw = (int)(i % W);
    const int ih = (int)((i / W) % H);
    const int id = (int)((i / ((int64_t)W * H)) % D);
    const int64_t nc = i / ((int64_t)W * H * D);
    // windows o with o*s - p <= i <= o*s - p + k - 1
    auto lo = [&](int v) { int a = v + p - (k - 1); return a <= 0 ? 0 : (a + s - 1) / s; };
    auto hi = [&](int v, int O) { int b = (v + p) / s; return b < O - 1 ? b : O - 1; };
    const int d0 = lo(id), d1 = hi(id, Do), h0 = lo(ih), h1 = hi(ih, Ho), w0 = lo(iw),
              w1 = hi(iw, Wo);
    const int64_t obase = nc * Do * Ho * Wo;
    float acc = accumulate ? Elt<T>::ld(dx + i) : 0.f;
    float sum = 0.f;
    for (int od = d0; od <= d1; ++od)
        for (int oh = h0; oh <= h1; ++oh)
            for (int ow = w0; ow <= w1; ++ow) {
                const int64_t o = obase + ((int64_t)od * Ho + oh) * Wo + ow;
                const int off = ((id - od * s + p) * k + (ih - oh * s + p)) * k + (iw - ow * s + p);
                if ((int)am[o] == off) sum += Elt<T>::ld(dy + o);
            }
    Elt<T>::st(dx + i, acc + sum);
}

// ---------------------------------------------------------------- trilinear
// Axis map of half-pixel resampling: src = (o + 1/2) * in/out - 1/2,
// clamped below at 0; i0 = floor(src), i1 = min(i0 + 1, in - 1),
// lam = src - i0.  Forward and backward call this same function.
__device__ __forceinline__ void lin_src(int o, int in, float scale, int& i0, int& i1,
                                        float& lam) {
    float src = __fmaf_rn((float)o + 0.5f, scale, -0.5f);
    if (src < 0.f) src = 0.f;
    int a = (int)floorf(src);
    if (a > in - 1) a = in - 1;
    i0 = a;
    i1 = a + 1 < in ? a + 1 : in - 1;
    lam = src - (float)a;
}

template <typename T>
__global__ __launch_bounds__(kEwThreads) void up_fwd_k(const T* __restrict__ x, int NC, int Di,
                                                       int Hi, int Wi, int Do, int Ho, int Wo,
                                                       float sd, float sh, float sw,
                                                       T* __restrict__ y) {
    const int64_t o = (int64_t)blockIdx.x * kEwThreads + threadIdx.x;
    const int64_t total = (int64_t)NC * Do * Ho * Wo;
    if (o >= total) return;
    const int ow = (int)(o % Wo);
    const int oh = (int)((o / Wo) % Ho);
    const int od = (int)((o / ((int64_t)Wo * Ho)) % Do);
    const int64_t nc = o / ((int64_t)Wo * Ho * Do);
    int d0, d1, h0, h1, w0, w1;
    float ld, lh, lw;
    lin_src(od, Di, sd, d0, d1, ld);
    lin_src(oh, Hi, sh, h0, h1, lh);
    lin_src(ow, Wi, sw, w0, w1, lw);
    const T* xp = x + nc * Di * Hi * Wi;
    auto at = [&](int d, int h, int w) { return Elt<T>::ld(xp + ((int64_t)d * Hi + h) * Wi + w); };
    const float c00 = at(d0, h0, w0) * (1.f - lw) + at(d0, h0, w1) * lw;
    const float c01 = at(d0, h1, w0) * (1.f - lw) + at(d0, h1, w1) * lw;
    const float c10 = at(d1, h0, w0) * (1.f - lw) + at(d1, h0, w1) * lw;
    const float c11 = at(d1, h1, w0) * (1.f - lw) + at(d1, h1, w1) * lw;
    const float c0 = c00 * (1.f - lh) + c01 * lh;
    const float c1 = c10 * (1.f - lh) + c11 * lh;
    Elt<T>::st(y + o, c0 * (1.f - ld) + c1 * ld);
}

// Outputs along one axis that read input index i, with their weights.
struct AxisTaps {
    int o[8];
    float w[8];
    int n;
};

__device__ __forceinline__ void axis_taps(int i, int in, int out, float scale, AxisTaps& t) {
    // src(o) in (i - 1, i + 1) <=> o in ((i - 1/2)/scale - 1/2, (i + 3/2)/scale - 1/2)
    int a = (int)floorf(((float)i - 0.5f) / scale - 0.5f) - 1;
    int b = (int)ceilf(((float)i + 1.5f) / scale - 0.5f) + 1;
    if (a < 0) a = 0;
    if (b > out - 1) b = out - 1;
    t.n = 0;
    for (int o = a; o <= b && t.n < 8; ++o) {
        int i0, i1;
        float lam;
        lin_src(o, in, scale, i0, i1, lam);
        float wt = 0.f;
        if (i0 == i) wt += 1.f - lam;
        if (i1 == i) wt += lam;
        if (i0 == i || i1 == i) {
            t.o[t.n] = o;
            t.w[t.n] = wt;
            ++t.n;
        }
    }
}

template <typename T>
__global__ __launch_bounds__(kEwThreads) void up_bwd_k(const T* __restrict__ dy, int NC, int Di,
                                                       int Hi, int Wi, int Do, int Ho, int Wo,
                                                       float sd, float sh, float sw,
                                                       T* __restrict__ dx, int accumulate) {
    const int64_t i = (int64_t)blockIdx.x * kEwThreads + threadIdx.x;
    const int64_t total = (int64_t)NC * Di * Hi * Wi;
    if (i >= total) return;
    const int iw = (int)(i % Wi);
    const int ih = (int)((i / Wi) % Hi);
    const int id = (int)((i / ((int64_t)Wi * Hi)) % Di);
    const int64_t nc = i / ((int64_t)Wi * Hi * Di);
    AxisTaps td, th, tw;
    axis_taps(id, Di, Do, sd, td);
    axis_taps(ih, Hi, Ho, sh, th);
    axis_taps(iw, Wi, Wo, sw, tw);
    const T* g = dy + nc * Do * Ho * Wo;
    float sum = 0.f;
    for (int a = 0; a < td.n; ++a)
        for (int b = 0; b < th.n; ++b) {
            const T* row = g + ((int64_t)td.o[a] * Ho + th.o[b]) * Wo;
            float r = 0.f;
            for (int c = 0; c < tw.n; ++c) r += tw.w[c] * Elt<T>::ld(row + tw.o[c]);
            sum += td.w[a] * th.w[b] * r;
        }
    const float base = accumulate ? Elt<T>::ld(dx + i) : 0.f;
    Elt<T>::st(dx + i, base + sum);
}

// ---------------------------------------------------------------- sigmoid fuse

template <typename T, int VEC>
__global__ __launch_bounds__(kEwThreads) void softmask_fwd_k(const T* __restrict__ z,
                                                             const T* __restrict__ t,
                                                             int64_t count, T* __restrict__ out,
                                                             T* __restrict__ m) {
    const int64_t i = ((int64_t)blockIdx.x * kEwThreads + threadIdx.x) * VEC;
    if (i >= count) return;
    float zv[VEC], tv[VEC];
    vload<T, VEC>(z + i, zv);
    vload<T, VEC>(t + i, tv);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        const float mm = sigmoidf(zv[j]);
        zv[j] = mm;
        tv[j] = (1.f + mm) * tv[j];
    }
    vstore<T, VEC>(out + i, tv);
    if (m) vstore<T, VEC>(m + i, zv);
}

// Optional per-channel sums of the stored dz (the bias gradient of the conv
// that produced z): one partial per block at part[c][n * chunks + chunk],
// chunks = V / (block elements); needs V to be a multiple of a block's
// elements.
struct SmBias {
    float* part;
    int64_t V;
    int C, N;
};

// One vector of the soft-mask backward; returns the sum of the stored dz.
template <typename T, int VEC>
__device__ __forceinline__ float softmask_bwd_body(const T* __restrict__ dout,
                                                   const T* __restrict__ t,
                                                   const T* __restrict__ m, int64_t i,
                                                   T* __restrict__ dt, int accumulate_dt,
                                                   T* __restrict__ dz, int m_is_z) {
    float g[VEC], tv[VEC], mv[VEC], a[VEC], b[VEC];
    vload<T, VEC>(dout + i, g);
    vload<T, VEC>(t + i, tv);
    vload<T, VEC>(m + i, mv);
    if (accumulate_dt) vload<T, VEC>(dt + i, b);
    if (m_is_z) {
        // m was not stored: recompute it from z and round it as the forward's
        // store would have (same sigmoid, same rounding), so the bits match
#pragma unroll
        for (int j = 0; j < VEC; ++j) mv[j] = Elt<T>::round(sigmoidf(mv[j]));
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        a[j] = (1.f + mv[j]) * g[j];
        if (accumulate_dt) a[j] += b[j];
        b[j] = g[j] * tv[j] * mv[j] * (1.f - mv[j]);
    }
    vstore<T, VEC>(dt + i, a);
    vstore<T, VEC>(dz + i, b);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < VEC; ++j) s += Elt<T>::round(b[j]);
    return s;
}

template <typename T, int VEC>
__global__ __launch_bounds__(kEwThreads) void softmask_bwd_k(
    const T* __restrict__ dout, const T* __restrict__ t, const T* __restrict__ m, int64_t count,
    T* __restrict__ dt, int accumulate_dt, T* __restrict__ dz, int m_is_z, SmBias sb) {
    const int64_t i = ((int64_t)blockIdx.x * kEwThreads + threadIdx.x) * VEC;
    if (sb.part) {
        // the block's share of dz's per-channel sum (the bias gradient of the
        // conv that produced z), over the stored values; V is a multiple of
        // the block's elements, so a block lies in one (n, c) plane
        float s = 0.f;
        if (i < count) s = softmask_bwd_body<T, VEC>(dout, t, m, i, dt, accumulate_dt, dz, m_is_z);
#pragma unroll
        for (int w = 32; w >= 1; w >>= 1) s += __shfl_xor(s, w, 64);
        __shared__ float red[kEwThreads / 64];
        if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
        __syncthreads();
        if (threadIdx.x == 0) {
            float a = 0.f;
#pragma unroll
            for (int w = 0; w < kEwThreads / 64; ++w) a += red[w];
            const int64_t e0 = (int64_t)blockIdx.x * kEwThreads * VEC;
            const int64_t plane = e0 / sb.V, chunk = (e0 - plane * sb.V) / (kEwThreads * VEC);
            const int64_t chunks = sb.V / (kEwThreads * VEC);
            const int64_t n = plane / sb.C, c = plane - n * sb.C;
            sb.part[c * (sb.N * chunks) + n * chunks + chunk] = a;
        }
        return;
    }
    if (i >= count) return;
    softmask_bwd_body<T, VEC>(dout, t, m, i, dt, accumulate_dt, dz, m_is_z);
}

template <typename T, int VEC>
__global__ __launch_bounds__(kEwThreads) void add_k(const T* __restrict__ a,
                                                    const T* __restrict__ b, int64_t count,
                                                    T* __restrict__ dst) {
    const int64_t i = ((int64_t)blockIdx.x * kEwThreads + threadIdx.x) * VEC;
    if (i >= count) return;
    float x[VEC], y[VEC];
    vload<T, VEC>(a + i, x);
    vload<T, VEC>(b + i, y);
#pragma unroll
    for (int j = 0; j < VEC; ++j) x[j] += y[j];
    vstore<T, VEC>(dst + i, x);
}

// ---------------------------------------------------------------- fast paths
// Grids are (plane chunk, n*c*depth): one block row per output (or input)
// depth plane, so in-plane indices need only 32-bit arithmetic.

// Max pool 3^3, stride 2, pad 1: the common case, same scan order and
// first-maximum rule as pool_fwd_k.
template <typename T>
__global__ __launch_bounds__(kEwThreads) void pool332_fwd_k(const T* __restrict__ x, int D,
                                                            int H, int W, int Do, int Ho, int Wo,
                                                            T* __restrict__ y,
                                                            uint8_t* __restrict__ am) {
    const int t = blockIdx.x * kEwThreads + threadIdx.x;
    if (t >= Ho * Wo) return;
    const int oh = t / Wo, ow = t - oh * Wo;
    const int plane = blockIdx.y;  // nc * Do + od
    const int nc = plane / Do, od = plane - nc * Do;
    const T* xp = x + (int64_t)nc * D * H * W;
    float best = 0.f;
    int arg = -1;
#pragma unroll
    for (int kd = 0; kd < 3; ++kd) {
        const int id = 2 * od - 1 + kd;
        if ((unsigned)id >= (unsigned)D) continue;
#pragma unroll
        for (int kh = 0; kh < 3; ++kh) {
            const int ih = 2 * oh - 1 + kh;
            if ((unsigned)ih >= (unsigned)H) continue;
            const T* row = xp + ((int64_t)id * H + ih) * W;
#pragma unroll
            for (int kw = 0; kw < 3; ++kw) {
                const int iw = 2 * ow - 1 + kw;
                if ((unsigned)iw >= (unsigned)W) continue;
                const float v = Elt<T>::ld(row + iw);
                if (arg < 0 || v > best) {
                    best = v;
                    arg = (kd * 3 + kh) * 3 + kw;
                }
            }
        }
    }
    const int64_t o = (int64_t)plane * Ho * Wo + t;
    Elt<T>::st(y + o, best);
    am[o] = (uint8_t)arg;
}

// Windows (3^3, stride 2, pad 1) containing input index i along one axis:
// even i -> window i/2 (tap 1); odd i -> windows (i-1)/2 (tap 2) and
// (i+1)/2 (tap 0), each only if inside [0, O).
__device__ __forceinline__ int pool332_windows(int i, int O, int (&o)[2], int (&tap)[2]) {
    if ((i & 1) == 0) {
        o[0] = i >> 1;
        tap[0] = 1;
        return o[0] < O ? 1 : 0;
    }
    int n = 0;
    if (((i - 1) >> 1) < O) { o[n] = (i - 1) >> 1; tap[n] = 2; ++n; }
    if (((i + 1) >> 1) < O) { o[n] = (i + 1) >> 1; tap[n] = 0; ++n; }
    return n;
}

template <typename T>
__global__ __launch_bounds__(kEwThreads) void pool332_bwd_k(const T* __restrict__ dy,
                                                            const uint8_t* __restrict__ am,
                                                            int D, int H, int W, int Do, int Ho,
                                                            int Wo, T* __restrict__ dx,
                                                            int accumulate) {
    const int t = blockIdx.x * kEwThreads + threadIdx.x;
    if (t >= H * W) return;
    const int ih = t / W, iw = t - ih * W;
    const int plane = blockIdx.y;  // nc * D + id
    const int nc = plane / D, id = plane - nc * D;
    int od[2], td[2], oh[2], th[2], ow[2], tw[2];
    const int nd = pool332_windows(id, Do, od, td);
    const int nh = pool332_windows(ih, Ho, oh, th);
    const int nw = pool332_windows(iw, Wo, ow, tw);
    const int64_t ob = (int64_t)nc * Do * Ho * Wo;
    float sum = 0.f;
    for (int a = 0; a < nd; ++a)
        for (int b = 0; b < nh; ++b) {
            const int64_t rb = ob + ((int64_t)od[a] * Ho + oh[b]) * Wo;
            for (int c = 0; c < nw; ++c) {
                const int off = (td[a] * 3 + th[b]) * 3 + tw[c];
                if ((int)am[rb + ow[c]] == off) sum += Elt<T>::ld(dy + rb + ow[c]);
            }
        }
    const int64_t i = (int64_t)plane * H * W + t;
    const float base = accumulate ? Elt<T>::ld(dx + i) : 0.f;
    Elt<T>::st(dx + i, base + sum);
}

// Trilinear with per-axis tables built once per block in LDS.  Axes longer
// than kAxisMax use the generic kernels.
constexpr int kAxisMax = 256;

template <typename T>
__global__ __launch_bounds__(kEwThreads) void up_fwd_tab_k(const T* __restrict__ x, int Di,
                                                           int Hi, int Wi, int Do, int Ho, int Wo,
                                                           float sd, float sh, float sw,
                                                           T* __restrict__ y) {
    __shared__ int h0s[kAxisMax], h1s[kAxisMax], w0s[kAxisMax], w1s[kAxisMax];
    __shared__ float lhs[kAxisMax], lws[kAxisMax];
    for (int i = threadIdx.x; i < Ho; i += kEwThreads) lin_src(i, Hi, sh, h0s[i], h1s[i], lhs[i]);
    for (int i = threadIdx.x; i < Wo; i += kEwThreads) lin_src(i, Wi, sw, w0s[i], w1s[i], lws[i]);
    __syncthreads();
    const int t = blockIdx.x * kEwThreads + threadIdx.x;
    if (t >= Ho * Wo) return;
    const int oh = t / Wo, ow = t - oh * Wo;
    const int plane = blockIdx.y;  // nc * Do + od
    const int nc = plane / Do, od = plane - nc * Do;
    int d0, d1;
    float ld;
    lin_src(od, Di, sd, d0, d1, ld);
    const int h0 = h0s[oh], h1 = h1s[oh], w0 = w0s[ow], w1 = w1s[ow];
    const float lh = lhs[oh], lw = lws[ow];
    const T* xp = x + (int64_t)nc * Di * Hi * Wi;
    auto at = [&](int d, int h, int w) { return Elt<T>::ld(xp + ((int64_t)d * Hi + h) * Wi + w); };
    const float c00 = at(d0, h0, w0) * (1.f - lw) + at(d0, h0, w1) * lw;
    const float c01 = at(d0, h1, w0) * (1.f - lw) + at(d0, h1, w1) * lw;
    const float c10 = at(d1, h0, w0) * (1.f - lw) + at(d1, h0, w1) * lw;
    const float c11 = at(d1, h1, w0) * (1.f - lw) + at(d1, h1, w1) * lw;
    const float c0 = c00 * (1.f - lh) + c01 * lh;
    const float c1 = c10 * (1.f - lh) + c11 * lh;
    Elt<T>::st(y + (int64_t)plane * Ho * Wo + t, c0 * (1.f - ld) + c1 * ld);
}

// Transpose of the trilinear resampling with per-axis tap tables: every
// block builds the tables of the three axes in LDS (an input index's output
// positions and weights), then each thread forms one input voxel's gradient.
template <typename T>
__global__ __launch_bounds__(kEwThreads) void up_bwd_tab_k(const T* __restrict__ dy, int NC,
                                                           int Di, int Hi, int Wi, int Do, int Ho,
                                                           int Wo, float sd, float sh, float sw,
                                                           T* __restrict__ dx, int accumulate) {
    extern __shared__ AxisTaps tabs[];  // [Di + Hi + Wi]
    AxisTaps* dts = tabs;
    AxisTaps* hts = tabs + Di;
    AxisTaps* wts = hts + Hi;
    for (int i = threadIdx.x; i < Di + Hi + Wi; i += kEwThreads) {
        if (i < Di)
            axis_taps(i, Di, Do, sd, dts[i]);
        else if (i < Di + Hi)
            axis_taps(i - Di, Hi, Ho, sh, hts[i - Di]);
        else
            axis_taps(i - Di - Hi, Wi, Wo, sw, wts[i - Di - Hi]);
    }
    __syncthreads();
    const int64_t t = (int64_t)blockIdx.x * kEwThreads + threadIdx.x;
    if (t >= (int64_t)NC * Di * Hi * Wi) return;
    const int iw = (int)(t % Wi), ih = (int)((t / Wi) % Hi), id = (int)((t / ((int64_t)Wi * Hi)) % Di);
    const int64_t nc = t / ((int64_t)Wi * Hi * Di);
    const AxisTaps& td = dts[id];
    const AxisTaps& th = hts[ih];
    const AxisTaps& tw = wts[iw];
    const T* g = dy + nc * Do * Ho * Wo;
    float sum = 0.f;
    for (int a = 0; a < td.n; ++a)
        for (int b = 0; b < th.n; ++b) {
            const T* row = g + ((int64_t)td.o[a] * Ho + th.o[b]) * Wo;
            float r = 0.f;
            for (int c = 0; c < tw.n; ++c) r += tw.w[c] * Elt<T>::ld(row + tw.o[c]);
            sum += td.w[a] * th.w[b] * r;
        }
    const float base = accumulate ? Elt<T>::ld(dx + t) : 0.f;
    Elt<T>::st(dx + t, base + sum);
}

// ---------------------------------------------------------------- exact x2, bf16
// When every axis doubles (out = 2 * in), the half-pixel weights are 1/4 and
// 3/4 exactly: fine o = 2m takes 1/4 c[m-1] + 3/4 c[m] (c[0] alone at m = 0),
// o = 2m + 1 takes 3/4 c[m] + 1/4 c[m+1] (c[m] alone at the last m).  The
// transpose gives coarse i 1/4 f[2i-1] + 3/4 f[2i] + 3/4 f[2i+1] + 1/4 f[2i+2]
// with the border terms folded the same way.  These are the same weights the
// general kernels compute, applied separably.

// Weight of coarse index m for fine index o along one doubled axis of coarse
// length n (0 if o does not read m).
__device__ __forceinline__ float x2_w(int o, int m, int n) {
    const int half = o >> 1;
    if ((o & 1) == 0) {  // 1/4 c[half-1] + 3/4 c[half]
        if (half == 0) return m == 0 ? 1.f : 0.f;
        return m == half ? 0.75f : (m == half - 1 ? 0.25f : 0.f);
    }
    if (half == n - 1) return m == half ? 1.f : 0.f;  // 3/4 c[half] + 1/4 c[half+1]
    return m == half ? 0.75f : (m == half + 1 ? 0.25f : 0.f);
}

// ---------------------------------------------------------------- plane-staged fast paths
// bfloat16 pooling and exact x2 upsampling.  A block owns a few consecutive
// depth planes of one (n, c) volume.  Phase A streams the source planes it
// needs with 16-byte loads (each source element read once per block) and
// reduces them along depth into LDS; phase B finishes the in-plane stencil
// from LDS and writes whole 8- or 4-element groups.  Neighbouring blocks
// share at most one or two halo planes; the XCD-aware block order keeps
// them in the same L2.

constexpr int kPlanes = 2;           // destination depth planes per block (pool gradient)
constexpr int kPlanesF = 2;          // output depth planes per block (pool forward)
constexpr size_t kPlaneLds = 65536;  // dynamic LDS limit of the staged kernels

// 8 consecutive elements p .. p+7 of a plane of n elements (p % 8 == 0);
// elements at or past n read as 0.  vec: n % 8 == 0 (16-byte aligned rows).
__device__ __forceinline__ void ld8(const bf16* __restrict__ plane, int p, int n, bool vec,
                                    float (&v)[8]) {
    if (vec) {
        const uint4 u = *reinterpret_cast<const uint4*>(plane + p);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = p + e < n ? bf2f(plane[p + e]) : 0.f;
    }
}

// Order-preserving key of a bfloat16 value (upper half) and a window tap:
// the unsigned maximum of keys is the largest value and, among equal values,
// the smallest scan index (the low byte holds 255 - index).  Signed zeros
// map to one key, as they compare equal.
__device__ __forceinline__ uint32_t pool_key_hi(uint32_t bits) {
    bits &= 0xffffu;
    if (bits == 0x8000u) bits = 0u;
    return ((bits & 0x8000u) ? (~bits & 0xffffu) : (bits | 0x8000u)) << 16;
}
__device__ __forceinline__ float pool_key_value(uint32_t key) {
    const uint32_t o = key >> 16;
    const uint32_t bits = (o & 0x8000u) ? (o & 0x7fffu) : (~o & 0xffffu);
    return __uint_as_float(bits << 16);
}

// Max pool 3^3, stride 2, pad 1, bf16, as maxima of order-preserving keys
// (value, then the first tap in (kd, kh, kw) scan order, as in pool_fwd_k).
// Phase A: per input (h, w) and output plane, the maximum key over the depth
// taps (low byte 255 - 9 kd), kept in LDS.  Phase B: the 3 x 3 in-plane
// window, each tap's key lowered by kh * 3 + kw; with Wo % 4 == 0 a thread
// forms four outputs of a row from the 3 x 9 keys their windows share.
__global__ __launch_bounds__(kEwThreads) void pool332_fwd_pl(const bf16* __restrict__ x, int D,
                                                             int H, int W, int Do, int Ho, int Wo,
                                                             int nblk, bf16* __restrict__ y,
                                                             uint8_t* __restrict__ am) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int HW = H * W, HW8 = (HW + 7) & ~7;
    uint32_t* mk = reinterpret_cast<uint32_t*>(smem);  // [kPlanesF][HW8] keys
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int nc = L / nblk, od0 = (L - nc * nblk) * kPlanesF;
    const bool vec = (HW & 7) == 0;
    const bf16* xv = x + (int64_t)nc * D * HW;
    for (int p = threadIdx.x * 8; p < HW; p += kEwThreads * 8) {
        uint32_t best[kPlanesF][8];
#pragma unroll
        for (int j = 0; j < kPlanesF; ++j)
#pragma unroll
            for (int e = 0; e < 8; ++e) best[j][e] = 0u;
        // all source planes are requested before any is used (clamped plane
        // index, so no load waits behind a branch)
        constexpr int NQ = 2 * kPlanesF + 1;
        uint4 raw[NQ];
        if (vec) {
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int id = min(max(2 * od0 - 1 + q, 0), D - 1);
                raw[q] = *reinterpret_cast<const uint4*>(xv + (int64_t)id * HW + p);
            }
        }
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int id = 2 * od0 - 1 + q;
            if (id < 0 || id >= D) continue;
            uint32_t kv[8];
            if (vec) {
                const uint32_t w[4] = {raw[q].x, raw[q].y, raw[q].z, raw[q].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    kv[2 * i] = pool_key_hi(w[i]);
                    kv[2 * i + 1] = pool_key_hi(w[i] >> 16);
                }
            } else {
                const bf16* pl = xv + (int64_t)id * HW;
#pragma unroll
                for (int e = 0; e < 8; ++e) kv[e] = p + e < HW ? pool_key_hi(pl[p + e]) : 0u;
            }
#pragma unroll
            for (int j = 0; j < kPlanesF; ++j) {
                const int kd = q - 2 * j;
                if (kd < 0 || kd > 2) continue;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    best[j][e] = max(best[j][e], kv[e] | (uint32_t)(255 - 9 * kd));
            }
        }
#pragma unroll
        for (int j = 0; j < kPlanesF; ++j) {
            uint4* dst = reinterpret_cast<uint4*>(mk + j * HW8 + p);
            dst[0] = make_uint4(best[j][0], best[j][1], best[j][2], best[j][3]);
            dst[1] = make_uint4(best[j][4], best[j][5], best[j][6], best[j][7]);
        }
    }
    __syncthreads();
    const int HWo = Ho * Wo;
    if ((Wo & 3) == 0) {
        const int Q = Wo >> 2, HQ = Ho * Q;
        for (int it = threadIdx.x; it < kPlanesF * HQ; it += kEwThreads) {
            const int j = it / HQ, r = it - j * HQ;
            const int od = od0 + j;
            if (od >= Do) break;
            const int oh = r / Q, ow0 = (r - oh * Q) * 4;
            uint32_t b[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int kh = 0; kh < 3; ++kh) {
                const int ih = 2 * oh - 1 + kh;
                if ((unsigned)ih >= (unsigned)H) continue;
                // columns 2 * ow0 - 1 .. 2 * ow0 + 7: tap kw of output e is c = 2e + kw;
                // a padding column keeps key 0, below every value
                const uint32_t* row = mk + j * HW8 + ih * W;
                uint32_t cw[9];
#pragma unroll
                for (int c = 0; c < 9; ++c) {
                    const int iw = 2 * ow0 - 1 + c;
                    cw[c] = (unsigned)iw < (unsigned)W ? row[iw] : 0u;
                }
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int kw = 0; kw < 3; ++kw) {
                        const uint32_t k = cw[2 * e + kw];
                        b[e] = max(b[e], k ? k - (uint32_t)(kh * 3 + kw) : 0u);
                    }
            }
            const int64_t o = ((int64_t)nc * Do + od) * HWo + oh * Wo + ow0;
            *reinterpret_cast<uint2*>(y + o) = make_uint2(
                pack_bf16x2(pool_key_value(b[0]), pool_key_value(b[1])),
                pack_bf16x2(pool_key_value(b[2]), pool_key_value(b[3])));
            *reinterpret_cast<uint32_t*>(am + o) =
                (255u - (b[0] & 0xffu)) | (255u - (b[1] & 0xffu)) << 8 |
                (255u - (b[2] & 0xffu)) << 16 | (255u - (b[3] & 0xffu)) << 24;
        }
        return;
    }
    for (int it = threadIdx.x; it < kPlanesF * HWo; it += kEwThreads) {
        const int j = it / HWo, r = it - j * HWo;
        const int od = od0 + j;
        if (od >= Do) break;
        const int oh = r / Wo, ow = r - oh * Wo;
        uint32_t b = 0u;
#pragma unroll
        for (int kh = 0; kh < 3; ++kh) {
            const int ih = 2 * oh - 1 + kh;
            if ((unsigned)ih >= (unsigned)H) continue;
#pragma unroll
            for (int kw = 0; kw < 3; ++kw) {
                const int iw = 2 * ow - 1 + kw;
                if ((unsigned)iw >= (unsigned)W) continue;
                b = max(b, mk[j * HW8 + ih * W + iw] - (uint32_t)(kh * 3 + kw));
            }
        }
        const int64_t o = ((int64_t)nc * Do + od) * HWo + r;
        y[o] = f2bf(pool_key_value(b));
        am[o] = (uint8_t)(255u - (b & 0xffu));
    }
}

// Order-preserving 16-bit codes of the two bfloat16 halves of a word: a
// value with the sign bit clear maps to v ^ 0x8000, one with it set to
// (v ^ 0xffff) + 1.  Codes order like the values, -0 and +0 share 0x8000
// (they compare equal) and every code is at least 1.  Packed 16-bit integer
// operations: the sign mask by an arithmetic shift, one xor, one subtract.
typedef __attribute__((ext_vector_type(2))) short pool_s16x2;
typedef __attribute__((ext_vector_type(2))) unsigned short pool_u16x2;
__device__ __forceinline__ uint32_t pool_codes2(uint32_t w) {
    const uint32_t m = __builtin_bit_cast(uint32_t, __builtin_bit_cast(pool_s16x2, w) >> 15);
    const uint32_t x = w ^ (m | 0x80008000u);
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(pool_u16x2, x) -
                                            __builtin_bit_cast(pool_u16x2, m));
}
// bf16 bits of a code (low 16 bits of c)
__device__ __forceinline__ uint32_t pool_code_bits(uint32_t c) {
    return (c & 0x8000u) ? (c & 0x7fffu) : (0x8000u | (0x8000u - c));
}
// Key of a padding column: below every value's key (those are at least
// 1 << 16) and still non-negative after the largest tap offset is taken off.
constexpr uint32_t kPoolPadKey = 8u;

// Max pool 3^3, stride 2, pad 1, bf16, W % 8 == 0 (so every 8-element group
// lies in one row and Wo % 4 == 0).  Keys as in pool332_fwd_pl: the 16-bit
// code of the value above 255 - (9 kd + 3 kh + kw), so the unsigned maximum
// is the first maximum in scan order together with its index.  The LDS key
// rows are padded: column iw at 4 + iw, a padding key at 3, so phase B reads
// the nine columns 2 ow0 - 1 .. 2 ow0 + 7 of four outputs with two aligned
// 16-byte reads and one 4-byte read, without bounds checks.  Phase B reduces
// each row over kw first (max3), then over kh.
__global__ __launch_bounds__(kEwThreads) void pool332_fwd_rows(const bf16* __restrict__ x, int D,
                                                               int H, int W, int Do, int Ho,
                                                               int Wo, int nblk,
                                                               bf16* __restrict__ y,
                                                               uint8_t* __restrict__ am) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int HW = H * W, RP = W + 4, PP = H * RP;
    uint32_t* mk = reinterpret_cast<uint32_t*>(smem);  // [kPlanesF][H][RP] keys
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int nc = L / nblk, od0 = (L - nc * nblk) * kPlanesF;
    const bf16* xv = x + (int64_t)nc * D * HW;
    constexpr int NQ = 2 * kPlanesF + 1;
    auto process = [&](int p, const uint4 (&raw)[NQ]) {
        const int ih = p / W, iw0 = p - ih * W;
        uint32_t best[kPlanesF][8];
#pragma unroll
        for (int j = 0; j < kPlanesF; ++j)
#pragma unroll
            for (int e = 0; e < 8; ++e) best[j][e] = 0u;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int id = 2 * od0 - 1 + q;
            if (id < 0 || id >= D) continue;
            const uint32_t c[4] = {pool_codes2(raw[q].x), pool_codes2(raw[q].y),
                                   pool_codes2(raw[q].z), pool_codes2(raw[q].w)};
#pragma unroll
            for (int j = 0; j < kPlanesF; ++j) {
                const int kd = q - 2 * j;
                if (kd < 0 || kd > 2) continue;
                const uint32_t tb = 255u - 9u * (uint32_t)kd;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    best[j][2 * i] = max(best[j][2 * i], (c[i] << 16) | tb);
                    best[j][2 * i + 1] = max(best[j][2 * i + 1], (c[i] & 0xffff0000u) | tb);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < kPlanesF; ++j) {
            uint32_t* row = mk + j * PP + ih * RP;
            uint4* dst = reinterpret_cast<uint4*>(row + 4 + iw0);
            dst[0] = make_uint4(best[j][0], best[j][1], best[j][2], best[j][3]);
            dst[1] = make_uint4(best[j][4], best[j][5], best[j][6], best[j][7]);
            if (iw0 == 0) row[3] = kPoolPadKey;
        }
    };
    auto fetch = [&](int p, uint4 (&raw)[NQ]) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int id = min(max(2 * od0 - 1 + q, 0), D - 1);
            raw[q] = *reinterpret_cast<const uint4*>(xv + (int64_t)id * HW + p);
        }
    };
    // both 8-element groups of a thread (a 48 x 56 plane has 336) are
    // requested before either is reduced
    {
        const int p0 = threadIdx.x * 8, p1 = p0 + kEwThreads * 8;
        uint4 r0[NQ], r1[NQ];
        if (p0 < HW) fetch(p0, r0);
        if (p1 < HW) fetch(p1, r1);
        if (p0 < HW) process(p0, r0);
        if (p1 < HW) process(p1, r1);
        for (int p = p1 + kEwThreads * 8; p < HW; p += kEwThreads * 8) {
            fetch(p, r0);
            process(p, r0);
        }
    }
    __syncthreads();
    // items it = tid, tid + 256, ... of the flattened (j, oh, q) range, the
    // indices stepped incrementally (no per-item division), 32-bit offsets
    const int Q = Wo >> 2, HQ = Ho * Q;
    const int jmax = min(kPlanesF, Do - od0);
    const int dq = kEwThreads / Q, dr = kEwThreads - dq * Q;
    int j = (int)threadIdx.x / HQ, oh, q;
    {
        const int r0 = (int)threadIdx.x - j * HQ;
        oh = r0 / Q;
        q = r0 - oh * Q;
    }
    bf16* yb = y + ((int64_t)nc * Do + od0) * (int64_t)(Ho * Wo);
    uint8_t* ab = am + ((int64_t)nc * Do + od0) * (int64_t)(Ho * Wo);
    for (; j < jmax;) {
        const int ow0 = 4 * q;
        uint32_t b[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int kh = 0; kh < 3; ++kh) {
            const int ih = 2 * oh - 1 + kh;
            if ((unsigned)ih >= (unsigned)H) continue;
            // columns 2 ow0 - 1 .. 2 ow0 + 7: tap kw of output e is column 2e + kw
            const uint32_t* row = mk + __mul24(j, PP) + __mul24(ih, RP) + 3 + 2 * ow0;
            const uint4 lo = *reinterpret_cast<const uint4*>(row + 1);
            const uint4 hi = *reinterpret_cast<const uint4*>(row + 5);
            const uint32_t cw[9] = {row[0], lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
            const uint32_t toff = 3u * (uint32_t)kh;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t m = max(max(cw[2 * e], cw[2 * e + 1] - 1u), cw[2 * e + 2] - 2u);
                b[e] = max(b[e], m - toff);
            }
        }
        const int o = __mul24(j, Ho * Wo) + __mul24(oh, Wo) + ow0;
        *reinterpret_cast<uint2*>(yb + o) =
            make_uint2(pool_code_bits(b[0] >> 16) | pool_code_bits(b[1] >> 16) << 16,
                       pool_code_bits(b[2] >> 16) | pool_code_bits(b[3] >> 16) << 16);
        *reinterpret_cast<uint32_t*>(ab + o) =
            (255u - (b[0] & 0xffu)) | (255u - (b[1] & 0xffu)) << 8 |
            (255u - (b[2] & 0xffu)) << 16 | (255u - (b[3] & 0xffu)) << 24;
        oh += dq;
        q += dr;
        if (q >= Q) {
            q -= Q;
            ++oh;
        }
        while (oh >= Ho) {
            oh -= Ho;
            ++j;
        }
    }
}

// Max-pool gradient (3^3, stride 2, pad 1), bf16, W % 8 == 0.  A block owns
// input planes 2*j0 .. 2*j0 + 2*kPlanes - 1, whose windows lie in output
// planes j0 .. j0 + kPlanes; their dy and argmax are staged in LDS, then
// each thread gathers 8 consecutive input voxels of a row.
__global__ __launch_bounds__(kEwThreads) void pool332_bwd_pl(const bf16* __restrict__ dy,
                                                             const uint8_t* __restrict__ am, int D,
                                                             int H, int W, int Do, int Ho, int Wo,
                                                             int nblk, bf16* __restrict__ dx,
                                                             int accumulate) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int NP = kPlanes + 1;
    const int HWo = Ho * Wo;
    bf16* sdy = reinterpret_cast<bf16*>(smem);                  // [NP][HWo]
    uint8_t* sam = smem + (size_t)NP * HWo * sizeof(bf16);      // [NP][HWo]
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int nc = L / nblk, j0 = (L - nc * nblk) * kPlanes;
    const int np = min(NP, Do - j0);
    const int64_t ob = ((int64_t)nc * Do + j0) * HWo;
    const int cnt = np * HWo;
    // dy and argmax of the block's output planes are one contiguous run each:
    // staged with 16-byte loads when the run and the LDS rows allow, every
    // load issued before the LDS writes
    const bool v_dy = (((uintptr_t)(dy + ob) | (uintptr_t)cnt * 2) & 15) == 0;
    const bool v_am = (((uintptr_t)(am + ob) | (uintptr_t)cnt | (uintptr_t)sam) & 15) == 0;
    if (v_dy && v_am) {
        const int ndy = cnt >> 3, nam = cnt >> 4;
        const uint4* gdy = reinterpret_cast<const uint4*>(dy + ob);
        const uint4* gam = reinterpret_cast<const uint4*>(am + ob);
        for (int i = threadIdx.x; i < ndy; i += kEwThreads) {
            const bool ha = i < nam;
            const uint4 d = gdy[i];
            const uint4 a = gam[ha ? i : 0];
            reinterpret_cast<uint4*>(sdy)[i] = d;
            if (ha) reinterpret_cast<uint4*>(sam)[i] = a;
        }
    } else {
        for (int i = threadIdx.x; i < cnt; i += kEwThreads) {
            sdy[i] = dy[ob + i];
            sam[i] = am[ob + i];
        }
    }
    __syncthreads();
    const int G = W >> 3;
    const int per_plane = H * G, ne = ((H + 1) >> 1) * G;  // items per plane, of even rows
    for (int it = threadIdx.x; it < 2 * kPlanes * per_plane; it += kEwThreads) {
        const int dl = it / per_plane;
        const int id = 2 * j0 + dl;
        if (id >= D) break;
        // even rows first, then odd rows, so a wave mostly shares the row
        // parity (and with it the number of h windows)
        int r = it - dl * per_plane, ih;
        if (r < ne) {
            ih = 2 * (r / G);
        } else {
            r -= ne;
            ih = 2 * (r / G) + 1;
        }
        const int g = r - (r / G) * G;
        const bool q4ok = 4 * g + 4 < Wo;  // the fifth window (ow = 4g + 4) exists
        float acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.f;
        // windows along an axis, in summation order: odd i -> (i-1)/2 with
        // tap 2, then (i+1)/2 with tap 0; even i -> i/2 with tap 1
        const int nd = (id & 1) ? 2 : 1, nh = (ih & 1) ? 2 : 1;
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            if (a >= nd) break;
            const int od = (id & 1) ? (id - 1 + 2 * a) >> 1 : id >> 1;
            const int td = (id & 1) ? 2 - 2 * a : 1;
            if (od >= Do) continue;
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                if (b >= nh) break;
                const int oh = (ih & 1) ? (ih - 1 + 2 * b) >> 1 : ih >> 1;
                const int th = (ih & 1) ? 2 - 2 * b : 1;
                if (oh >= Ho) continue;
                // windows ow = 4g .. 4g+4 of output row (od, oh): target column
                // within the group e = 2q - 1 + kw
                const int rb = ((od - j0) * Ho + oh) * Wo + 4 * g;
                const int ptap = td * 3 + th;
                const uint32_t am4 = *reinterpret_cast<const uint32_t*>(sam + rb);
                const uint2 dy4 = *reinterpret_cast<const uint2*>(sdy + rb);
                const int am_4 = sam[q4ok ? rb + 4 : rb];
                const float dy_4 = bf2f(sdy[q4ok ? rb + 4 : rb]);
#pragma unroll
                for (int q = 0; q < 5; ++q) {
                    const int arg = q < 4 ? (int)((am4 >> (8 * q)) & 0xffu) : am_4;
                    const uint32_t half = q < 2 ? dy4.x : dy4.y;
                    const float v = q == 4 ? dy_4
                                           : __uint_as_float((q & 1) ? (half & 0xffff0000u)
                                                                     : (half << 16));
                    const int row = arg / 3, kw = arg - row * 3;
                    const float vm = (row == ptap && (q < 4 || q4ok)) ? v : 0.f;
                    if (2 * q - 1 >= 0) acc[2 * q - 1 < 0 ? 0 : 2 * q - 1] += kw == 0 ? vm : 0.f;
                    if (2 * q <= 7) acc[2 * q > 7 ? 7 : 2 * q] += kw == 1 ? vm : 0.f;
                    if (2 * q + 1 <= 7) acc[2 * q + 1 > 7 ? 7 : 2 * q + 1] += kw == 2 ? vm : 0.f;
                }
            }
        }
        bf16* q = dx + (((int64_t)nc * D + id) * H + ih) * W + 8 * g;
        uint4* q4 = reinterpret_cast<uint4*>(q);
        if (accumulate) {
            const uint4 o = *q4;
            const uint32_t ws[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc[2 * i] += __uint_as_float(ws[i] << 16);
                acc[2 * i + 1] += __uint_as_float(ws[i] & 0xffff0000u);
            }
        }
        uint32_t w4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w4[i] = pack_bf16x2(acc[2 * i], acc[2 * i + 1]);
        *q4 = make_uint4(w4[0], w4[1], w4[2], w4[3]);
    }
}

// Max-pool gradient (3^3, stride 2, pad 1), bf16, W % 8 == 0, in scatter
// form through a float32 LDS tile.  A block owns input planes
// [2 j0, 2 j0 + 2 kp) of one (n, c) volume and reads the windows of output
// planes j0 .. j0 + kp (the last one only reaches the block's planes through
// its kd = 0 taps).  An item is a 2 x 2 group of windows of one output plane
// (rows 2i, 2i + 1, columns 2k, 2k + 1); each window adds its dy to the input
// voxel its argmax names, if the block owns it.  Windows whose (od, oh, ow)
// parities agree never overlap, so their targets are distinct: the block
// deposits the eight parity classes in eight steps separated by barriers,
// each a plain LDS read-add-write (a fixed order per voxel: deterministic).
// Then each thread rounds 8 consecutive voxels (after adding the old value
// when accumulating) and stores them with one 16-byte store.
constexpr int kScItems = 2;  // items per thread
__global__ __launch_bounds__(kEwThreads) void pool332_bwd_sc(const bf16* __restrict__ dy,
                                                             const uint8_t* __restrict__ am,
                                                             int D, int H, int W, int Do, int Ho,
                                                             int Wo, int kp, int nblk,
                                                             bf16* __restrict__ dx,
                                                             int accumulate) {
    extern __shared__ __align__(16) float tile[];  // [2 kp][H][W]
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int nc = L / nblk, j0 = (L - nc * nblk) * kp;
    const int np = min(2 * kp, D - 2 * j0);  // owned input planes
    const int HW = H * W;
    const int HI = (Ho + 1) >> 1, WK = Wo >> 1, per = HI * WK;
    const int nitems = min(kp + 1, Do - j0) * per;
    // every item's dy and argmax pairs requested first (Wo is even, so a pair
    // of columns 2k, 2k + 1 is one aligned 4-byte dy load and 2-byte argmax load)
    uint32_t dv[kScItems][2], av[kScItems][2];
    int odr[kScItems], ii[kScItems], kk[kScItems];
    const bf16* dyb = dy + ((int64_t)nc * Do + j0) * (int64_t)(Ho * Wo);
    const uint8_t* amb = am + ((int64_t)nc * Do + j0) * (int64_t)(Ho * Wo);
#pragma unroll
    for (int m = 0; m < kScItems; ++m) {
        const int it = threadIdx.x + m * kEwThreads;
        dv[m][0] = dv[m][1] = 0u;
        av[m][0] = av[m][1] = 0xffffu;  // no window: arguments past 26 deposit nothing
        odr[m] = -1;
        ii[m] = kk[m] = 0;
        if (it < nitems) {
            const int o = it / per, r = it - o * per;
            const int i = r / WK, k = r - i * WK;
            odr[m] = o;
            ii[m] = i;
            kk[m] = k;
            const int b = __mul24(o, Ho * Wo) + __mul24(2 * i, Wo) + 2 * k;
            dv[m][0] = *reinterpret_cast<const uint32_t*>(dyb + b);
            av[m][0] = *reinterpret_cast<const uint16_t*>(amb + b);
            if (2 * i + 1 < Ho) {
                dv[m][1] = *reinterpret_cast<const uint32_t*>(dyb + b + Wo);
                av[m][1] = *reinterpret_cast<const uint16_t*>(amb + b + Wo);
            }
        }
    }
    for (int e = threadIdx.x * 4; e < np * HW; e += kEwThreads * 4)
        *reinterpret_cast<float4*>(tile + e) = make_float4(0.f, 0.f, 0.f, 0.f);
    // target of each window in the tile (-1: none, or outside the block's planes)
    int tg[kScItems][2][2];
#pragma unroll
    for (int m = 0; m < kScItems; ++m)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const uint32_t arg = (av[m][b] >> (8 * c)) & 0xffu;
                // arg = 9 kd + 3 kh + kw, arg < 27
                const uint32_t kd = __umul24(arg, 57u) >> 9, r = arg - __umul24(9u, kd);
                const uint32_t kh = __umul24(r, 11u) >> 5, kw = r - __umul24(3u, kh);
                const int tp = 2 * odr[m] - 1 + (int)kd;  // plane, relative to 2 j0
                const int ih = 2 * (2 * ii[m] + b) - 1 + (int)kh;
                const int iw = 2 * (2 * kk[m] + c) - 1 + (int)kw;
                const bool ok = arg < 27u && (unsigned)tp < (unsigned)np &&
                                (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W;
                tg[m][b][c] = ok ? __mul24(tp, H * W) + __mul24(ih, W) + iw : -1;
            }
#pragma unroll
    for (int pd = 0; pd < 2; ++pd)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                __syncthreads();
#pragma unroll
                for (int m = 0; m < kScItems; ++m) {
                    const int t = tg[m][b][c];
                    if (t >= 0 && ((j0 + odr[m]) & 1) == pd) {
                        const uint32_t h = dv[m][b];
                        tile[t] += __uint_as_float(c ? (h & 0xffff0000u) : (h << 16));
                    }
                }
            }
    __syncthreads();
    bf16* out = dx + ((int64_t)nc * D + 2 * j0) * HW;
    for (int e = threadIdx.x * 8; e < np * HW; e += kEwThreads * 8) {
        const float4 s0 = *reinterpret_cast<const float4*>(tile + e);
        const float4 s1 = *reinterpret_cast<const float4*>(tile + e + 4);
        float acc[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        uint4* q4 = reinterpret_cast<uint4*>(out + e);
        if (accumulate) {
            const uint4 o = *q4;
            const uint32_t ws[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc[2 * i] += __uint_as_float(ws[i] << 16);
                acc[2 * i + 1] += __uint_as_float(ws[i] & 0xffff0000u);
            }
        }
        *q4 = make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                         pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
    }
}

// Output planes per block of the scatter-form pool gradient (0: not taken):
// the largest kp whose tile fits 24 KB and whose items fit the block.
static int pool_sc_kp(int D, int H, int W, int Do, int Ho, int Wo) {
    if (W % 8 != 0 || Wo % 2 != 0) return 0;
    const int64_t per = (int64_t)((Ho + 1) / 2) * (Wo / 2);
    int kp = (int)(24576 / ((int64_t)2 * H * W * 4));
    kp = min(kp, Do);
    while (kp >= 1 && (kp + 1) * per > (int64_t)kScItems * kEwThreads) --kp;
    (void)D;
    return kp < 1 ? 0 : kp;
}

// Exact x2 trilinear, bf16, Wi % 4 == 0.  A block owns fine planes
// 2*m0 .. 2*m0 + 2*kPlanes - 1.  Phase A blends coarse planes m0-1 .. m0+kPlanes
// along depth into LDS (float32); phase B blends rows and columns and writes
// 8 fine voxels of a row per item.
// With STATS, the block also sums (y - shift) and its square over the fine
// values it stores (as stored, bf16), shift = the first fine value of sample
// 0 of its channel (= the coarse value there), into the BN statistics
// partial (c, n * nblk + block): the statistics pass of a batch norm applied
// to y, without reading y again.
struct UpStats {
    float* part;  // [C][N * nblk] pairs, then the C shifts
    int C, N;
};

template <bool STATS>
__global__ __launch_bounds__(kEwThreads) void up2_fwd_pl(const bf16* __restrict__ x, int Di,
                                                         int Hi, int Wi, int nblk,
                                                         bf16* __restrict__ y, UpStats us) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int NF = 2 * kPlanes;
    const int HWi = Hi * Wi, HW8 = (HWi + 7) & ~7;
    float* t = reinterpret_cast<float*>(smem);  // [NF][HW8]
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int nc = L / nblk, m0 = (L - nc * nblk) * kPlanes;
    const int Do = 2 * Di, Ho = 2 * Hi, Wo = 2 * Wi;
    [[maybe_unused]] float s1 = 0.f, s2 = 0.f, shift = 0.f;
    if constexpr (STATS) shift = bf2f(x[(int64_t)(nc % us.C) * Di * Hi * Wi]);
    const bool vec = (HWi & 7) == 0;
    const bf16* xv = x + (int64_t)nc * Di * HWi;
    for (int p = threadIdx.x * 8; p < HWi; p += kEwThreads * 8) {
        float acc[NF][8];
#pragma unroll
        for (int l = 0; l < NF; ++l)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[l][e] = 0.f;
        // all coarse planes are requested before any is used (clamped plane
        // index, so no load waits behind a branch)
        constexpr int NQ = kPlanes + 2;
        uint4 raw[NQ];
        if (vec) {
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int md = min(max(m0 - 1 + q, 0), Di - 1);
                raw[q] = *reinterpret_cast<const uint4*>(xv + (int64_t)md * HWi + p);
            }
        }
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int md = m0 - 1 + q;
            if (md < 0 || md >= Di) continue;
            float v[8];
            if (vec) {
                const uint32_t w[4] = {raw[q].x, raw[q].y, raw[q].z, raw[q].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    v[2 * i] = __uint_as_float(w[i] << 16);
                    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
                }
            } else {
                ld8(xv + (int64_t)md * HWi, p, HWi, false, v);
            }
#pragma unroll
            for (int l = 0; l < NF; ++l) {
                const float wd = x2_w(2 * m0 + l, md, Di);
                if (wd != 0.f)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[l][e] += wd * v[e];
            }
        }
#pragma unroll
        for (int l = 0; l < NF; ++l) {
            float4* d4 = reinterpret_cast<float4*>(t + l * HW8 + p);
            d4[0] = make_float4(acc[l][0], acc[l][1], acc[l][2], acc[l][3]);
            d4[1] = make_float4(acc[l][4], acc[l][5], acc[l][6], acc[l][7]);
        }
    }
    __syncthreads();
    // an item is two fine rows 2 mh, 2 mh + 1 by 8 fine columns 8g .. 8g + 7:
    // they blend coarse rows mh - 1, mh, mh + 1 at coarse columns 4g - 1 ..
    // 4g + 4 (one 16-byte and two 4-byte LDS reads per row).  A border takes
    // its one existing neighbour with weight 1: its missing row or column is
    // read clamped and weighted 0.
    // Items it = tid, tid + 256, ... of the flattened (l, mh, g) range; the
    // indices step incrementally (no per-item division) and the offsets are
    // 32-bit products of small values (full-rate 24-bit multiplies).
    const int G = Wi >> 2, HG = Hi * G;
    const int lmax = min(NF, Do - 2 * m0);
    const int dq = kEwThreads / G, dr = kEwThreads - dq * G;
    int l = (int)threadIdx.x / HG, mh, g;
    {
        const int r0 = (int)threadIdx.x - l * HG;
        mh = r0 / G;
        g = r0 - mh * G;
    }
    bf16* yb = y + ((int64_t)nc * Do + 2 * m0) * Ho * Wo;
    for (; l < lmax;) {
        const float* tl = t + l * HW8;
        const int mhW = __mul24(mh, Wi);
        const int roff[3] = {mh > 0 ? mhW - Wi : mhW, mhW, mh < Hi - 1 ? mhW + Wi : mhW};
        const int cl = max(4 * g - 1, 0), cr = min(4 * g + 4, Wi - 1);
        float A[6], B[6], Dn[6];
        auto rd6 = [&](int ro, float (&v)[6]) {
            const float* q = tl + ro;
            const float4 m = *reinterpret_cast<const float4*>(q + 4 * g);
            v[0] = q[cl];
            v[1] = m.x;
            v[2] = m.y;
            v[3] = m.z;
            v[4] = m.w;
            v[5] = q[cr];
        };
        rd6(roff[0], A);
        rd6(roff[1], B);
        rd6(roff[2], Dn);
        // fine row 2 mh: 1/4 row mh-1 + 3/4 row mh; 2 mh + 1: 3/4 row mh + 1/4 row mh+1
        const float wea = mh == 0 ? 0.f : 0.25f, web = mh == 0 ? 1.f : 0.75f;
        const float wob = mh == Hi - 1 ? 1.f : 0.75f, wod = mh == Hi - 1 ? 0.f : 0.25f;
        // columns: fine 8g + 2k reads coarse 4g + k - 1, 4g + k (row[k], row[k + 1]);
        // fine 8g + 2k + 1 reads 4g + k, 4g + k + 1 (row[k + 1], row[k + 2])
        const float c0l = g == 0 ? 0.f : 0.25f, c0r = g == 0 ? 1.f : 0.75f;
        const float c7l = g == G - 1 ? 1.f : 0.75f, c7r = g == G - 1 ? 0.f : 0.25f;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            float row[6];
#pragma unroll
            for (int c = 0; c < 6; ++c)
                row[c] = half == 0 ? fmaf(web, B[c], wea * A[c]) : fmaf(wod, Dn[c], wob * B[c]);
            float out[8];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                out[2 * k] = k == 0 ? fmaf(c0r, row[1], c0l * row[0])
                                    : fmaf(0.75f, row[k + 1], 0.25f * row[k]);
                out[2 * k + 1] = k == 3 ? fmaf(c7r, row[5], c7l * row[4])
                                        : fmaf(0.25f, row[k + 2], 0.75f * row[k + 1]);
            }
            uint32_t w4[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) w4[i] = pack_bf16x2(out[2 * i], out[2 * i + 1]);
            // fine row 2 mh + half of plane l: (l Ho + 2 mh + half) Wo, Wo = 2 Wi
            *reinterpret_cast<uint4*>(yb + __mul24(l, Ho * Wo) + 4 * mhW + half * Wo + 8 * g) =
                make_uint4(w4[0], w4[1], w4[2], w4[3]);
            if constexpr (STATS) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float lo = __uint_as_float(w4[i] << 16) - shift;
                    const float hi = __uint_as_float(w4[i] & 0xffff0000u) - shift;
                    s1 += lo;
                    s2 += lo * lo;
                    s1 += hi;
                    s2 += hi * hi;
                }
            }
        }
        mh += dq;
        g += dr;
        if (g >= G) {
            g -= G;
            ++mh;
        }
        while (mh >= Hi) {
            mh -= Hi;
            ++l;
        }
    }
    if constexpr (STATS) {
        // fixed-order block sum: xor butterfly in each wave, then the waves in order
        __shared__ float red[2][kEwThreads / 64];
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) {
            s1 += __shfl_xor(s1, m, 64);
            s2 += __shfl_xor(s2, m, 64);
        }
        if ((threadIdx.x & 63) == 0) {
            red[0][threadIdx.x >> 6] = s1;
            red[1][threadIdx.x >> 6] = s2;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            float a = 0.f, b = 0.f;
#pragma unroll
            for (int wv = 0; wv < kEwThreads / 64; ++wv) {
                a += red[0][wv];
                b += red[1][wv];
            }
            const int c = nc % us.C, n = nc / us.C, blk = L - nc * nblk;
            const int slices = us.N * nblk;
            float* o = us.part + ((int64_t)c * slices + (int64_t)n * nblk + blk) * 2;
            o[0] = a;
            o[1] = b;
            if (n == 0 && blk == 0) us.part[(int64_t)us.C * slices * 2 + c] = shift;
        }
    }
}

// Transpose of up2_fwd_pl, bf16, Wi % 4 == 0.  A block owns coarse planes
// m0 .. m0 + kPlanes - 1; phase A blends fine planes 2*m0-1 .. 2*m0+2*kPlanes
// along depth into LDS (float32), phase B gathers the 4 x 10 fine rows and
// columns of 4 consecutive coarse voxels of a row.
// With BN, the fine gradient is not read but formed on the fly: dy holds the
// gradient of a = relu(BN(h)) and the fine input is the BN backward's dh =
// k (g - a - (h - mean) b), g = dy where h * scale + shift > 0 (the forward's
// coefficients), rounded as its store would be -- the batch norm's apply pass
// and this transpose in one kernel (h and dh at the fine size).
struct UpBn {
    const bf16* h;       // BN input, fine
    const float* mean;   // saved batch mean [C]
    const float* fcoef;  // forward scale [C], shift [C]
    BnBwdStats st;
    int C, N;
};

template <bool BN>
__global__ __launch_bounds__(kEwThreads) void up2_bwd_pl(const bf16* __restrict__ dy, int Di,
                                                         int Hi, int Wi, int nblk,
                                                         bf16* __restrict__ dx, int accumulate,
                                                         UpBn ub) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int Do = 2 * Di, Ho = 2 * Hi, Wo = 2 * Wi;
    const int HWo = Ho * Wo;  // a multiple of 8 (Wo % 8 == 0)
    float* t = reinterpret_cast<float*>(smem);  // [kPlanes][HWo]
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int nc = L / nblk, m0 = (L - nc * nblk) * kPlanes;
    const bf16* gv = dy + (int64_t)nc * Do * HWo;
    [[maybe_unused]] float bk = 0.f, ba = 0.f, bb = 0.f, bmean = 0.f, fsc = 0.f, fsh = 0.f;
    [[maybe_unused]] const bf16* hv = nullptr;
    if constexpr (BN) {
        // every lane is active here, as the coefficient reduction needs
        const int c = nc % ub.C;
        bn_bwd_coefs(ub.N, (int64_t)Do * HWo, c, ub.st,
                     nc < ub.C && L - nc * nblk == 0 && threadIdx.x == 0, bk, ba, bb);
        bmean = ub.mean[c];
        fsc = ub.fcoef[c];
        fsh = ub.fcoef[ub.C + c];
        hv = ub.h + (int64_t)nc * Do * HWo;
    }
    for (int p = threadIdx.x * 8; p < HWo; p += kEwThreads * 8) {
        float acc[kPlanes][8];
#pragma unroll
        for (int l = 0; l < kPlanes; ++l)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[l][e] = 0.f;
        // all fine planes are requested before any is used (clamped index)
        constexpr int NQ = 2 * kPlanes + 2;
        uint4 raw[NQ];
        [[maybe_unused]] uint4 rawh[NQ];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int od = min(max(2 * m0 - 1 + q, 0), Do - 1);
            raw[q] = *reinterpret_cast<const uint4*>(gv + (int64_t)od * HWo + p);
            if constexpr (BN) rawh[q] = *reinterpret_cast<const uint4*>(hv + (int64_t)od * HWo + p);
        }
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int od = 2 * m0 - 1 + q;
            if (od < 0 || od >= Do) continue;
            float v[8];
            {
                const uint32_t w[4] = {raw[q].x, raw[q].y, raw[q].z, raw[q].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    v[2 * i] = __uint_as_float(w[i] << 16);
                    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
                }
                if constexpr (BN) {
                    const uint32_t hw[4] = {rawh[q].x, rawh[q].y, rawh[q].z, rawh[q].w};
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float h0 = __uint_as_float(hw[i] << 16);
                        const float h1 = __uint_as_float(hw[i] & 0xffff0000u);
                        const float g0 = fmaf(h0, fsc, fsh) > 0.f ? v[2 * i] : 0.f;
                        const float g1 = fmaf(h1, fsc, fsh) > 0.f ? v[2 * i + 1] : 0.f;
                        v[2 * i] = Elt<bf16>::round(bk * (g0 - ba - (h0 - bmean) * bb));
                        v[2 * i + 1] = Elt<bf16>::round(bk * (g1 - ba - (h1 - bmean) * bb));
                    }
                }
            }
#pragma unroll
            for (int l = 0; l < kPlanes; ++l) {
                if (m0 + l >= Di) continue;
                const float wd = x2_w(od, m0 + l, Di);
                if (wd != 0.f)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[l][e] += wd * v[e];
            }
        }
#pragma unroll
        for (int l = 0; l < kPlanes; ++l) {
            float4* d4 = reinterpret_cast<float4*>(t + l * HWo + p);
            d4[0] = make_float4(acc[l][0], acc[l][1], acc[l][2], acc[l][3]);
            d4[1] = make_float4(acc[l][4], acc[l][5], acc[l][6], acc[l][7]);
        }
    }
    __syncthreads();
    const int G = Wi >> 2;
    for (int it = threadIdx.x; it < kPlanes * Hi * G; it += kEwThreads) {
        const int l = it / (Hi * G), r = it - l * (Hi * G);
        const int m = m0 + l;
        if (m >= Di) break;
        const int ih = r / G, g = r - ih * G;
        float rowacc[10];  // fine columns 8g-1 .. 8g+8 blended over the fine rows
#pragma unroll
        for (int j = 0; j < 10; ++j) rowacc[j] = 0.f;
        // transpose weights of coarse index i over fine 2i-1, 2i, 2i+1, 2i+2:
        // 1/4, 3/4, 3/4, 1/4, with the missing fine neighbour at a border
        // folded into the middle weight (1)
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
            const int oh = 2 * ih - 1 + hh;
            if (oh < 0 || oh >= Ho) continue;
            const float wh = (hh == 0 || hh == 3) ? 0.25f
                             : (hh == 1 ? (ih == 0 ? 1.f : 0.75f) : (ih == Hi - 1 ? 1.f : 0.75f));
            const float* src = t + l * HWo + oh * Wo;
            const float4 a = *reinterpret_cast<const float4*>(src + 8 * g);
            const float4 b = *reinterpret_cast<const float4*>(src + 8 * g + 4);
            rowacc[1] += wh * a.x; rowacc[2] += wh * a.y; rowacc[3] += wh * a.z;
            rowacc[4] += wh * a.w; rowacc[5] += wh * b.x; rowacc[6] += wh * b.y;
            rowacc[7] += wh * b.z; rowacc[8] += wh * b.w;
            if (g > 0) rowacc[0] += wh * src[8 * g - 1];
            if (8 * g + 8 < Wo) rowacc[9] += wh * src[8 * g + 8];
        }
        float out[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            // fine columns 2mw-1 .. 2mw+2 are rowacc[2k .. 2k+3]; rowacc[0]
            // and rowacc[9] stay 0 where those columns do not exist
            const int mw = 4 * g + k;
            float v = 0.f;
            v += 0.25f * rowacc[2 * k];
            v += (mw == 0 ? 1.f : 0.75f) * rowacc[2 * k + 1];
            v += (mw == Wi - 1 ? 1.f : 0.75f) * rowacc[2 * k + 2];
            v += 0.25f * rowacc[2 * k + 3];
            out[k] = v;
        }
        uint2* q2 = reinterpret_cast<uint2*>(dx + (((int64_t)nc * Di + m) * Hi + ih) * Wi + 4 * g);
        if (accumulate) {
            const uint2 o = *q2;
            out[0] += __uint_as_float(o.x << 16);
            out[1] += __uint_as_float(o.x & 0xffff0000u);
            out[2] += __uint_as_float(o.y << 16);
            out[3] += __uint_as_float(o.y & 0xffff0000u);
        }
        *q2 = make_uint2(pack_bf16x2(out[0], out[1]),
                         pack_bf16x2(out[2], out[3]));
    }
}

// Transpose of up2_fwd_pl walking a chunk of coarse planes [m0, m1) of one
// (n, c) volume (bf16, Wi % 4 == 0, a fine plane of at most 2 * 256 groups
// of 8).  Each fine plane the chunk reaches is read, and with BN transformed
// as in up2_bwd_pl, exactly once, in increasing order; its depth weights add
// it to the two coarse planes it reaches (register sums, the order of
// up2_bwd_pl).  A completed coarse plane's depth sums go to one of two LDS
// buffers and, after one barrier, are finished in-plane as in up2_bwd_pl,
// while the next two fine planes are already requested.
constexpr int kUpChunk = 24;  // coarse planes per block (a 24-plane volume: one block)
constexpr int kUpItems = 2;  // fine 8-element groups per thread

template <bool BN>
__global__ __launch_bounds__(kEwThreads) void up2_bwd_roll(const bf16* __restrict__ dy, int Di,
                                                           int Hi, int Wi, int nchunk,
                                                           bf16* __restrict__ dx, int accumulate,
                                                           UpBn ub) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int Do = 2 * Di, Ho = 2 * Hi, Wo = 2 * Wi;
    const int HWo = Ho * Wo, NG = HWo >> 3;
    float* t = reinterpret_cast<float*>(smem);  // [2][HWo]
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int nc = L / nchunk, ch = L - nc * nchunk;
    const int m0 = ch * kUpChunk, m1 = min(m0 + kUpChunk, Di);
    const bf16* gv = dy + (int64_t)nc * Do * HWo;
    [[maybe_unused]] float bk = 0.f, ba = 0.f, bb = 0.f, bmean = 0.f, fsc = 0.f, fsh = 0.f;
    [[maybe_unused]] const bf16* hv = nullptr;
    if constexpr (BN) {
        // every lane is active here, as the coefficient reduction needs
        const int c = nc % ub.C;
        bn_bwd_coefs(ub.N, (int64_t)Do * HWo, c, ub.st, nc < ub.C && ch == 0 && threadIdx.x == 0,
                     bk, ba, bb);
        bmean = ub.mean[c];
        fsc = ub.fcoef[c];
        fsh = ub.fcoef[ub.C + c];
        hv = ub.h + (int64_t)nc * Do * HWo;
    }
    bool live[kUpItems];
#pragma unroll
    for (int j = 0; j < kUpItems; ++j) live[j] = threadIdx.x + j * kEwThreads < NG;
    // two fine planes in flight: raw dy (and h) per item
    uint4 rg[2][kUpItems];
    [[maybe_unused]] uint4 rh[2][kUpItems];
    auto issue = [&](int s, int od) {
        if (od < 0 || od >= Do) return;
#pragma unroll
        for (int j = 0; j < kUpItems; ++j) {
            if (!live[j]) continue;
            const int64_t o = (int64_t)od * HWo + (threadIdx.x + j * kEwThreads) * 8;
            rg[s][j] = *reinterpret_cast<const uint4*>(gv + o);
            if constexpr (BN) rh[s][j] = *reinterpret_cast<const uint4*>(hv + o);
        }
    };
    float cur[kUpItems][8], nxt[kUpItems][8];
#pragma unroll
    for (int j = 0; j < kUpItems; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) cur[j][e] = nxt[j][e] = 0.f;
    // fine plane od (loaded in slot s) added to coarse planes ma (into cur)
    // and mb (into nxt, when mb >= 0)
    auto consume = [&](int s, int od, int ma, int mb) {
        if (od < 0 || od >= Do) return;
        const float wa = x2_w(od, ma, Di), wb = mb >= 0 ? x2_w(od, mb, Di) : 0.f;
#pragma unroll
        for (int j = 0; j < kUpItems; ++j) {
            if (!live[j]) continue;
            float v[8];
            const uint32_t w[4] = {rg[s][j].x, rg[s][j].y, rg[s][j].z, rg[s][j].w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[2 * i] = __uint_as_float(w[i] << 16);
                v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
            }
            if constexpr (BN) {
                const uint32_t hw[4] = {rh[s][j].x, rh[s][j].y, rh[s][j].z, rh[s][j].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float h0 = __uint_as_float(hw[i] << 16);
                    const float h1 = __uint_as_float(hw[i] & 0xffff0000u);
                    const float g0 = fmaf(h0, fsc, fsh) > 0.f ? v[2 * i] : 0.f;
                    const float g1 = fmaf(h1, fsc, fsh) > 0.f ? v[2 * i + 1] : 0.f;
                    v[2 * i] = Elt<bf16>::round(bk * (g0 - ba - (h0 - bmean) * bb));
                    v[2 * i + 1] = Elt<bf16>::round(bk * (g1 - ba - (h1 - bmean) * bb));
                }
            }
            if (wa != 0.f)
#pragma unroll
                for (int e = 0; e < 8; ++e) cur[j][e] += wa * v[e];
            if (wb != 0.f)
#pragma unroll
                for (int e = 0; e < 8; ++e) nxt[j][e] += wb * v[e];
        }
    };
    // coarse m0 starts with fine planes 2 m0 - 1 and 2 m0 (they reach m0 - 1 and m0)
    issue(0, 2 * m0 - 1);
    issue(1, 2 * m0);
    consume(0, 2 * m0 - 1, m0, -1);
    consume(1, 2 * m0, m0, -1);
    issue(0, 2 * m0 + 1);
    issue(1, 2 * m0 + 2);
    const int G = Wi >> 2;
    for (int m = m0; m < m1; ++m) {
        // fine planes 2m + 1 and 2m + 2 complete coarse m and start m + 1
        const int mb = m + 1 < m1 ? m + 1 : -1;
        consume(0, 2 * m + 1, m, mb);
        consume(1, 2 * m + 2, m, mb);
        if (mb >= 0) {
            issue(0, 2 * m + 3);
            issue(1, 2 * m + 4);
        }
        float* tb = t + (m & 1) * HWo;
#pragma unroll
        for (int j = 0; j < kUpItems; ++j) {
            if (!live[j]) continue;
            float4* d4 = reinterpret_cast<float4*>(tb + (threadIdx.x + j * kEwThreads) * 8);
            d4[0] = make_float4(cur[j][0], cur[j][1], cur[j][2], cur[j][3]);
            d4[1] = make_float4(cur[j][4], cur[j][5], cur[j][6], cur[j][7]);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                cur[j][e] = nxt[j][e];
                nxt[j][e] = 0.f;
            }
        }
        __syncthreads();
        for (int it = threadIdx.x; it < Hi * G; it += kEwThreads) {
            const int ih = it / G, g = it - ih * G;
            float rowacc[10];  // fine columns 8g-1 .. 8g+8 blended over the fine rows
#pragma unroll
            for (int j = 0; j < 10; ++j) rowacc[j] = 0.f;
#pragma unroll
            for (int hh = 0; hh < 4; ++hh) {
                const int oh = 2 * ih - 1 + hh;
                if (oh < 0 || oh >= Ho) continue;
                const float wh = (hh == 0 || hh == 3)
                                     ? 0.25f
                                     : (hh == 1 ? (ih == 0 ? 1.f : 0.75f)
                                                : (ih == Hi - 1 ? 1.f : 0.75f));
                const float* src = tb + oh * Wo;
                const float4 a = *reinterpret_cast<const float4*>(src + 8 * g);
                const float4 b = *reinterpret_cast<const float4*>(src + 8 * g + 4);
                rowacc[1] += wh * a.x; rowacc[2] += wh * a.y; rowacc[3] += wh * a.z;
                rowacc[4] += wh * a.w; rowacc[5] += wh * b.x; rowacc[6] += wh * b.y;
                rowacc[7] += wh * b.z; rowacc[8] += wh * b.w;
                if (g > 0) rowacc[0] += wh * src[8 * g - 1];
                if (8 * g + 8 < Wo) rowacc[9] += wh * src[8 * g + 8];
            }
            float out[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int mw = 4 * g + k;
                float v = 0.f;
                v += 0.25f * rowacc[2 * k];
                v += (mw == 0 ? 1.f : 0.75f) * rowacc[2 * k + 1];
                v += (mw == Wi - 1 ? 1.f : 0.75f) * rowacc[2 * k + 2];
                v += 0.25f * rowacc[2 * k + 3];
                out[k] = v;
            }
            uint2* q2 =
                reinterpret_cast<uint2*>(dx + (((int64_t)nc * Di + m) * Hi + ih) * Wi + 4 * g);
            if (accumulate) {
                const uint2 o = *q2;
                out[0] += __uint_as_float(o.x << 16);
                out[1] += __uint_as_float(o.x & 0xffff0000u);
                out[2] += __uint_as_float(o.y << 16);
                out[3] += __uint_as_float(o.y & 0xffff0000u);
            }
            *q2 = make_uint2(pack_bf16x2(out[0], out[1]), pack_bf16x2(out[2], out[3]));
        }
    }
}

// taken where every thread has a fine group (smaller planes leave most lanes
// idle through the per-plane steps; there the plane-pair blocks are faster)
static bool up2_roll_ok(int Hi, int Wi) {
    const int64_t ng = (int64_t)4 * Hi * Wi / 8;
    return Wi % 4 == 0 && ng >= kEwThreads && ng <= (int64_t)kUpItems * kEwThreads;
}

// ---------------------------------------------------------------- launchers
rat3d_status pool_fwd(int N, int C, int D, int H, int W, int k, int s, int p, rat3d_dtype dt,
                      const void* x, void* y, uint8_t* argmax, hipStream_t st) {
    const int Do = out_dim(D, k, s, p), Ho = out_dim(H, k, s, p), Wo = out_dim(W, k, s, p);
    const int64_t total = (int64_t)N * C * Do * Ho * Wo;
    const unsigned blocks = (unsigned)ceil_div(total, kEwThreads);
    const double es = dt == RAT3D_BF16 ? 2.0 : 4.0;
    ProfScope ps("pool_fwd", st, 0.0, es * ((double)N * C * D * H * W + total) + total);
    const int HW8 = (H * W + 7) & ~7;
    const size_t lds_f = (size_t)kPlanesF * HW8 * 4;
    const size_t lds_r = (size_t)kPlanesF * H * (W + 4) * 4;
    if (k == 3 && s == 2 && p == 1 && dt == RAT3D_BF16 && W % 8 == 0 && lds_r <= kPlaneLds) {
        const int nblk = (int)ceil_div(Do, kPlanesF);
        pool332_fwd_rows<<<(unsigned)((int64_t)N * C * nblk), kEwThreads, lds_r, st>>>(
            (const bf16*)x, D, H, W, Do, Ho, Wo, nblk, (bf16*)y, argmax);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (k == 3 && s == 2 && p == 1 && dt == RAT3D_BF16 && lds_f <= kPlaneLds) {
        const int nblk = (int)ceil_div(Do, kPlanesF);
        pool332_fwd_pl<<<(unsigned)((int64_t)N * C * nblk), kEwThreads, lds_f, st>>>(
            (const bf16*)x, D, H, W, Do, Ho, Wo, nblk, (bf16*)y, argmax);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (k == 3 && s == 2 && p == 1 && (int64_t)N * C * Do < 65536) {
        const dim3 grid((unsigned)ceil_div((int64_t)Ho * Wo, kEwThreads), N * C * Do);
        if (dt == RAT3D_BF16)
            pool332_fwd_k<bf16><<<grid, kEwThreads, 0, st>>>((const bf16*)x, D, H, W, Do, Ho, Wo,
                                                             (bf16*)y, argmax);
        else
            pool332_fwd_k<float><<<grid, kEwThreads, 0, st>>>((const float*)x, D, H, W, Do, Ho,
                                                              Wo, (float*)y, argmax);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (dt == RAT3D_BF16)
        pool_fwd_k<bf16><<<blocks, kEwThreads, 0, st>>>((const bf16*)x, N * C, D, H, W, k, s, p,
                                                        Do, Ho, Wo, (bf16*)y, argmax);
    else
        pool_fwd_k<float><<<blocks, kEwThreads, 0, st>>>((const float*)x, N * C, D, H, W, k, s,
                                                         p, Do, Ho, Wo, (float*)y, argmax);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status pool_bwd(int N, int C, int D, int H, int W, int k, int s, int p, rat3d_dtype dt,
                      const void* dy, const uint8_t* argmax, void* dx, int accumulate,
                      hipStream_t st) {
    const int Do = out_dim(D, k, s, p), Ho = out_dim(H, k, s, p), Wo = out_dim(W, k, s, p);
    const int64_t total = (int64_t)N * C * D * H * W;
    const unsigned blocks = (unsigned)ceil_div(total, kEwThreads);
    const double es = dt == RAT3D_BF16 ? 2.0 : 4.0;
    const double small = (double)N * C * Do * Ho * Wo;
    ProfScope ps("pool_bwd", st, 0.0, es * (small + total * (1 + accumulate)) + small);
    const size_t lds_b = (size_t)(kPlanes + 1) * Ho * Wo * 3;
    const int kp = k == 3 && s == 2 && p == 1 && dt == RAT3D_BF16 ? pool_sc_kp(D, H, W, Do, Ho, Wo)
                                                                  : 0;
    if (kp > 0) {
        const int nblk = (int)ceil_div(D, 2 * kp);
        pool332_bwd_sc<<<(unsigned)((int64_t)N * C * nblk), kEwThreads,
                         (size_t)2 * kp * H * W * sizeof(float), st>>>(
            (const bf16*)dy, argmax, D, H, W, Do, Ho, Wo, kp, nblk, (bf16*)dx, accumulate);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (k == 3 && s == 2 && p == 1 && dt == RAT3D_BF16 && W % 8 == 0 && lds_b <= kPlaneLds) {
        const int nblk = (int)ceil_div(D, 2 * kPlanes);
        pool332_bwd_pl<<<(unsigned)((int64_t)N * C * nblk), kEwThreads, lds_b, st>>>(
            (const bf16*)dy, argmax, D, H, W, Do, Ho, Wo, nblk, (bf16*)dx, accumulate);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (k == 3 && s == 2 && p == 1 && (int64_t)N * C * D < 65536) {
        const dim3 grid((unsigned)ceil_div((int64_t)H * W, kEwThreads), N * C * D);
        if (dt == RAT3D_BF16)
            pool332_bwd_k<bf16><<<grid, kEwThreads, 0, st>>>((const bf16*)dy, argmax, D, H, W, Do,
                                                             Ho, Wo, (bf16*)dx, accumulate);
        else
            pool332_bwd_k<float><<<grid, kEwThreads, 0, st>>>((const float*)dy, argmax, D, H, W,
                                                              Do, Ho, Wo, (float*)dx, accumulate);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (dt == RAT3D_BF16)
        pool_bwd_k<bf16><<<blocks, kEwThreads, 0, st>>>((const bf16*)dy, argmax, N * C, D, H, W,
                                                        k, s, p, Do, Ho, Wo, (bf16*)dx,
                                                        accumulate);
    else
        pool_bwd_k<float><<<blocks, kEwThreads, 0, st>>>((const float*)dy, argmax, N * C, D, H,
                                                         W, k, s, p, Do, Ho, Wo, (float*)dx,
                                                         accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

static float up_scale(int in, int out) { return (float)in / (float)out; }

rat3d_status up_fwd(int N, int C, int Di, int Hi, int Wi, int Do, int Ho, int Wo,
                    rat3d_dtype dt, const void* x, void* y, hipStream_t st) {
    const int64_t total = (int64_t)N * C * Do * Ho * Wo;
    const unsigned blocks = (unsigned)ceil_div(total, kEwThreads);
    const float sd = up_scale(Di, Do), sh = up_scale(Hi, Ho), sw = up_scale(Wi, Wo);
    ProfScope ps("up_fwd", st, 0.0,
                 (dt == RAT3D_BF16 ? 2.0 : 4.0) * ((double)N * C * Di * Hi * Wi + total));
    const bool x2 = Do == 2 * Di && Ho == 2 * Hi && Wo == 2 * Wi;
    const size_t lds_f = (size_t)2 * kPlanes * ((Hi * Wi + 7) & ~7) * sizeof(float);
    if (x2 && dt == RAT3D_BF16 && Wi % 4 == 0 && lds_f <= kPlaneLds) {
        const int nblk = (int)ceil_div(Di, kPlanes);
        up2_fwd_pl<false><<<(unsigned)((int64_t)N * C * nblk), kEwThreads, lds_f, st>>>(
            (const bf16*)x, Di, Hi, Wi, nblk, (bf16*)y, UpStats{});
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (Ho <= kAxisMax && Wo <= kAxisMax && (int64_t)N * C * Do < 65536) {
        const dim3 grid((unsigned)ceil_div((int64_t)Ho * Wo, kEwThreads), N * C * Do);
        if (dt == RAT3D_BF16)
            up_fwd_tab_k<bf16><<<grid, kEwThreads, 0, st>>>((const bf16*)x, Di, Hi, Wi, Do, Ho, Wo,
                                                            sd, sh, sw, (bf16*)y);
        else
            up_fwd_tab_k<float><<<grid, kEwThreads, 0, st>>>((const float*)x, Di, Hi, Wi, Do, Ho,
                                                             Wo, sd, sh, sw, (float*)y);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (dt == RAT3D_BF16)
        up_fwd_k<bf16><<<blocks, kEwThreads, 0, st>>>((const bf16*)x, N * C, Di, Hi, Wi, Do, Ho,
                                                      Wo, sd, sh, sw, (bf16*)y);
    else
        up_fwd_k<float><<<blocks, kEwThreads, 0, st>>>((const float*)x, N * C, Di, Hi, Wi, Do,
                                                       Ho, Wo, sd, sh, sw, (float*)y);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status up_bwd(int N, int C, int Di, int Hi, int Wi, int Do, int Ho, int Wo,
                    rat3d_dtype dt, const void* dy, void* dx, int accumulate, hipStream_t st) {
    const int64_t total = (int64_t)N * C * Di * Hi * Wi;
    const unsigned blocks = (unsigned)ceil_div(total, kEwThreads);
    const float sd = up_scale(Di, Do), sh = up_scale(Hi, Ho), sw = up_scale(Wi, Wo);
    ProfScope ps("up_bwd", st, 0.0,
                 (dt == RAT3D_BF16 ? 2.0 : 4.0) *
                     ((double)N * C * Do * Ho * Wo + total * (1 + accumulate)));
    const bool x2 = Do == 2 * Di && Ho == 2 * Hi && Wo == 2 * Wi;
    const size_t lds_b = (size_t)kPlanes * Ho * Wo * sizeof(float);
    if (x2 && dt == RAT3D_BF16 && up2_roll_ok(Hi, Wi) &&
        (size_t)2 * Ho * Wo * sizeof(float) <= kPlaneLds) {
        const int nchunk = (int)ceil_div(Di, kUpChunk);
        up2_bwd_roll<false><<<(unsigned)((int64_t)N * C * nchunk), kEwThreads,
                              (size_t)2 * Ho * Wo * sizeof(float), st>>>(
            (const bf16*)dy, Di, Hi, Wi, nchunk, (bf16*)dx, accumulate, UpBn{});
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (x2 && dt == RAT3D_BF16 && Wi % 4 == 0 && lds_b <= kPlaneLds) {
        const int nblk = (int)ceil_div(Di, kPlanes);
        up2_bwd_pl<false><<<(unsigned)((int64_t)N * C * nblk), kEwThreads, lds_b, st>>>(
            (const bf16*)dy, Di, Hi, Wi, nblk, (bf16*)dx, accumulate, UpBn{});
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (Di <= kAxisMax && Hi <= kAxisMax && Wi <= kAxisMax) {
        const size_t lds = (size_t)(Di + Hi + Wi) * sizeof(AxisTaps);
        if (dt == RAT3D_BF16)
            up_bwd_tab_k<bf16><<<blocks, kEwThreads, lds, st>>>((const bf16*)dy, N * C, Di, Hi, Wi,
                                                                Do, Ho, Wo, sd, sh, sw, (bf16*)dx,
                                                                accumulate);
        else
            up_bwd_tab_k<float><<<blocks, kEwThreads, lds, st>>>((const float*)dy, N * C, Di, Hi,
                                                                 Wi, Do, Ho, Wo, sd, sh, sw,
                                                                 (float*)dx, accumulate);
        RAT3D_LAUNCH_CHECK();
        return RAT3D_OK;
    }
    if (dt == RAT3D_BF16)
        up_bwd_k<bf16><<<blocks, kEwThreads, 0, st>>>((const bf16*)dy, N * C, Di, Hi, Wi, Do, Ho,
                                                      Wo, sd, sh, sw, (bf16*)dx, accumulate);
    else
        up_bwd_k<float><<<blocks, kEwThreads, 0, st>>>((const float*)dy, N * C, Di, Hi, Wi, Do,
                                                       Ho, Wo, sd, sh, sw, (float*)dx,
                                                       accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status softmask_fwd(int64_t count, rat3d_dtype dt, const void* z, const void* t,
                          void* out, void* m, hipStream_t st) {
    ProfScope ps("softmask_fwd", st, 0.0, (dt == RAT3D_BF16 ? 2.0 : 4.0) * count * (m ? 4 : 3));
    if (dt == RAT3D_BF16) {
        if (count % 8 == 0)
            softmask_fwd_k<bf16, 8><<<(unsigned)ceil_div(count / 8, kEwThreads), kEwThreads, 0,
                                      st>>>((const bf16*)z, (const bf16*)t, count, (bf16*)out,
                                            (bf16*)m);
        else
            softmask_fwd_k<bf16, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0,
                                      st>>>((const bf16*)z, (const bf16*)t, count, (bf16*)out,
                                            (bf16*)m);
    } else {
        if (count % 4 == 0)
            softmask_fwd_k<float, 4><<<(unsigned)ceil_div(count / 4, kEwThreads), kEwThreads, 0,
                                       st>>>((const float*)z, (const float*)t, count,
                                             (float*)out, (float*)m);
        else
            softmask_fwd_k<float, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0,
                                       st>>>((const float*)z, (const float*)t, count,
                                             (float*)out, (float*)m);
    }
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status softmask_bwd(int64_t count, rat3d_dtype dt, const void* dout, const void* t,
                          const void* m, void* dt_out, int accumulate_dt, void* dz,
                          hipStream_t st, int m_is_z, float* bias_part, int N, int C,
                          int64_t V) {
    if (bias_part && !(dt == RAT3D_BF16 && V > 0 && V % (kEwThreads * 8) == 0 &&
                       count == (int64_t)N * C * V)) {
        set_error("softmask_bwd: per-channel dz sums need bf16 planes of whole blocks");
        return RAT3D_EUNSUPPORTED;
    }
    const SmBias sb{bias_part, V, C, N};
    ProfScope ps("softmask_bwd", st, 0.0,
                 (dt == RAT3D_BF16 ? 2.0 : 4.0) * count * (5 + accumulate_dt));
    if (dt == RAT3D_BF16) {
        if (count % 8 == 0)
            softmask_bwd_k<bf16, 8><<<(unsigned)ceil_div(count / 8, kEwThreads), kEwThreads, 0,
                                      st>>>((const bf16*)dout, (const bf16*)t, (const bf16*)m,
                                            count, (bf16*)dt_out, accumulate_dt, (bf16*)dz, m_is_z, sb);
        else
            softmask_bwd_k<bf16, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0,
                                      st>>>((const bf16*)dout, (const bf16*)t, (const bf16*)m,
                                            count, (bf16*)dt_out, accumulate_dt, (bf16*)dz, m_is_z, SmBias{});
    } else {
        if (count % 4 == 0)
            softmask_bwd_k<float, 4><<<(unsigned)ceil_div(count / 4, kEwThreads), kEwThreads, 0,
                                       st>>>((const float*)dout, (const float*)t,
                                             (const float*)m, count, (float*)dt_out,
                                             accumulate_dt, (float*)dz, m_is_z, SmBias{});
        else
            softmask_bwd_k<float, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0,
                                       st>>>((const float*)dout, (const float*)t,
                                             (const float*)m, count, (float*)dt_out,
                                             accumulate_dt, (float*)dz, m_is_z, SmBias{});
    }
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status add_tensors(int64_t count, rat3d_dtype dt, const void* a, const void* b, void* dst,
                         hipStream_t st) {
    ProfScope ps("add", st, 0.0, (dt == RAT3D_BF16 ? 2.0 : 4.0) * count * 3);
    if (dt == RAT3D_BF16) {
        if (count % 8 == 0)
            add_k<bf16, 8><<<(unsigned)ceil_div(count / 8, kEwThreads), kEwThreads, 0, st>>>(
                (const bf16*)a, (const bf16*)b, count, (bf16*)dst);
        else
            add_k<bf16, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0, st>>>(
                (const bf16*)a, (const bf16*)b, count, (bf16*)dst);
    } else {
        if (count % 4 == 0)
            add_k<float, 4><<<(unsigned)ceil_div(count / 4, kEwThreads), kEwThreads, 0, st>>>(
                (const float*)a, (const float*)b, count, (float*)dst);
        else
            add_k<float, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0, st>>>(
                (const float*)a, (const float*)b, count, (float*)dst);
    }
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

// ---------------------------------------------------------------- x2 upsampling + BN + ReLU
// The soft-mask branch's y = relu(BN(up(xc))) with an exact x2 upsampling:
// the forward writes h = up(xc) (kept: the backward needs it) and takes the
// BN statistics partials from the same pass; the backward forms the
// gradient of h on the fly inside the upsampling transpose (see up2_fwd_pl
// and up2_bwd_pl).  bf16, Wi % 4 == 0, one workspace as batch norm's.
static int up2_nblk(int Di) { return (int)ceil_div(Di, kPlanes); }

bool up2_bn_ok(int N, int C, int Di, int Hi, int Wi, rat3d_dtype dt) {
    const int64_t V = (int64_t)8 * Di * Hi * Wi;
    const size_t lds_f = (size_t)2 * kPlanes * ((Hi * Wi + 7) & ~7) * sizeof(float);
    const size_t lds_b = (size_t)kPlanes * 4 * Hi * Wi * sizeof(float);
    return dt == RAT3D_BF16 && Wi % 4 == 0 && V % 8 == 0 && lds_f <= kPlaneLds &&
           lds_b <= kPlaneLds &&
           (size_t)N * up2_nblk(Di) <= bn_max_slices(BnGeom{N, C, V});
}

rat3d_status up2_bn_relu_fwd(int N, int C, int Di, int Hi, int Wi, const void* xc, void* h,
                             float eps, float momentum, const float* gamma, const float* beta,
                             void* y, float* save_mean, float* save_invstd, float* run_mean,
                             float* run_var, float* save_coef, void* bn_ws, hipStream_t st) {
    if (!up2_bn_ok(N, C, Di, Hi, Wi, RAT3D_BF16)) {
        set_error("up2_bn_relu_fwd: unsupported shape");
        return RAT3D_EUNSUPPORTED;
    }
    const int nblk = up2_nblk(Di);
    const BnGeom g{N, C, (int64_t)8 * Di * Hi * Wi};
    const size_t lds_f = (size_t)2 * kPlanes * ((Hi * Wi + 7) & ~7) * sizeof(float);
    {
        ProfScope ps("up_fwd", st, 0.0, 2.0 * ((double)N * C * Di * Hi * Wi + (double)N * C * g.V));
        up2_fwd_pl<true><<<(unsigned)((int64_t)N * C * nblk), kEwThreads, lds_f, st>>>(
            (const bf16*)xc, Di, Hi, Wi, nblk, (bf16*)h, UpStats{(float*)bn_ws, C, N});
        RAT3D_LAUNCH_CHECK();
    }
    return bn_fwd_apply_from(g, eps, momentum, h, gamma, beta, y, save_mean, save_invstd,
                             run_mean, run_var, save_coef, (const float*)bn_ws, N * nblk, st);
}

rat3d_status bn_relu_bwd_up2(int N, int C, int Di, int Hi, int Wi, const void* dy, const void* h,
                             const float* gamma, const float* save_mean,
                             const float* save_invstd, const float* fwd_coef, float* dgamma,
                             float* dbeta, int accumulate, void* bn_ws, void* dxc,
                             hipStream_t st) {
    if (!up2_bn_ok(N, C, Di, Hi, Wi, RAT3D_BF16) || !fwd_coef) {
        set_error("bn_relu_bwd_up2: unsupported shape");
        return RAT3D_EUNSUPPORTED;
    }
    const BnGeom g{N, C, (int64_t)8 * Di * Hi * Wi};
    UpBn ub;
    ub.h = (const bf16*)h;
    ub.mean = save_mean;
    ub.fcoef = fwd_coef;
    ub.C = C;
    ub.N = N;
    const rat3d_status s0 = bn_bwd_stats_x(g, dy, h, gamma, save_mean, save_invstd, fwd_coef,
                                           dgamma, dbeta, accumulate, bn_ws, st, &ub.st);
    if (s0 != RAT3D_OK) return s0;
    const int nblk = up2_nblk(Di);
    const size_t lds_b = (size_t)kPlanes * 4 * Hi * Wi * sizeof(float);
    ProfScope ps("bn_bwd_apply_up", st, 0.0,
                 2.0 * (2.0 * N * C * g.V + (double)N * C * Di * Hi * Wi));
    if (up2_roll_ok(Hi, Wi)) {
        const int nchunk = (int)ceil_div(Di, kUpChunk);
        up2_bwd_roll<true><<<(unsigned)((int64_t)N * C * nchunk), kEwThreads,
                             (size_t)2 * 4 * Hi * Wi * sizeof(float), st>>>(
            (const bf16*)dy, Di, Hi, Wi, nchunk, (bf16*)dxc, 0, ub);
    } else {
        up2_bwd_pl<true><<<(unsigned)((int64_t)N * C * nblk), kEwThreads, lds_b, st>>>(
            (const bf16*)dy, Di, Hi, Wi, nblk, (bf16*)dxc, 0, ub);
    }
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace rat3d
