// Soft-mask branch kernels of the residual attention module: max pooling
// down (with a uint8 argmax), trilinear resampling up, and the sigmoid fuse
// out = (1 + sigmoid(z)) * T.  All are HBM-bound elementwise/stencil kernels;
// every backward is written in gather form (one thread per destination
// element, no atomics), so results are deterministic.
#include "common.hpp"
#include "kernels.hpp"
#include "vec.hpp"
#include "prof.hpp"

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
__device__ __forceinline__ float sigmoidf(float z) { return 1.f / (1.f + expf(-z)); }

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

template <typename T, int VEC>
__global__ __launch_bounds__(kEwThreads) void softmask_bwd_k(
    const T* __restrict__ dout, const T* __restrict__ t, const T* __restrict__ m, int64_t count,
    T* __restrict__ dt, int accumulate_dt, T* __restrict__ dz) {
    const int64_t i = ((int64_t)blockIdx.x * kEwThreads + threadIdx.x) * VEC;
    if (i >= count) return;
    float g[VEC], tv[VEC], mv[VEC], a[VEC], b[VEC];
    vload<T, VEC>(dout + i, g);
    vload<T, VEC>(t + i, tv);
    vload<T, VEC>(m + i, mv);
    if (accumulate_dt) vload<T, VEC>(dt + i, b);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        a[j] = (1.f + mv[j]) * g[j];
        if (accumulate_dt) a[j] += b[j];
        b[j] = g[j] * tv[j] * mv[j] * (1.f - mv[j]);
    }
    vstore<T, VEC>(dt + i, a);
    vstore<T, VEC>(dz + i, b);
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

// ---------------------------------------------------------------- launchers
rat3d_status pool_fwd(int N, int C, int D, int H, int W, int k, int s, int p, rat3d_dtype dt,
                      const void* x, void* y, uint8_t* argmax, hipStream_t st) {
    const int Do = out_dim(D, k, s, p), Ho = out_dim(H, k, s, p), Wo = out_dim(W, k, s, p);
    const int64_t total = (int64_t)N * C * Do * Ho * Wo;
    const unsigned blocks = (unsigned)ceil_div(total, kEwThreads);
    const double es = dt == RAT3D_BF16 ? 2.0 : 4.0;
    ProfScope ps("pool_fwd", st, 0.0, es * ((double)N * C * D * H * W + total) + total);
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
                          hipStream_t st) {
    ProfScope ps("softmask_bwd", st, 0.0,
                 (dt == RAT3D_BF16 ? 2.0 : 4.0) * count * (5 + accumulate_dt));
    if (dt == RAT3D_BF16) {
        if (count % 8 == 0)
            softmask_bwd_k<bf16, 8><<<(unsigned)ceil_div(count / 8, kEwThreads), kEwThreads, 0,
                                      st>>>((const bf16*)dout, (const bf16*)t, (const bf16*)m,
                                            count, (bf16*)dt_out, accumulate_dt, (bf16*)dz);
        else
            softmask_bwd_k<bf16, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0,
                                      st>>>((const bf16*)dout, (const bf16*)t, (const bf16*)m,
                                            count, (bf16*)dt_out, accumulate_dt, (bf16*)dz);
    } else {
        if (count % 4 == 0)
            softmask_bwd_k<float, 4><<<(unsigned)ceil_div(count / 4, kEwThreads), kEwThreads, 0,
                                       st>>>((const float*)dout, (const float*)t,
                                             (const float*)m, count, (float*)dt_out,
                                             accumulate_dt, (float*)dz);
        else
            softmask_bwd_k<float, 1><<<(unsigned)ceil_div(count, kEwThreads), kEwThreads, 0,
                                       st>>>((const float*)dout, (const float*)t,
                                             (const float*)m, count, (float*)dt_out,
                                             accumulate_dt, (float*)dz);
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

}  // namespace rat3d
