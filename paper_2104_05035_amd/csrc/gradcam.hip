// Inference-mode pieces of the explainable block: 3D Grad-CAM of the full
// network (use-case section: gradient-weighted class activation mapping).
//   * BN with the running statistics (forward and input gradient): an affine
//     map per channel, y = act(x * s + t [+ r]), s = gamma / sqrt(var + eps),
//     t = beta - mean * s; backward dx = s * g, g = dy masked by y > 0;
//   * the gradient seed d logit_k / d top = fc_w[k] / V at the last stage
//     (average pool, then the linear layer), and the logits themselves;
//   * alpha[n, c] = voxel mean of the target map's gradient; the map
//     cam[n, v] = max(0, sum_c alpha[n, c] A[n, c, v]); its trilinear
//     resampling to the input size (half-pixel centres, any ratio).
// All bandwidth-bound; every reduction runs in a fixed order (no atomics).
#include "kernels.hpp"
#include "prof.hpp"
#include "vec.hpp"

namespace rat3d {
namespace {

constexpr int kThreads = 256;

// One (n, c) plane per group of `chunks` blocks; each thread VEC elements.
template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void bn_eval_fwd_k(
    const T* __restrict__ x, const T* __restrict__ res, T* __restrict__ y, int C, int64_t V,
    int chunks, int relu, float eps, const float* __restrict__ gamma,
    const float* __restrict__ beta, const float* __restrict__ rmean,
    const float* __restrict__ rvar) {
    const int plane = blockIdx.x / chunks;
    const int64_t i = ((int64_t)(blockIdx.x - plane * chunks) * kThreads + threadIdx.x) * VEC;
    if (i >= V) return;
    const int c = plane % C;
    const float s = gamma[c] / sqrtf(rvar[c] + eps);
    const float t = beta[c] - rmean[c] * s;
    const int64_t o = (int64_t)plane * V + i;
    float v[VEC], r[VEC];
    vload<T, VEC>(x + o, v);
    if (res) vload<T, VEC>(res + o, r);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        float a = fmaf(v[j], s, t);
        if (res) a += r[j];
        v[j] = relu ? fmaxf(a, 0.f) : a;
    }
    vstore<T, VEC>(y + o, v);
}

// dx = s * g and dres (=|+=) g, g = dy * [y > 0] under ReLU.
template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void bn_eval_bwd_k(
    const T* __restrict__ dy, const T* __restrict__ y, T* __restrict__ dx, T* __restrict__ dres,
    int dres_acc, int C, int64_t V, int chunks, int relu, float eps,
    const float* __restrict__ gamma, const float* __restrict__ rvar) {
    const int plane = blockIdx.x / chunks;
    const int64_t i = ((int64_t)(blockIdx.x - plane * chunks) * kThreads + threadIdx.x) * VEC;
    if (i >= V) return;
    const int c = plane % C;
    const float s = gamma[c] / sqrtf(rvar[c] + eps);
    const int64_t o = (int64_t)plane * V + i;
    float g[VEC], m[VEC], d[VEC];
    vload<T, VEC>(dy + o, g);
    if (relu) {
        vload<T, VEC>(y + o, m);
#pragma unroll
        for (int j = 0; j < VEC; ++j) g[j] = m[j] > 0.f ? g[j] : 0.f;
    }
    if (dx) {
#pragma unroll
        for (int j = 0; j < VEC; ++j) d[j] = s * g[j];
        vstore<T, VEC>(dx + o, d);
    }
    if (dres) {
        if (dres_acc) {
            vload<T, VEC>(dres + o, d);
#pragma unroll
            for (int j = 0; j < VEC; ++j) g[j] += d[j];
        }
        vstore<T, VEC>(dres + o, g);
    }
}

// dtop[n, c, v] = fc_w[k_n, c] / V, k_n = classes[n] clamped into range.
template <typename T>
__global__ __launch_bounds__(kThreads) void gradcam_seed_k(const float* __restrict__ fc_w,
                                                           const int32_t* __restrict__ classes,
                                                           int classes_n, int C, int64_t V,
                                                           int64_t count, T* __restrict__ dtop) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= count) return;
    const int64_t plane = i / V;
    const int n = (int)(plane / C), c = (int)(plane % C);
    int k = classes[n];
    k = k < 0 ? 0 : (k >= classes_n ? classes_n - 1 : k);
    Elt<T>::st(dtop + i, fc_w[(int64_t)k * C + c] / (float)V);
}

// logits[n, k] = sum_c fc_w[k, c] * mean_v top[n, c, v] + fc_b[k]; one block
// per volume, channel means in fixed order, then a fixed-order tree.
template <typename T>
__global__ __launch_bounds__(kThreads) void gradcam_logits_k(const T* __restrict__ top, int C,
                                                             int64_t V, int classes_n,
                                                             const float* __restrict__ fc_w,
                                                             const float* __restrict__ fc_b,
                                                             float* __restrict__ logits) {
    __shared__ float red[8][kThreads];
    const int n = blockIdx.x;
    float acc[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = 0.f;
    for (int c = threadIdx.x; c < C; c += kThreads) {
        const T* p = top + ((int64_t)n * C + c) * V;
        float s = 0.f;
        for (int64_t v = 0; v < V; ++v) s += Elt<T>::ld(p + v);
        const float mean = s / (float)V;
        for (int k = 0; k < classes_n; ++k) acc[k] = fmaf(fc_w[(int64_t)k * C + c], mean, acc[k]);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) red[k][threadIdx.x] = acc[k];
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w)
            for (int k = 0; k < classes_n; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x < classes_n)
        logits[n * classes_n + threadIdx.x] = red[threadIdx.x][0] + fc_b[threadIdx.x];
}

// alpha[plane] = mean of dA over the plane's V voxels; one block per plane.
template <typename T>
__global__ __launch_bounds__(kThreads) void gradcam_alpha_k(const T* __restrict__ dA, int64_t V,
                                                            float* __restrict__ alpha) {
    __shared__ float red[kThreads];
    const T* p = dA + (int64_t)blockIdx.x * V;
    float s = 0.f;
    for (int64_t v = threadIdx.x; v < V; v += kThreads) s += Elt<T>::ld(p + v);
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) alpha[blockIdx.x] = red[0] / (float)V;
}

// cam[n, v] = max(0, sum_c alpha[n, c] A[n, c, v]), channels in order.
template <typename T>
__global__ __launch_bounds__(kThreads) void gradcam_map_k(const T* __restrict__ A,
                                                          const float* __restrict__ alpha, int N,
                                                          int C, int64_t V,
                                                          float* __restrict__ cam) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= (int64_t)N * V) return;
    const int n = (int)(i / V);
    const int64_t v = i - (int64_t)n * V;
    const T* p = A + (int64_t)n * C * V + v;
    const float* a = alpha + (int64_t)n * C;
    float s = 0.f;
    for (int c = 0; c < C; ++c) s = fmaf(a[c], Elt<T>::ld(p + (int64_t)c * V), s);
    cam[i] = fmaxf(s, 0.f);
}

// One axis of the half-pixel resampling: taps i0, i1 and the weight of i1.
__device__ __forceinline__ void axis_taps(int o, int in, int out, int& i0, int& i1, float& l) {
    float src = ((float)o + 0.5f) * ((float)in / (float)out) - 0.5f;
    src = fmaxf(src, 0.f);
    i0 = min((int)src, in - 1);
    i1 = min(i0 + 1, in - 1);
    l = src - (float)i0;
}

// Trilinear resampling of float32 maps [N][Di][Hi][Wi] to [N][Do][Ho][Wo].
__global__ __launch_bounds__(kThreads) void gradcam_up_k(const float* __restrict__ src, int N,
                                                         int Di, int Hi, int Wi, int Do, int Ho,
                                                         int Wo, float* __restrict__ dst) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t total = (int64_t)N * Do * Ho * Wo;
    if (i >= total) return;
    const int ow = (int)(i % Wo);
    const int oh = (int)((i / Wo) % Ho);
    const int od = (int)((i / ((int64_t)Wo * Ho)) % Do);
    const int n = (int)(i / ((int64_t)Wo * Ho * Do));
    int d0, d1, h0, h1, w0, w1;
    float ld, lh, lw;
    axis_taps(od, Di, Do, d0, d1, ld);
    axis_taps(oh, Hi, Ho, h0, h1, lh);
    axis_taps(ow, Wi, Wo, w0, w1, lw);
    const float* p = src + (int64_t)n * Di * Hi * Wi;
    auto at = [&](int d, int h, int w) { return p[((int64_t)d * Hi + h) * Wi + w]; };
    const float c00 = at(d0, h0, w0) * (1.f - lw) + at(d0, h0, w1) * lw;
    const float c01 = at(d0, h1, w0) * (1.f - lw) + at(d0, h1, w1) * lw;
    const float c10 = at(d1, h0, w0) * (1.f - lw) + at(d1, h0, w1) * lw;
    const float c11 = at(d1, h1, w0) * (1.f - lw) + at(d1, h1, w1) * lw;
    const float c0 = c00 * (1.f - lh) + c01 * lh;
    const float c1 = c10 * (1.f - lh) + c11 * lh;
    dst[i] = c0 * (1.f - ld) + c1 * ld;
}

template <typename T, int VEC>
rat3d_status bn_eval_fwd_t(const BnGeom& g, int relu, float eps, const void* x, const void* res,
                           const float* gamma, const float* beta, const float* rmean,
                           const float* rvar, void* y, hipStream_t st) {
    const int chunks = (int)ceil_div(g.V, (int64_t)kThreads * VEC);
    bn_eval_fwd_k<T, VEC><<<(unsigned)((int64_t)g.N * g.C * chunks), kThreads, 0, st>>>(
        (const T*)x, (const T*)res, (T*)y, g.C, g.V, chunks, relu, eps, gamma, beta, rmean, rvar);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

template <typename T, int VEC>
rat3d_status bn_eval_bwd_t(const BnGeom& g, int relu, float eps, const void* dy, const void* y,
                           const float* gamma, const float* rvar, void* dx, void* dres,
                           int dres_acc, hipStream_t st) {
    const int chunks = (int)ceil_div(g.V, (int64_t)kThreads * VEC);
    bn_eval_bwd_k<T, VEC><<<(unsigned)((int64_t)g.N * g.C * chunks), kThreads, 0, st>>>(
        (const T*)dy, (const T*)y, (T*)dx, (T*)dres, dres_acc, g.C, g.V, chunks, relu, eps, gamma,
        rvar);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace

rat3d_status bn_eval_fwd(const BnGeom& g, rat3d_dtype dt, int relu, float eps, const void* x,
                         const void* residual, const float* gamma, const float* beta,
                         const float* run_mean, const float* run_var, void* y, hipStream_t st) {
    const size_t esz = dt == RAT3D_BF16 ? 2 : 4;
    ProfScope ps("bn_eval_fwd", st, 0.0,
                 (double)esz * g.N * g.C * g.V * (residual ? 3.0 : 2.0));
    if (dt == RAT3D_BF16)
        return g.V % 8 == 0
                   ? bn_eval_fwd_t<bf16, 8>(g, relu, eps, x, residual, gamma, beta, run_mean,
                                            run_var, y, st)
                   : bn_eval_fwd_t<bf16, 1>(g, relu, eps, x, residual, gamma, beta, run_mean,
                                            run_var, y, st);
    return g.V % 4 == 0 ? bn_eval_fwd_t<float, 4>(g, relu, eps, x, residual, gamma, beta,
                                                  run_mean, run_var, y, st)
                        : bn_eval_fwd_t<float, 1>(g, relu, eps, x, residual, gamma, beta,
                                                  run_mean, run_var, y, st);
}

rat3d_status bn_eval_bwd(const BnGeom& g, rat3d_dtype dt, int relu, float eps, const void* dy,
                         const void* y, const float* gamma, const float* run_var, void* dx,
                         void* dres, int dres_acc, hipStream_t st) {
    const size_t esz = dt == RAT3D_BF16 ? 2 : 4;
    ProfScope ps("bn_eval_bwd", st, 0.0,
                 (double)esz * g.N * g.C * g.V *
                     (1.0 + relu + (dx ? 1.0 : 0.0) + (dres ? 1.0 + dres_acc : 0.0)));
    if (dt == RAT3D_BF16)
        return g.V % 8 == 0 ? bn_eval_bwd_t<bf16, 8>(g, relu, eps, dy, y, gamma, run_var, dx,
                                                     dres, dres_acc, st)
                            : bn_eval_bwd_t<bf16, 1>(g, relu, eps, dy, y, gamma, run_var, dx,
                                                     dres, dres_acc, st);
    return g.V % 4 == 0 ? bn_eval_bwd_t<float, 4>(g, relu, eps, dy, y, gamma, run_var, dx, dres,
                                                  dres_acc, st)
                        : bn_eval_bwd_t<float, 1>(g, relu, eps, dy, y, gamma, run_var, dx, dres,
                                                  dres_acc, st);
}

rat3d_status gradcam_seed(int N, int C, int64_t V, int classes_n, rat3d_dtype dt,
                          const float* fc_w, const int32_t* classes, void* dtop, hipStream_t st) {
    const int64_t count = (int64_t)N * C * V;
    const unsigned grid = (unsigned)ceil_div(count, kThreads);
    if (dt == RAT3D_BF16)
        gradcam_seed_k<bf16><<<grid, kThreads, 0, st>>>(fc_w, classes, classes_n, C, V, count,
                                                        (bf16*)dtop);
    else
        gradcam_seed_k<float><<<grid, kThreads, 0, st>>>(fc_w, classes, classes_n, C, V, count,
                                                         (float*)dtop);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status gradcam_logits(int N, int C, int64_t V, int classes_n, rat3d_dtype dt,
                            const void* top, const float* fc_w, const float* fc_b,
                            float* logits, hipStream_t st) {
    if (classes_n > 8) {
        set_error("gradcam: at most 8 classes");
        return RAT3D_EUNSUPPORTED;
    }
    if (dt == RAT3D_BF16)
        gradcam_logits_k<bf16><<<N, kThreads, 0, st>>>((const bf16*)top, C, V, classes_n, fc_w,
                                                       fc_b, logits);
    else
        gradcam_logits_k<float><<<N, kThreads, 0, st>>>((const float*)top, C, V, classes_n, fc_w,
                                                        fc_b, logits);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status gradcam_maps(int N, int C, int Dt, int Ht, int Wt, rat3d_dtype dt, const void* A,
                          const void* dA, float* alpha, float* cam, int D0, int H0, int W0,
                          float* cam_up, hipStream_t st) {
    const int64_t V = (int64_t)Dt * Ht * Wt;
    ProfScope ps("gradcam_maps", st, 0.0,
                 (dt == RAT3D_BF16 ? 2.0 : 4.0) * 2.0 * N * C * V + 4.0 * N * V);
    if (dt == RAT3D_BF16) {
        gradcam_alpha_k<bf16><<<(unsigned)(N * C), kThreads, 0, st>>>((const bf16*)dA, V, alpha);
        RAT3D_LAUNCH_CHECK();
        gradcam_map_k<bf16><<<(unsigned)ceil_div((int64_t)N * V, kThreads), kThreads, 0, st>>>(
            (const bf16*)A, alpha, N, C, V, cam);
    } else {
        gradcam_alpha_k<float><<<(unsigned)(N * C), kThreads, 0, st>>>((const float*)dA, V,
                                                                       alpha);
        RAT3D_LAUNCH_CHECK();
        gradcam_map_k<float><<<(unsigned)ceil_div((int64_t)N * V, kThreads), kThreads, 0, st>>>(
            (const float*)A, alpha, N, C, V, cam);
    }
    RAT3D_LAUNCH_CHECK();
    if (cam_up) {
        const int64_t total = (int64_t)N * D0 * H0 * W0;
        gradcam_up_k<<<(unsigned)ceil_div(total, kThreads), kThreads, 0, st>>>(
            cam, N, Dt, Ht, Wt, D0, H0, W0, cam_up);
        RAT3D_LAUNCH_CHECK();
    }
    return RAT3D_OK;
}

}  // namespace rat3d
