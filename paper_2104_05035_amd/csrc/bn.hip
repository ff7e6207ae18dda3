// Training-mode 3D batch normalisation fused with ReLU and the residual add.
//
// Forward:  (1) per (channel, slice) partial sums of (x - shift) and its
//           square, shift = the channel's first element (guards the
//           one-pass variance against a large mean); (2) per channel, the
//           partials are combined in float64 in a fixed order into mean,
//           biased variance, invstd, the apply coefficients and the running
//           statistics; (3) y = act(x * scale + bias [+ residual]).
// Backward: (1) per (channel, slice) partial sums of g and g * (x - mean),
//           g = dy masked by y > 0; (2) per channel dbeta, dgamma and the
//           apply coefficients; (3) dx = k * (g - dbeta/M - xhat * dgamma/M),
//           dresidual = g (or dresidual += g, one rounding).  Without a residual, y > 0 is the same test as
//           x * scale + shift > 0 with the forward's own float coefficients
//           (the apply computes exactly that value before the max with 0), so
//           given those coefficients the backward reads x instead of x and y.
// NCDHW: one (n, c) plane is V contiguous voxels; a slice is a contiguous
// segment of one plane, so per-element indexing needs no division.  A
// channel's partials are the N * SP segment sums of its planes, combined in
// a fixed order.  Everything is HBM-bound: loads and stores are 16-byte
// vectors when V allows.
#include "common.hpp"
#include "kernels.hpp"
#include "vec.hpp"
#include "prof.hpp"

namespace rat3d {

constexpr int kBnThreads = 256;

struct BnSlices {
    int per_plane;    // segments per (n, c) plane
    int per_channel;  // N * per_plane partials per channel
    int64_t len;      // elements per segment (multiple of the vector width)
};

static BnSlices bn_slices(const BnGeom& g) {
    int64_t want = ceil_div(2048, (int64_t)g.C * g.N);  // aim for ~2048 blocks in total
    int64_t by_size = ceil_div(g.V, 16384);              // at least ~16K elements per segment
    int64_t s = want < by_size ? want : by_size;
    if (s < 1) s = 1;
    int64_t len = ceil_div(g.V, s);
    len = ceil_div(len, 8) * 8;
    s = ceil_div(g.V, len);
    return BnSlices{(int)s, (int)(s * g.N), len};
}

size_t bn_ws_bytes(const BnGeom& g) {
    const BnSlices sl = bn_slices(g);
    // partial pairs (2 floats per slice) + 4 floats of coefficients per channel
    return ((size_t)g.C * sl.per_channel * 2 + (size_t)g.C * 4) * sizeof(float);
}

// Block reduction of two floats; result valid in thread 0.
__device__ __forceinline__ void block_sum2(float& a, float& b) {
    __shared__ float ra[kBnThreads], rb[kBnThreads];
    ra[threadIdx.x] = a;
    rb[threadIdx.x] = b;
    __syncthreads();
    for (int w = kBnThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) {
            ra[threadIdx.x] += ra[threadIdx.x + w];
            rb[threadIdx.x] += rb[threadIdx.x + w];
        }
        __syncthreads();
    }
    a = ra[0];
    b = rb[0];
}

// Block (c, n * SP + seg): segment seg of plane (n, c).
template <typename T, int VEC>
__global__ __launch_bounds__(kBnThreads) void bn_fwd_stats(const T* __restrict__ x, int C,
                                                           int64_t V, int SP, int64_t len,
                                                           float* __restrict__ part) {
    const int c = blockIdx.x, sidx = blockIdx.y;
    const int n = sidx / SP, seg = sidx - n * SP;
    const float shift = Elt<T>::ld(x + (int64_t)c * V);
    const int64_t beg = (int64_t)seg * len;
    const int64_t cnt = (beg + len < V ? beg + len : V) - beg;
    const T* p = x + ((int64_t)n * C + c) * V + beg;
    float s1 = 0.f, s2 = 0.f;
    for (int64_t e = (int64_t)threadIdx.x * VEC; e < cnt; e += (int64_t)kBnThreads * VEC) {
        float v[VEC];
        vload<T, VEC>(p + e, v);
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            const float d = v[j] - shift;
            s1 += d;
            s2 += d * d;
        }
    }
    block_sum2(s1, s2);
    if (threadIdx.x == 0) {
        float* o = part + ((int64_t)c * gridDim.y + sidx) * 2;
        o[0] = s1;
        o[1] = s2;
    }
}

// One thread per channel: combine slice partials (fixed order, float64).
template <typename T>
__global__ void bn_fwd_finalize(const T* __restrict__ x, int N, int C, int64_t V, int slices,
                                const float* __restrict__ part, const float* __restrict__ gamma,
                                const float* __restrict__ beta, float eps, float momentum,
                                float* __restrict__ save_mean, float* __restrict__ save_invstd,
                                float* __restrict__ run_mean, float* __restrict__ run_var,
                                float* __restrict__ coef, float* __restrict__ save_coef) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    const double shift = (double)Elt<T>::ld(x + (int64_t)c * V);
    double s1 = 0.0, s2 = 0.0;
    for (int i = 0; i < slices; ++i) {
        s1 += (double)part[((int64_t)c * slices + i) * 2];
        s2 += (double)part[((int64_t)c * slices + i) * 2 + 1];
    }
    const double M = (double)N * (double)V;
    const double dm = s1 / M;
    double var = s2 / M - dm * dm;
    if (var < 0.0) var = 0.0;
    const double mean = shift + dm;
    const double invstd = 1.0 / sqrt(var + (double)eps);
    save_mean[c] = (float)mean;
    save_invstd[c] = (float)invstd;
    const float scale = (float)((double)gamma[c] * invstd);
    const float bias = (float)((double)beta[c] - mean * (double)scale);
    coef[c] = scale;
    coef[C + c] = bias;
    if (save_coef) {
        save_coef[c] = scale;
        save_coef[C + c] = bias;
    }
    if (run_mean) run_mean[c] = (float)((1.0 - momentum) * run_mean[c] + momentum * mean);
    if (run_var) {
        const double unb = M > 1.0 ? var * M / (M - 1.0) : var;
        run_var[c] = (float)((1.0 - momentum) * run_var[c] + momentum * unb);
    }
}

// One-dimensional grid: block b covers chunk b % cpp of plane b / cpp.
template <typename T, int VEC, bool RELU, bool RES>
__global__ __launch_bounds__(kBnThreads) void bn_fwd_apply(const T* __restrict__ x,
                                                           const T* __restrict__ r, int C,
                                                           int64_t V, unsigned cpp,
                                                           const float* __restrict__ coef,
                                                           T* __restrict__ y) {
    const int plane = (int)(blockIdx.x / cpp);  // wave-uniform
    const int64_t e = ((int64_t)(blockIdx.x - (unsigned)plane * cpp) * kBnThreads + threadIdx.x) * VEC;
    if (e >= V) return;
    const int c = plane % C;
    const int64_t i = (int64_t)plane * V + e;
    const float sc = coef[c], sh = coef[C + c];
    float v[VEC];
    vload<T, VEC>(x + i, v);
    float rv[VEC];
    if constexpr (RES) vload<T, VEC>(r + i, rv);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        float o = fmaf(v[j], sc, sh);
        if constexpr (RES) o += rv[j];
        if constexpr (RELU) o = fmaxf(o, 0.f);
        v[j] = o;
    }
    vstore<T, VEC>(y + i, v);
}

// ReLU mask of the backward: none, y > 0, or x * scale + shift > 0.
enum { kMaskNone = 0, kMaskY = 1, kMaskX = 2 };

template <typename T, int VEC, int MASK>
__global__ __launch_bounds__(kBnThreads) void bn_bwd_stats(const T* __restrict__ dy,
                                                           const T* __restrict__ x,
                                                           const T* __restrict__ y, int C,
                                                           int64_t V, int SP, int64_t len,
                                                           const float* __restrict__ save_mean,
                                                           const float* __restrict__ fcoef,
                                                           float* __restrict__ part) {
    const int c = blockIdx.x, sidx = blockIdx.y;
    const int n = sidx / SP, seg = sidx - n * SP;
    const float mean = save_mean[c];
    const float fsc = MASK == kMaskX ? fcoef[c] : 0.f, fsh = MASK == kMaskX ? fcoef[C + c] : 0.f;
    const int64_t beg = (int64_t)seg * len;
    const int64_t cnt = (beg + len < V ? beg + len : V) - beg;
    const int64_t base = ((int64_t)n * C + c) * V + beg;
    float s1 = 0.f, s2 = 0.f;
    for (int64_t e = (int64_t)threadIdx.x * VEC; e < cnt; e += (int64_t)kBnThreads * VEC) {
        const int64_t idx = base + e;
        float g[VEC], xv[VEC];
        vload<T, VEC>(dy + idx, g);
        vload<T, VEC>(x + idx, xv);
        if constexpr (MASK == kMaskY) {
            float yv[VEC];
            vload<T, VEC>(y + idx, yv);
#pragma unroll
            for (int j = 0; j < VEC; ++j) g[j] = yv[j] > 0.f ? g[j] : 0.f;
        } else if constexpr (MASK == kMaskX) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) g[j] = fmaf(xv[j], fsc, fsh) > 0.f ? g[j] : 0.f;
        }
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            s1 += g[j];
            s2 += g[j] * (xv[j] - mean);
        }
    }
    block_sum2(s1, s2);
    if (threadIdx.x == 0) {
        float* o = part + ((int64_t)c * gridDim.y + sidx) * 2;
        o[0] = s1;
        o[1] = s2;
    }
}

__global__ void bn_bwd_finalize(int N, int C, int64_t V, int slices,
                                const float* __restrict__ part, const float* __restrict__ gamma,
                                const float* __restrict__ save_invstd,
                                float* __restrict__ dgamma, float* __restrict__ dbeta,
                                int accumulate, float* __restrict__ coef) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    double s1 = 0.0, s2 = 0.0;
    for (int i = 0; i < slices; ++i) {
        s1 += (double)part[((int64_t)c * slices + i) * 2];
        s2 += (double)part[((int64_t)c * slices + i) * 2 + 1];
    }
    const double invstd = save_invstd[c];
    const double db = s1, dg = s2 * invstd;
    dbeta[c] = (float)(accumulate ? (double)dbeta[c] + db : db);
    dgamma[c] = (float)(accumulate ? (double)dgamma[c] + dg : dg);
    const double M = (double)N * (double)V;
    // dx = k * (g - db/M - (x - mean) * invstd * dg/M)
    const double k = (double)gamma[c] * invstd;
    coef[c] = (float)k;
    coef[C + c] = (float)(db / M);
    coef[2 * C + c] = (float)(invstd * dg / M);
}

// DRES: 0 no residual gradient, 1 dres = g, 2 dres += g (one rounding).
template <typename T, int VEC, int MASK, int DRES>
__global__ __launch_bounds__(kBnThreads) void bn_bwd_apply(
    const T* __restrict__ dy, const T* __restrict__ x, const T* __restrict__ y, int C, int64_t V,
    unsigned cpp, const float* __restrict__ save_mean, const float* __restrict__ fcoef,
    const float* __restrict__ coef, T* __restrict__ dx, T* __restrict__ dres) {
    const int plane = (int)(blockIdx.x / cpp);  // wave-uniform
    const int64_t e = ((int64_t)(blockIdx.x - (unsigned)plane * cpp) * kBnThreads + threadIdx.x) * VEC;
    if (e >= V) return;
    const int c = plane % C;
    const int64_t i = (int64_t)plane * V + e;
    const float k = coef[c], a = coef[C + c], b = coef[2 * C + c], mean = save_mean[c];
    float g[VEC], xv[VEC];
    vload<T, VEC>(dy + i, g);
    vload<T, VEC>(x + i, xv);
    if constexpr (MASK == kMaskY) {
        float yv[VEC];
        vload<T, VEC>(y + i, yv);
#pragma unroll
        for (int j = 0; j < VEC; ++j) g[j] = yv[j] > 0.f ? g[j] : 0.f;
    } else if constexpr (MASK == kMaskX) {
        const float fsc = fcoef[c], fsh = fcoef[C + c];
#pragma unroll
        for (int j = 0; j < VEC; ++j) g[j] = fmaf(xv[j], fsc, fsh) > 0.f ? g[j] : 0.f;
    }
    if constexpr (DRES == 1) vstore<T, VEC>(dres + i, g);
    if constexpr (DRES == 2) {
        float o[VEC];
        vload<T, VEC>(dres + i, o);
#pragma unroll
        for (int j = 0; j < VEC; ++j) o[j] += g[j];
        vstore<T, VEC>(dres + i, o);
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) xv[j] = k * (g[j] - a - (xv[j] - mean) * b);
    vstore<T, VEC>(dx + i, xv);
}

// ---------------------------------------------------------------- launchers
template <typename T, int VEC>
static rat3d_status bn_fwd_t(const BnGeom& g, int relu, float eps, float momentum, const T* x,
                             const T* r, const float* gamma, const float* beta, T* y,
                             float* save_mean, float* save_invstd, float* run_mean,
                             float* run_var, float* save_coef, void* ws, hipStream_t st) {
    const BnSlices sl = bn_slices(g);
    float* part = (float*)ws;
    float* coef = part + (size_t)g.C * sl.per_channel * 2;
    const double tb = (double)g.N * g.C * g.V * sizeof(T);
    {
    ProfScope ps("bn_fwd_stats", st, 0.0, tb);
    bn_fwd_stats<T, VEC><<<dim3(g.C, sl.per_channel), kBnThreads, 0, st>>>(
        x, g.C, g.V, sl.per_plane, sl.len, part);
    RAT3D_LAUNCH_CHECK();
    }
    bn_fwd_finalize<T><<<(unsigned)ceil_div(g.C, 64), 64, 0, st>>>(
        x, g.N, g.C, g.V, sl.per_channel, part, gamma, beta, eps, momentum, save_mean,
        save_invstd, run_mean, run_var, coef, save_coef);
    RAT3D_LAUNCH_CHECK();
    const unsigned cpp = (unsigned)ceil_div(g.V / VEC, kBnThreads);  // chunks per plane
    const unsigned grid = cpp * (unsigned)(g.N * g.C);
    ProfScope ps("bn_fwd_apply", st, 0.0, tb * (r ? 3 : 2));
    if (relu && r)
        bn_fwd_apply<T, VEC, true, true><<<grid, kBnThreads, 0, st>>>(x, r, g.C, g.V, cpp, coef, y);
    else if (relu)
        bn_fwd_apply<T, VEC, true, false><<<grid, kBnThreads, 0, st>>>(x, r, g.C, g.V, cpp, coef, y);
    else if (r)
        bn_fwd_apply<T, VEC, false, true><<<grid, kBnThreads, 0, st>>>(x, r, g.C, g.V, cpp, coef, y);
    else
        bn_fwd_apply<T, VEC, false, false><<<grid, kBnThreads, 0, st>>>(x, r, g.C, g.V, cpp, coef, y);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

template <typename T, int VEC>
static rat3d_status bn_bwd_t(const BnGeom& g, int relu, const T* dy, const T* x, const T* y,
                             const float* gamma, const float* save_mean,
                             const float* save_invstd, const float* fwd_coef, T* dx, T* dres,
                             int dres_acc, float* dgamma, float* dbeta, int accumulate, void* ws,
                             hipStream_t st) {
    const BnSlices sl = bn_slices(g);
    float* part = (float*)ws;
    float* coef = part + (size_t)g.C * sl.per_channel * 2;
    const dim3 sg(g.C, sl.per_channel);
    const double tb = (double)g.N * g.C * g.V * sizeof(T);
    const int mask = !relu ? kMaskNone : (fwd_coef ? kMaskX : kMaskY);
    {
    ProfScope ps("bn_bwd_stats", st, 0.0, tb * (mask == kMaskY ? 3 : 2));
#define RAT3D_BN_ST(M)                                                                       \
    bn_bwd_stats<T, VEC, M><<<sg, kBnThreads, 0, st>>>(dy, x, y, g.C, g.V, sl.per_plane,     \
                                                       sl.len, save_mean, fwd_coef, part)
    if (mask == kMaskY) RAT3D_BN_ST(kMaskY);
    else if (mask == kMaskX) RAT3D_BN_ST(kMaskX);
    else RAT3D_BN_ST(kMaskNone);
#undef RAT3D_BN_ST
    RAT3D_LAUNCH_CHECK();
    }
    bn_bwd_finalize<<<(unsigned)ceil_div(g.C, 64), 64, 0, st>>>(
        g.N, g.C, g.V, sl.per_channel, part, gamma, save_invstd, dgamma, dbeta, accumulate, coef);
    RAT3D_LAUNCH_CHECK();
    const unsigned cpp = (unsigned)ceil_div(g.V / VEC, kBnThreads);  // chunks per plane
    const unsigned grid = cpp * (unsigned)(g.N * g.C);
    ProfScope ps("bn_bwd_apply", st, 0.0,
                 tb * ((mask == kMaskY ? 4 : 3) + (dres ? (dres_acc ? 2 : 1) : 0)));
#define RAT3D_BN_BWD(M, D)                                                                 \
    bn_bwd_apply<T, VEC, M, D><<<grid, kBnThreads, 0, st>>>(dy, x, y, g.C, g.V, cpp,      \
                                                            save_mean, fwd_coef, coef, dx, dres)
    const int dmode = dres ? (dres_acc ? 2 : 1) : 0;
    if (mask == kMaskY && dmode == 2) RAT3D_BN_BWD(kMaskY, 2);
    else if (mask == kMaskY && dmode == 1) RAT3D_BN_BWD(kMaskY, 1);
    else if (mask == kMaskY) RAT3D_BN_BWD(kMaskY, 0);
    else if (mask == kMaskX && dmode == 2) RAT3D_BN_BWD(kMaskX, 2);
    else if (mask == kMaskX && dmode == 1) RAT3D_BN_BWD(kMaskX, 1);
    else if (mask == kMaskX) RAT3D_BN_BWD(kMaskX, 0);
    else if (dmode == 2) RAT3D_BN_BWD(kMaskNone, 2);
    else if (dmode == 1) RAT3D_BN_BWD(kMaskNone, 1);
    else RAT3D_BN_BWD(kMaskNone, 0);
#undef RAT3D_BN_BWD
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status bn_fwd(const BnGeom& g, rat3d_dtype dt, int relu, float eps, float momentum,
                    const void* x, const void* residual, const float* gamma, const float* beta,
                    void* y, float* save_mean, float* save_invstd, float* run_mean,
                    float* run_var, float* save_coef, void* ws, hipStream_t st) {
    if (dt == RAT3D_BF16) {
        if (g.V % 8 == 0)
            return bn_fwd_t<bf16, 8>(g, relu, eps, momentum, (const bf16*)x, (const bf16*)residual,
                                     gamma, beta, (bf16*)y, save_mean, save_invstd, run_mean,
                                     run_var, save_coef, ws, st);
        return bn_fwd_t<bf16, 1>(g, relu, eps, momentum, (const bf16*)x, (const bf16*)residual,
                                 gamma, beta, (bf16*)y, save_mean, save_invstd, run_mean, run_var,
                                 save_coef, ws, st);
    }
    if (g.V % 4 == 0)
        return bn_fwd_t<float, 4>(g, relu, eps, momentum, (const float*)x, (const float*)residual,
                                  gamma, beta, (float*)y, save_mean, save_invstd, run_mean,
                                  run_var, save_coef, ws, st);
    return bn_fwd_t<float, 1>(g, relu, eps, momentum, (const float*)x, (const float*)residual,
                              gamma, beta, (float*)y, save_mean, save_invstd, run_mean, run_var,
                              save_coef, ws, st);
}

rat3d_status bn_bwd(const BnGeom& g, rat3d_dtype dt, int relu, const void* dy, const void* x,
                    const void* y, const float* gamma, const float* save_mean,
                    const float* save_invstd, const float* fwd_coef, void* dx, void* dres,
                    int dres_acc, float* dgamma, float* dbeta, int accumulate, void* ws,
                    hipStream_t st) {
    if (dt == RAT3D_BF16) {
        if (g.V % 8 == 0)
            return bn_bwd_t<bf16, 8>(g, relu, (const bf16*)dy, (const bf16*)x, (const bf16*)y,
                                     gamma, save_mean, save_invstd, fwd_coef, (bf16*)dx,
                                     (bf16*)dres, dres_acc, dgamma, dbeta, accumulate, ws, st);
        return bn_bwd_t<bf16, 1>(g, relu, (const bf16*)dy, (const bf16*)x, (const bf16*)y, gamma,
                                 save_mean, save_invstd, fwd_coef, (bf16*)dx, (bf16*)dres,
                                 dres_acc, dgamma, dbeta, accumulate, ws, st);
    }
    if (g.V % 4 == 0)
        return bn_bwd_t<float, 4>(g, relu, (const float*)dy, (const float*)x, (const float*)y,
                                  gamma, save_mean, save_invstd, fwd_coef, (float*)dx,
                                  (float*)dres, dres_acc, dgamma, dbeta, accumulate, ws, st);
    return bn_bwd_t<float, 1>(g, relu, (const float*)dy, (const float*)x, (const float*)y, gamma,
                              save_mean, save_invstd, fwd_coef, (float*)dx, (float*)dres,
                              dres_acc, dgamma, dbeta, accumulate, ws, st);
}

}  // namespace rat3d
