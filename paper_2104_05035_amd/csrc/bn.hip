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
// Step (2) runs at the start of every block of step (3): each block combines
// its channel's partials itself (the same fixed order everywhere, so every
// block gets the same coefficients) and one block per channel stores the
// per-channel outputs -- no separate per-channel kernel between the passes.
//           dresidual = g (or dresidual += g, one rounding).  Without a residual, y > 0 is the same test as
//           x * scale + shift > 0 with the forward's own float coefficients
//           (the apply computes exactly that value before the max with 0), so
//           given those coefficients the backward reads x instead of x and y.
// NCDHW: one (n, c) plane is V contiguous voxels; a slice is a contiguous
// segment of one plane, so per-element indexing needs no division.  A
// channel's partials are the N * SP segment sums of its planes, combined in
// a fixed order.  Everything is HBM-bound: loads and stores are 16-byte
// vectors when V allows.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "vec.hpp"
#include "prof.hpp"
#include "bn_coef.hpp"

namespace rat3d {

constexpr int kBnThreads = 256;
constexpr int kStatsUnroll = 4;  // vectors per tensor in flight per thread in the statistics passes
// vectors per thread in the apply passes, measured per variant: the two-stream
// forward apply (least work per wave to hide its coefficient reduction
// behind) and the one that also reduces its residual's BN coefficients gain
// from four; the plain residual apply runs best with one
template <int RES> constexpr int fwd_apply_u() { return RES == 1 ? 1 : 4; }
constexpr int kBwdApplyU = 1;

struct BnSlices {
    int per_plane;    // segments per (n, c) plane
    int per_channel;  // N * per_plane partials per channel
    int64_t len;      // elements per segment (multiple of the vector width)
};

static BnSlices bn_slices(const BnGeom& g) {
    // many short segments stream faster than a few long ones (measured on
    // 264 MB reads): aim for ~16K blocks of at least ~8K elements
    int64_t want = ceil_div(16384, (int64_t)g.C * g.N);
    int64_t by_size = ceil_div(g.V, 8192);
    int64_t s = want < by_size ? want : by_size;
    if (s < 1) s = 1;
    int64_t len = ceil_div(g.V, s);
    len = ceil_div(len, 8) * 8;
    s = ceil_div(g.V, len);
    return BnSlices{(int)s, (int)(s * g.N), len};
}

size_t bn_ws_bytes(const BnGeom& g) {
    const BnSlices sl = bn_slices(g);
    // partial pairs (2 floats per slice) + the forward's shift per channel
    return ((size_t)g.C * sl.per_channel * 2 + (size_t)g.C) * sizeof(float);
}

// Block reduction of two floats; result valid in thread 0.  Each wave sums
// its lanes with an xor butterfly, then thread 0 adds the four wave sums in
// order: one barrier instead of a shared-memory tree (a fixed order).
__device__ __forceinline__ void block_sum2(float& a, float& b) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        a += __shfl_xor(a, m, 64);
        b += __shfl_xor(b, m, 64);
    }
    __shared__ float ra[kBnThreads / 64], rb[kBnThreads / 64];
    if ((threadIdx.x & 63) == 0) {
        ra[threadIdx.x >> 6] = a;
        rb[threadIdx.x >> 6] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a = ra[0];
        b = rb[0];
#pragma unroll
        for (int w = 1; w < kBnThreads / 64; ++w) {
            a += ra[w];
            b += rb[w];
        }
    }
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
    constexpr int64_t kStep = (int64_t)kBnThreads * VEC;
    // kStatsUnroll vectors in flight per thread; vectors past the segment end
    // load its last vector (clamped address, cnt % VEC == 0) and add nothing
    for (int64_t e = (int64_t)threadIdx.x * VEC; e < cnt; e += kStatsUnroll * kStep) {
        float v[kStatsUnroll][VEC];
#pragma unroll
        for (int u = 0; u < kStatsUnroll; ++u) {
            const int64_t eu = e + u * kStep;
            vload<T, VEC>(p + (eu < cnt ? eu : cnt - VEC), v[u]);
        }
#pragma unroll
        for (int u = 0; u < kStatsUnroll; ++u) {
            const bool in = e + u * kStep < cnt;
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                const float d = in ? v[u][j] - shift : 0.f;
                s1 += d;
                s2 += d * d;
            }
        }
    }
    block_sum2(s1, s2);
    if (threadIdx.x == 0) {
        float* o = part + ((int64_t)c * gridDim.y + sidx) * 2;
        o[0] = s1;
        o[1] = s2;
        // the shift, kept beside the partials so the apply never reads x for
        // it (x may be overwritten by an in-place apply)
        if (sidx == 0) part[(int64_t)C * gridDim.y * 2 + c] = shift;
    }
}


// One-dimensional grid: block b covers chunk b % cpp of plane b / cpp.  The
// block first loads its elements, then derives its channel's coefficients
// from the statistics partials (the first chunk of plane (0, c) stores them).
// RES: 0 no residual, 1 y += r, 2 y += BN_r(r) with the residual's own batch
// norm (no ReLU) formed here from its statistics partials `rst` and rounded as
// its own apply would store it.
template <typename T, int VEC, bool RELU, int RES>
__global__ __launch_bounds__(kBnThreads) void bn_fwd_apply(const T* __restrict__ x,
                                                           const T* __restrict__ r, int N, int C,
                                                           int64_t V, unsigned cpp,
                                                           BnFwdStats st, T* __restrict__ y,
                                                           uint8_t* __restrict__ ybits,
                                                           BnFwdStats rst) {
    constexpr int U = fwd_apply_u<RES>();
    constexpr int64_t kStep = (int64_t)kBnThreads * VEC;
    const int plane = (int)(blockIdx.x / cpp);  // wave-uniform
    const unsigned chunk = blockIdx.x - (unsigned)plane * cpp;
    const int64_t e0 = (int64_t)chunk * kStep * U + (int64_t)threadIdx.x * VEC;
    const int c = plane % C;
    const int64_t base = (int64_t)plane * V;
    // every vector is loaded before the coefficients are formed; vectors past
    // the end load the plane's last vector (V % VEC == 0), so every lane takes
    // part in the coefficient reduction, and store nothing
    float v[U][VEC];
    [[maybe_unused]] float rv[U][VEC];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t e = e0 + u * kStep;
        const int64_t i = base + (e < V ? e : V - VEC);
        vload<T, VEC>(x + i, v[u]);
        if constexpr (RES) vload<T, VEC>(r + i, rv[u]);
    }
    float sc, sh;
    const bool owner = plane < C && chunk == 0 && threadIdx.x == 0;
    bn_fwd_coefs(N, C, V, st.slices, c, st.part, st.gamma, st.beta, st.eps, st.momentum, owner,
                 st.save_mean, st.save_invstd, st.run_mean, st.run_var, st.save_coef, sc, sh);
    [[maybe_unused]] float rsc = 1.f, rsh = 0.f;
    if constexpr (RES == 2)
        bn_fwd_coefs(N, C, V, rst.slices, c, rst.part, rst.gamma, rst.beta, rst.eps,
                     rst.momentum, owner, rst.save_mean, rst.save_invstd, rst.run_mean,
                     rst.run_var, rst.save_coef, rsc, rsh);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t e = e0 + u * kStep;
        if (e >= V) break;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            float o = fmaf(v[u][j], sc, sh);
            if constexpr (RES == 1) o += rv[u][j];
            if constexpr (RES == 2) o += Elt<T>::round(fmaf(rv[u][j], rsc, rsh));
            if constexpr (RELU) o = fmaxf(o, 0.f);
            v[u][j] = o;
        }
        if constexpr (sizeof(T) == 2 && VEC == 8) {
            if (ybits) {
                // the stored bf16 values, and bit j = (y_j > 0) of them
                uint32_t w[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) w[q] = pack_bf16x2(v[u][2 * q], v[u][2 * q + 1]);
                *reinterpret_cast<uint4*>(y + base + e) = make_uint4(w[0], w[1], w[2], w[3]);
                uint32_t byte = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    byte |= ((int16_t)(w[q] & 0xffffu) > 0 ? 1u : 0u) << (2 * q);
                    byte |= ((int16_t)(w[q] >> 16) > 0 ? 1u : 0u) << (2 * q + 1);
                }
                ybits[(base + e) >> 3] = (uint8_t)byte;
                continue;
            }
        }
        vstore<T, VEC>(y + base + e, v[u]);
    }
}

// ReLU mask of the backward: none, y > 0, x * scale + shift > 0, or the
// forward's y > 0 bits (bf16, VEC 8: one byte per vector).
enum { kMaskNone = 0, kMaskY = 1, kMaskX = 2, kMaskBits = 3 };

bool bn_bits_ok(const BnGeom& g, rat3d_dtype dt) { return dt == RAT3D_BF16 && g.V % 8 == 0; }

template <typename T, int VEC, int MASK>
__global__ __launch_bounds__(kBnThreads) void bn_bwd_stats(const T* __restrict__ dy,
                                                           const T* __restrict__ x,
                                                           const T* __restrict__ y,
                                                           const uint8_t* __restrict__ ybits,
                                                           int C, int64_t V, int SP, int64_t len,
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
    // kStatsUnroll vectors of each tensor in flight per thread, all loads
    // issued before any is used; past the segment end the last vector is
    // loaded (clamped) and adds nothing
    constexpr int64_t kStep = (int64_t)kBnThreads * VEC;
    constexpr int U = kStatsUnroll;
    for (int64_t e = (int64_t)threadIdx.x * VEC; e < cnt; e += U * kStep) {
        float g[U][VEC], xv[U][VEC];
        [[maybe_unused]] float yv[U][VEC];
        [[maybe_unused]] uint32_t yb[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t eu = e + u * kStep;
            const int64_t idx = base + (eu < cnt ? eu : cnt - VEC);
            vload<T, VEC>(dy + idx, g[u]);
            vload<T, VEC>(x + idx, xv[u]);
            if constexpr (MASK == kMaskY) vload<T, VEC>(y + idx, yv[u]);
            if constexpr (MASK == kMaskBits) yb[u] = ybits[idx >> 3];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool in = e + u * kStep < cnt;
            if constexpr (MASK == kMaskY) {
#pragma unroll
                for (int j = 0; j < VEC; ++j) g[u][j] = yv[u][j] > 0.f ? g[u][j] : 0.f;
            } else if constexpr (MASK == kMaskBits) {
#pragma unroll
                for (int j = 0; j < VEC; ++j) g[u][j] = (yb[u] >> j) & 1u ? g[u][j] : 0.f;
            } else if constexpr (MASK == kMaskX) {
#pragma unroll
                for (int j = 0; j < VEC; ++j) g[u][j] = fmaf(xv[u][j], fsc, fsh) > 0.f ? g[u][j] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                const float gj = in ? g[u][j] : 0.f;
                s1 += gj;
                s2 += gj * (xv[u][j] - mean);
            }
        }
    }
    block_sum2(s1, s2);
    if (threadIdx.x == 0) {
        float* o = part + ((int64_t)c * gridDim.y + sidx) * 2;
        o[0] = s1;
        o[1] = s2;
    }
}

// DRES: 0 no residual gradient, 1 dres = g, 2 dres += g (one rounding).
template <typename T, int VEC, int MASK, int DRES>
__global__ __launch_bounds__(kBnThreads) void bn_bwd_apply(
    const T* __restrict__ dy, const T* __restrict__ x, const T* __restrict__ y,
    const uint8_t* __restrict__ ybits, int N, int C, int64_t V, unsigned cpp,
    const float* __restrict__ save_mean, const float* __restrict__ fcoef, BnBwdStats st,
    T* __restrict__ dx, T* __restrict__ dres) {
    constexpr int U = kBwdApplyU;
    constexpr int64_t kStep = (int64_t)kBnThreads * VEC;
    const int plane = (int)(blockIdx.x / cpp);  // wave-uniform
    const unsigned chunk = blockIdx.x - (unsigned)plane * cpp;
    const int64_t e0 = (int64_t)chunk * kStep * U + (int64_t)threadIdx.x * VEC;
    const int c = plane % C;
    const int64_t base = (int64_t)plane * V;
    // as in the forward apply: every load first (clamped), every lane in the
    // coefficient reduction
    float g[U][VEC], xv[U][VEC];
    [[maybe_unused]] float yv[U][VEC], ov[U][VEC];
    [[maybe_unused]] uint32_t yb[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t e = e0 + u * kStep;
        const int64_t i = base + (e < V ? e : V - VEC);
        vload<T, VEC>(dy + i, g[u]);
        vload<T, VEC>(x + i, xv[u]);
        if constexpr (MASK == kMaskY) vload<T, VEC>(y + i, yv[u]);
        if constexpr (MASK == kMaskBits) yb[u] = ybits[i >> 3];
        if constexpr (DRES == 2) vload<T, VEC>(dres + i, ov[u]);
    }
    float k, a, b;
    bn_bwd_coefs(N, V, c, st, plane < C && chunk == 0 && threadIdx.x == 0, k, a, b);
    const float mean = save_mean[c];
    [[maybe_unused]] const float fsc = MASK == kMaskX ? fcoef[c] : 0.f;
    [[maybe_unused]] const float fsh = MASK == kMaskX ? fcoef[C + c] : 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t e = e0 + u * kStep;
        if (e >= V) break;
        const int64_t i = base + e;
        if constexpr (MASK == kMaskY) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) g[u][j] = yv[u][j] > 0.f ? g[u][j] : 0.f;
        } else if constexpr (MASK == kMaskBits) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) g[u][j] = (yb[u] >> j) & 1u ? g[u][j] : 0.f;
        } else if constexpr (MASK == kMaskX) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) g[u][j] = fmaf(xv[u][j], fsc, fsh) > 0.f ? g[u][j] : 0.f;
        }
        if constexpr (DRES == 1) vstore<T, VEC>(dres + i, g[u]);
        if constexpr (DRES == 2) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) ov[u][j] += g[u][j];
            vstore<T, VEC>(dres + i, ov[u]);
        }
#pragma unroll
        for (int j = 0; j < VEC; ++j) xv[u][j] = k * (g[u][j] - a - (xv[u][j] - mean) * b);
        vstore<T, VEC>(dx + i, xv[u]);
    }
}

// ---------------------------------------------------------------- launchers
template <typename T, int VEC>
static rat3d_status bn_fwd_t(const BnGeom& g, int relu, float eps, float momentum, const T* x,
                             const T* r, const float* gamma, const float* beta, T* y,
                             float* save_mean, float* save_invstd, float* run_mean,
                             float* run_var, float* save_coef, uint8_t* ybits, void* ws,
                             hipStream_t st) {
    const BnSlices sl = bn_slices(g);
    float* part = (float*)ws;
    const double tb = (double)g.N * g.C * g.V * sizeof(T);
    {
    ProfScope ps("bn_fwd_stats", st, 0.0, tb);
    bn_fwd_stats<T, VEC><<<dim3(g.C, sl.per_channel), kBnThreads, 0, st>>>(
        x, g.C, g.V, sl.per_plane, sl.len, part);
    RAT3D_LAUNCH_CHECK();
    }
    const BnFwdStats fs{part,     sl.per_channel, gamma,   beta,   eps,      momentum,
                        save_mean, save_invstd,   run_mean, run_var, save_coef};
    const int fu = r ? fwd_apply_u<1>() : fwd_apply_u<0>();
    const unsigned cpp = (unsigned)ceil_div(g.V / VEC, kBnThreads * fu);  // chunks per plane
    const unsigned grid = cpp * (unsigned)(g.N * g.C);
    ProfScope ps("bn_fwd_apply", st, 0.0, tb * (r ? 3 : 2) + (ybits ? tb / 16 : 0.0));
#define RAT3D_BN_FWD(RL, RS)                                                                 \
    bn_fwd_apply<T, VEC, RL, RS><<<grid, kBnThreads, 0, st>>>(x, r, g.N, g.C, g.V, cpp, fs, y, \
                                                              ybits, BnFwdStats{})
    if (relu && r) RAT3D_BN_FWD(true, 1);
    else if (relu) RAT3D_BN_FWD(true, 0);
    else if (r) RAT3D_BN_FWD(false, 1);
    else RAT3D_BN_FWD(false, 0);
#undef RAT3D_BN_FWD
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

template <typename T, int VEC>
static rat3d_status bn_bwd_t(const BnGeom& g, int relu, const T* dy, const T* x, const T* y,
                             const uint8_t* ybits, const float* gamma, const float* save_mean,
                             const float* save_invstd, const float* fwd_coef, T* dx, T* dres,
                             int dres_acc, float* dgamma, float* dbeta, int accumulate, void* ws,
                             hipStream_t st) {
    const BnSlices sl = bn_slices(g);
    float* part = (float*)ws;
    const dim3 sg(g.C, sl.per_channel);
    const double tb = (double)g.N * g.C * g.V * sizeof(T);
    const int mask = !relu ? kMaskNone : (fwd_coef ? kMaskX : (ybits ? kMaskBits : kMaskY));
    // bytes of the mask operand: y, its bits, or nothing
    const double mb = mask == kMaskY ? tb : (mask == kMaskBits ? tb / 16 : 0.0);
    {
    ProfScope ps("bn_bwd_stats", st, 0.0, tb * 2 + mb);
#define RAT3D_BN_ST(M)                                                                        \
    bn_bwd_stats<T, VEC, M><<<sg, kBnThreads, 0, st>>>(dy, x, y, ybits, g.C, g.V, sl.per_plane, \
                                                       sl.len, save_mean, fwd_coef, part)
    if (mask == kMaskY) RAT3D_BN_ST(kMaskY);
    else if (mask == kMaskX) RAT3D_BN_ST(kMaskX);
    else if (mask == kMaskBits) RAT3D_BN_ST(kMaskBits);
    else RAT3D_BN_ST(kMaskNone);
#undef RAT3D_BN_ST
    RAT3D_LAUNCH_CHECK();
    }
    const BnBwdStats bs{part, sl.per_channel, gamma, save_invstd, dgamma, dbeta, accumulate};
    const unsigned cpp = (unsigned)ceil_div(g.V / VEC, kBnThreads * kBwdApplyU);  // chunks per plane
    const unsigned grid = cpp * (unsigned)(g.N * g.C);
    ProfScope ps("bn_bwd_apply", st, 0.0,
                 tb * (3 + (dres ? (dres_acc ? 2 : 1) : 0)) + mb);
#define RAT3D_BN_BWD(M, D)                                                                    \
    bn_bwd_apply<T, VEC, M, D><<<grid, kBnThreads, 0, st>>>(dy, x, y, ybits, g.N, g.C, g.V, cpp, \
                                                            save_mean, fwd_coef, bs, dx, dres)
#define RAT3D_BN_BWD_M(M)                      \
    if (dmode == 2) RAT3D_BN_BWD(M, 2);        \
    else if (dmode == 1) RAT3D_BN_BWD(M, 1);   \
    else RAT3D_BN_BWD(M, 0);
    const int dmode = dres ? (dres_acc ? 2 : 1) : 0;
    if (mask == kMaskY) {
        RAT3D_BN_BWD_M(kMaskY)
    } else if (mask == kMaskX) {
        RAT3D_BN_BWD_M(kMaskX)
    } else if (mask == kMaskBits) {
        RAT3D_BN_BWD_M(kMaskBits)
    } else {
        RAT3D_BN_BWD_M(kMaskNone)
    }
#undef RAT3D_BN_BWD_M
#undef RAT3D_BN_BWD
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status bn_fwd(const BnGeom& g, rat3d_dtype dt, int relu, float eps, float momentum,
                    const void* x, const void* residual, const float* gamma, const float* beta,
                    void* y, float* save_mean, float* save_invstd, float* run_mean,
                    float* run_var, float* save_coef, uint8_t* ybits, void* ws, hipStream_t st) {
    if (ybits && !(relu && bn_bits_ok(g, dt))) {
        set_error("bn_fwd: y > 0 bits need bf16, a ReLU and V % 8 == 0");
        return RAT3D_EUNSUPPORTED;
    }
    if (dt == RAT3D_BF16) {
        if (g.V % 8 == 0)
            return bn_fwd_t<bf16, 8>(g, relu, eps, momentum, (const bf16*)x, (const bf16*)residual,
                                     gamma, beta, (bf16*)y, save_mean, save_invstd, run_mean,
                                     run_var, save_coef, ybits, ws, st);
        return bn_fwd_t<bf16, 1>(g, relu, eps, momentum, (const bf16*)x, (const bf16*)residual,
                                 gamma, beta, (bf16*)y, save_mean, save_invstd, run_mean, run_var,
                                 save_coef, nullptr, ws, st);
    }
    if (g.V % 4 == 0)
        return bn_fwd_t<float, 4>(g, relu, eps, momentum, (const float*)x, (const float*)residual,
                                  gamma, beta, (float*)y, save_mean, save_invstd, run_mean,
                                  run_var, save_coef, nullptr, ws, st);
    return bn_fwd_t<float, 1>(g, relu, eps, momentum, (const float*)x, (const float*)residual,
                              gamma, beta, (float*)y, save_mean, save_invstd, run_mean, run_var,
                              save_coef, nullptr, ws, st);
}

rat3d_status bn_bwd(const BnGeom& g, rat3d_dtype dt, int relu, const void* dy, const void* x,
                    const void* y, const uint8_t* ybits, const float* gamma,
                    const float* save_mean, const float* save_invstd, const float* fwd_coef,
                    void* dx, void* dres, int dres_acc, float* dgamma, float* dbeta,
                    int accumulate, void* ws, hipStream_t st) {
    if (ybits && !(relu && bn_bits_ok(g, dt))) {
        set_error("bn_bwd: y > 0 bits need bf16, a ReLU and V % 8 == 0");
        return RAT3D_EUNSUPPORTED;
    }
    if (dt == RAT3D_BF16) {
        if (g.V % 8 == 0)
            return bn_bwd_t<bf16, 8>(g, relu, (const bf16*)dy, (const bf16*)x, (const bf16*)y,
                                     ybits, gamma, save_mean, save_invstd, fwd_coef, (bf16*)dx,
                                     (bf16*)dres, dres_acc, dgamma, dbeta, accumulate, ws, st);
        return bn_bwd_t<bf16, 1>(g, relu, (const bf16*)dy, (const bf16*)x, (const bf16*)y,
                                 nullptr, gamma, save_mean, save_invstd, fwd_coef, (bf16*)dx,
                                 (bf16*)dres, dres_acc, dgamma, dbeta, accumulate, ws, st);
    }
    if (g.V % 4 == 0)
        return bn_bwd_t<float, 4>(g, relu, (const float*)dy, (const float*)x, (const float*)y,
                                  nullptr, gamma, save_mean, save_invstd, fwd_coef, (float*)dx,
                                  (float*)dres, dres_acc, dgamma, dbeta, accumulate, ws, st);
    return bn_bwd_t<float, 1>(g, relu, (const float*)dy, (const float*)x, (const float*)y,
                              nullptr, gamma, save_mean, save_invstd, fwd_coef, (float*)dx,
                              (float*)dres, dres_acc, dgamma, dbeta, accumulate, ws, st);
}

// ---------------------------------------------------------------- pieces for fused passes
// The backward statistics pass alone (bf16, V % 8 == 0, mask from x with the
// forward's coefficients); *bs receives what an apply done elsewhere needs.
rat3d_status bn_bwd_stats_x(const BnGeom& g, const void* dy, const void* x, const float* gamma,
                            const float* save_mean, const float* save_invstd,
                            const float* fwd_coef, float* dgamma, float* dbeta, int accumulate,
                            void* ws, hipStream_t st, BnBwdStats* bs) {
    if (g.V % 8 != 0 || !fwd_coef) {
        set_error("bn_bwd_stats_x: needs V %% 8 == 0 and the forward's coefficients");
        return RAT3D_EUNSUPPORTED;
    }
    const BnSlices sl = bn_slices(g);
    float* part = (float*)ws;
    const double tb = (double)g.N * g.C * g.V * sizeof(bf16);
    ProfScope ps("bn_bwd_stats", st, 0.0, tb * 2);
    bn_bwd_stats<bf16, 8, kMaskX><<<dim3(g.C, sl.per_channel), kBnThreads, 0, st>>>(
        (const bf16*)dy, (const bf16*)x, nullptr, nullptr, g.C, g.V, sl.per_plane, sl.len,
        save_mean, fwd_coef, part);
    RAT3D_LAUNCH_CHECK();
    *bs = BnBwdStats{part, sl.per_channel, gamma, save_invstd, dgamma, dbeta, accumulate};
    return RAT3D_OK;
}

size_t bn_max_slices(const BnGeom& g) { return (size_t)bn_slices(g).per_channel; }

// The forward apply (BN + ReLU, no residual, bf16, V % 8 == 0) from statistics
// partials someone else produced: `slices` pairs per channel at part, the
// shift of channel c at part[C * slices * 2 + c].
rat3d_status bn_fwd_apply_from(const BnGeom& g, float eps, float momentum, const void* x,
                               const float* gamma, const float* beta, void* y,
                               float* save_mean, float* save_invstd, float* run_mean,
                               float* run_var, float* save_coef, const float* part, int slices,
                               hipStream_t st) {
    if (g.V % 8 != 0) {
        set_error("bn_fwd_apply_from: needs V %% 8 == 0");
        return RAT3D_EUNSUPPORTED;
    }
    const BnFwdStats fs{part,     slices,      gamma,    beta,    eps,      momentum,
                        save_mean, save_invstd, run_mean, run_var, save_coef};
    const int fu = fwd_apply_u<0>();
    const unsigned cpp = (unsigned)ceil_div(g.V / 8, kBnThreads * fu);
    const unsigned grid = cpp * (unsigned)(g.N * g.C);
    const double tb = (double)g.N * g.C * g.V * sizeof(bf16);
    ProfScope ps("bn_fwd_apply", st, 0.0, tb * 2);
    bn_fwd_apply<bf16, 8, true, 0><<<grid, kBnThreads, 0, st>>>(
        (const bf16*)x, nullptr, g.N, g.C, g.V, cpp, fs, (bf16*)y, nullptr, BnFwdStats{});
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

// y = relu(BN(x) + BN_r(r)): the residual passes through its own batch norm
// (no ReLU) whose apply happens inside this one (bf16, V % 8 == 0); both
// statistics passes first, each into its own workspace (bn_ws_bytes each).
// The residual's BN stores its mean, invstd and running statistics as its own
// forward would; its normalised values are never stored.
rat3d_status bn_fwd_res_bn(const BnGeom& g, float eps, float momentum, const void* x,
                           const float* gamma, const float* beta, void* y, float* save_mean,
                           float* save_invstd, float* run_mean, float* run_var,
                           uint8_t* ybits, void* ws, const void* r, const float* rgamma,
                           const float* rbeta, float* rsave_mean, float* rsave_invstd,
                           float* rrun_mean, float* rrun_var, void* rws, hipStream_t st) {
    if (g.V % 8 != 0 || (ybits && !bn_bits_ok(g, RAT3D_BF16))) {
        set_error("bn_fwd_res_bn: needs V %% 8 == 0");
        return RAT3D_EUNSUPPORTED;
    }
    const BnSlices sl = bn_slices(g);
    const double tb = (double)g.N * g.C * g.V * sizeof(bf16);
    {
        ProfScope ps("bn_fwd_stats", st, 0.0, tb * 2);
        bn_fwd_stats<bf16, 8><<<dim3(g.C, sl.per_channel), kBnThreads, 0, st>>>(
            (const bf16*)x, g.C, g.V, sl.per_plane, sl.len, (float*)ws);
        RAT3D_LAUNCH_CHECK();
        bn_fwd_stats<bf16, 8><<<dim3(g.C, sl.per_channel), kBnThreads, 0, st>>>(
            (const bf16*)r, g.C, g.V, sl.per_plane, sl.len, (float*)rws);
        RAT3D_LAUNCH_CHECK();
    }
    const BnFwdStats fs{(const float*)ws, sl.per_channel, gamma,    beta,    eps,    momentum,
                        save_mean,        save_invstd,    run_mean, run_var, nullptr};
    const BnFwdStats rs{(const float*)rws, sl.per_channel, rgamma,    rbeta,    eps,    momentum,
                        rsave_mean,        rsave_invstd,   rrun_mean, rrun_var, nullptr};
    const unsigned cpp = (unsigned)ceil_div(g.V / 8, kBnThreads * fwd_apply_u<2>());
    const unsigned grid = cpp * (unsigned)(g.N * g.C);
    ProfScope ps("bn_fwd_apply", st, 0.0, tb * 3 + (ybits ? tb / 16 : 0.0));
    bn_fwd_apply<bf16, 8, true, 2><<<grid, kBnThreads, 0, st>>>(
        (const bf16*)x, (const bf16*)r, g.N, g.C, g.V, cpp, fs, (bf16*)y, ybits, rs);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace rat3d
