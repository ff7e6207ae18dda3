// Per-channel batch-norm coefficients from the statistics partials, for the
// apply kernels (batch norm's own and the fused ones of the soft-mask branch).
// Every wave that needs a channel's coefficients combines the channel's
// partials itself, in one fixed order, so all of them get the same bits; the
// one wave told it is the owner also stores the per-channel outputs.
#pragma once

#include "common.hpp"

namespace rat3d {

// Sums the slice partial pairs of channel c in float64 in a fixed order:
// lane l adds slices l, l + 64, ... in turn, then an xor butterfly over the
// wave; every lane of every wave ends with the same bits (each butterfly
// level adds the same pairs of values, and float addition commutes).  All
// 64 lanes must be active.
__device__ __forceinline__ void wave_sum_partials(const float* __restrict__ part, int c,
                                                  int slices, double& s1, double& s2) {
    const int lane = (int)(threadIdx.x & 63);
    const float2* pc = reinterpret_cast<const float2*>(part + (int64_t)c * slices * 2);
    double a = 0.0, b = 0.0;
    // four loads in flight per lane; slices past the end add nothing
    for (int i = lane; i < slices; i += 256) {
        float2 q[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) q[u] = pc[i + 64 * u < slices ? i + 64 * u : i];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const bool in = i + 64 * u < slices;
            a += in ? (double)q[u].x : 0.0;
            b += in ? (double)q[u].y : 0.0;
        }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        a += __shfl_xor(a, m, 64);
        b += __shfl_xor(b, m, 64);
    }
    s1 = a;
    s2 = b;
}

// Per channel: combine the slice partials in a fixed order in float64 into
// the apply coefficients (scale, shift).  Every apply block of the channel
// evaluates this identically; the block given `owner` also stores mean,
// invstd, the coefficients and the running statistics.
__device__ __forceinline__ void bn_fwd_coefs(int N, int C, int64_t V,
                                             int slices, int c, const float* __restrict__ part,
                                             const float* __restrict__ gamma,
                                             const float* __restrict__ beta, float eps,
                                             float momentum, bool owner,
                                             float* __restrict__ save_mean,
                                             float* __restrict__ save_invstd,
                                             float* __restrict__ run_mean,
                                             float* __restrict__ run_var,
                                             float* __restrict__ save_coef, float& scale,
                                             float& bias) {
    const double shift = (double)part[(int64_t)C * slices * 2 + c];
    double s1, s2;
    wave_sum_partials(part, c, slices, s1, s2);
    const double M = (double)N * (double)V;
    const double dm = s1 / M;
    double var = s2 / M - dm * dm;
    if (var < 0.0) var = 0.0;
    const double mean = shift + dm;
    const double invstd = 1.0 / sqrt(var + (double)eps);
    scale = (float)((double)gamma[c] * invstd);
    bias = (float)((double)beta[c] - mean * (double)scale);
    if (!owner) return;
    save_mean[c] = (float)mean;
    save_invstd[c] = (float)invstd;
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

struct BnFwdStats {
    const float* part;
    int slices;
    const float* gamma;
    const float* beta;
    float eps, momentum;
    float *save_mean, *save_invstd, *run_mean, *run_var, *save_coef;
};

struct BnBwdStats {
    const float* part;
    int slices;
    const float* gamma;
    const float* save_invstd;
    float *dgamma, *dbeta;
    int accumulate;
};

// Per channel: dbeta, dgamma and the apply coefficients from the slice
// partials (fixed order, float64).  Every apply block of the channel
// evaluates this identically; the block given `owner` stores dgamma, dbeta.
__device__ __forceinline__ void bn_bwd_coefs(int N, int64_t V, int c, const BnBwdStats& st,
                                             bool owner, float& k, float& a, float& b) {
    double s1, s2;
    wave_sum_partials(st.part, c, st.slices, s1, s2);
    const double invstd = st.save_invstd[c];
    const double db = s1, dg = s2 * invstd;
    if (owner) {
        st.dbeta[c] = (float)(st.accumulate ? (double)st.dbeta[c] + db : db);
        st.dgamma[c] = (float)(st.accumulate ? (double)st.dgamma[c] + dg : dg);
    }
    const double M = (double)N * (double)V;
    // dx = k * (g - db/M - (x - mean) * invstd * dg/M)
    k = (float)((double)st.gamma[c] * invstd);
    a = (float)(db / M);
    b = (float)(invstd * dg / M);
}

}  // namespace rat3d
