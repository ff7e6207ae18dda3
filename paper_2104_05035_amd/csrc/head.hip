// Classifier head (global average pool -> FC -> softmax cross-entropy, with
// its backward), the SGD update, and small fill/cast kernels.
#include "common.hpp"
#include "kernels.hpp"
#include "prof.hpp"

namespace rat3d {

// Workspace: g [N][C] pooled features, dl [N][classes] logit gradients.
size_t head_ws_bytes(int N, int C, int classes) {
    return ((size_t)N * C + (size_t)N * classes) * sizeof(float);
}

template <typename T>
__global__ __launch_bounds__(256) void gap_k(const T* __restrict__ x, int64_t V,
                                             float* __restrict__ g) {
    __shared__ float red[256];
    const T* p = x + (int64_t)blockIdx.x * V;
    float s = 0.f;
    for (int64_t i = threadIdx.x; i < V; i += 256) s += Elt<T>::ld(p + i);
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) g[blockIdx.x] = red[0] / (float)V;
}

// One block: logits, loss, logit gradients, FC gradients.
__global__ __launch_bounds__(256) void fc_ce_k(const float* __restrict__ g, int N, int C,
                                               int classes, const float* __restrict__ w,
                                               const float* __restrict__ b,
                                               const int32_t* __restrict__ labels,
                                               float* __restrict__ logits,
                                               float* __restrict__ loss, float* __restrict__ dl,
                                               float* __restrict__ dw, float* __restrict__ db,
                                               int accumulate) {
    __shared__ float lg[256];
    __shared__ float ls[256];
    __shared__ float sdl[256];
    const int t = threadIdx.x;
    if (t < N * classes) {
        const int n = t / classes, j = t - n * classes;
        float s = b[j];
        for (int c = 0; c < C; ++c) s += w[j * C + c] * g[n * C + c];
        lg[t] = s;
        logits[t] = s;
    }
    __syncthreads();
    if (t < N) {
        // labels outside [0, classes) are clamped into range
        const int lab = min(max((int)labels[t], 0), classes - 1);
        float mx = lg[t * classes];
        for (int j = 1; j < classes; ++j) mx = fmaxf(mx, lg[t * classes + j]);
        float se = 0.f;
        for (int j = 0; j < classes; ++j) se += expf(lg[t * classes + j] - mx);
        const float lse = mx + logf(se);
        ls[t] = lse - lg[t * classes + lab];
        for (int j = 0; j < classes; ++j) {
            const float sm = expf(lg[t * classes + j] - lse);
            const float d = (sm - (j == lab ? 1.f : 0.f)) / (float)N;
            sdl[t * classes + j] = d;
            dl[t * classes + j] = d;
        }
    }
    __syncthreads();
    if (t == 0) {
        float s = 0.f;
        for (int n = 0; n < N; ++n) s += ls[n];
        *loss = s / (float)N;
    }
    // dW[j][c] = sum_n dl[n][j] g[n][c];  db[j] = sum_n dl[n][j]
    for (int e = t; e < classes * C; e += 256) {
        const int j = e / C, c = e - j * C;
        float s = 0.f;
        for (int n = 0; n < N; ++n) s += sdl[n * classes + j] * g[n * C + c];
        dw[e] = accumulate ? dw[e] + s : s;
    }
    if (t < classes) {
        float s = 0.f;
        for (int n = 0; n < N; ++n) s += sdl[n * classes + t];
        db[t] = accumulate ? db[t] + s : s;
    }
}

// dx[n][c][v] = (sum_j dl[n][j] w[j][c]) / V
template <typename T>
__global__ __launch_bounds__(256) void gap_bwd_k(const float* __restrict__ dl,
                                                 const float* __restrict__ w, int C, int classes,
                                                 int64_t V, int64_t total, T* __restrict__ dx) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int64_t nc = i / V;
    const int n = (int)(nc / C), c = (int)(nc - (int64_t)n * C);
    float s = 0.f;
    for (int j = 0; j < classes; ++j) s += dl[n * classes + j] * w[j * C + c];
    Elt<T>::st(dx + i, s / (float)V);
}

__global__ void sgd_k(int64_t count, float lr, float* __restrict__ p,
                      const float* __restrict__ g) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < count) p[i] = __fmaf_rn(-lr, g[i], p[i]);  // one rounding of p - lr*g
}

__global__ void cast_k(int64_t count, const float* __restrict__ s, bf16* __restrict__ d) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < count) d[i] = f2bf(s[i]);
}

__global__ void fill_k(int64_t count, float v, float* __restrict__ d) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < count) d[i] = v;
}

rat3d_status head_fwd_bwd(int N, int C, int64_t V, int classes, rat3d_dtype dt, const void* x,
                          const float* fc_w, const float* fc_b, const int32_t* labels,
                          float* logits, float* loss, void* dx, float* dfc_w, float* dfc_b,
                          int accumulate, void* ws, hipStream_t st) {
    float* g = (float*)ws;
    float* dl = g + (size_t)N * C;
    if (dt == RAT3D_BF16) gap_k<bf16><<<N * C, 256, 0, st>>>((const bf16*)x, V, g);
    else gap_k<float><<<N * C, 256, 0, st>>>((const float*)x, V, g);
    RAT3D_LAUNCH_CHECK();
    fc_ce_k<<<1, 256, 0, st>>>(g, N, C, classes, fc_w, fc_b, labels, logits, loss, dl, dfc_w,
                               dfc_b, accumulate);
    RAT3D_LAUNCH_CHECK();
    const int64_t total = (int64_t)N * C * V;
    const unsigned blocks = (unsigned)ceil_div(total, 256);
    if (dt == RAT3D_BF16)
        gap_bwd_k<bf16><<<blocks, 256, 0, st>>>(dl, fc_w, C, classes, V, total, (bf16*)dx);
    else
        gap_bwd_k<float><<<blocks, 256, 0, st>>>(dl, fc_w, C, classes, V, total, (float*)dx);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status sgd_update(int64_t count, float lr, float* params, const float* grads,
                        hipStream_t st) {
    if (count == 0) return RAT3D_OK;
    ProfScope ps("sgd", st, 0.0, 12.0 * count);
    sgd_k<<<(unsigned)ceil_div(count, 256), 256, 0, st>>>(count, lr, params, grads);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status cast_f32_bf16(int64_t count, const float* src, bf16* dst, hipStream_t st) {
    if (count == 0) return RAT3D_OK;
    ProfScope ps("cast", st, 0.0, 6.0 * count);
    cast_k<<<(unsigned)ceil_div(count, 256), 256, 0, st>>>(count, src, dst);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status fill_f32(int64_t count, float value, float* dst, hipStream_t st) {
    if (count == 0) return RAT3D_OK;
    fill_k<<<(unsigned)ceil_div(count, 256), 256, 0, st>>>(count, value, dst);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace rat3d
