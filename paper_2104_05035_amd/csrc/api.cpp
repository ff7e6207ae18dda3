// C ABI of librat3d: argument validation and dispatch to the kernel
// launchers.  Nothing here allocates device memory.
#include <cstdarg>
#include <cstdio>
#include <string>

#include "kernels.hpp"

namespace rat3d {

int device_cus() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        cache[dev] = n;
    }
    return cache[dev];
}

}  // namespace rat3d

namespace rat3d {

static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
}

static rat3d_status fail(rat3d_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
static bool valid_dtype(rat3d_dtype d) { return d == RAT3D_F32 || d == RAT3D_BF16; }
static size_t esize(rat3d_dtype d) { return d == RAT3D_BF16 ? 2 : 4; }

#define RAT3D_REQUIRE(cond, st, ...) \
    do {                             \
        if (!(cond)) return fail(st, __VA_ARGS__); \
    } while (0)

#define RAT3D_ACT(p, name)                                                        \
    do {                                                                          \
        RAT3D_REQUIRE((p) != nullptr, RAT3D_EINVAL, "%s must not be NULL", name); \
        RAT3D_REQUIRE(aligned16(p), RAT3D_EALIGN, "%s must be 16-byte aligned", name); \
    } while (0)

static rat3d_status check_conv(const rat3d_conv3d_desc* d, ConvGeom* g) {
    RAT3D_REQUIRE(d != nullptr, RAT3D_EINVAL, "conv descriptor is NULL");
    RAT3D_REQUIRE(d->n >= 1 && d->c_in >= 1 && d->c_out >= 1 && d->d >= 1 && d->h >= 1 &&
                      d->w >= 1,
                  RAT3D_EINVAL, "conv sizes must be >= 1");
    RAT3D_REQUIRE(d->k >= 1 && d->stride >= 1 && d->pad >= 0 && d->pad < d->k, RAT3D_EINVAL,
                  "conv needs k >= 1, stride >= 1, 0 <= pad < k (k=%d stride=%d pad=%d)", d->k,
                  d->stride, d->pad);
    RAT3D_REQUIRE(valid_dtype(d->dtype), RAT3D_EUNSUPPORTED, "unsupported dtype %d",
                  (int)d->dtype);
    RAT3D_REQUIRE(d->k <= 15, RAT3D_EUNSUPPORTED, "kernel size above 15 is not built");
    *g = make_geom(d->n, d->c_in, d->c_out, d->d, d->h, d->w, d->k, d->stride, d->pad);
    RAT3D_REQUIRE(g->Do >= 1 && g->Ho >= 1 && g->Wo >= 1, RAT3D_EINVAL,
                  "conv output would be empty");
    const double big = 9.0e18;
    RAT3D_REQUIRE((double)d->n * d->c_in * d->d * d->h * d->w < big &&
                      (double)d->n * d->c_out * g->Do * g->Ho * g->Wo < big,
                  RAT3D_EINVAL, "tensor too large");
    RAT3D_REQUIRE((double)d->n * g->Do * g->Ho * g->Wo / 64.0 < 2.0e9 &&
                      (double)d->n * d->d * d->h * d->w / 64.0 < 2.0e9,
                  RAT3D_EUNSUPPORTED, "tensor too large for one launch");
    return RAT3D_OK;
}

rat3d_status check_conv_desc(const rat3d_conv3d_desc* d, ConvGeom* g) { return check_conv(d, g); }

rat3d_status check_act(const void* p, const char* name) {
    RAT3D_ACT(p, name);
    return RAT3D_OK;
}

static rat3d_status check_ws(void* ws, size_t ws_bytes, size_t need) {
    if (need == 0) return RAT3D_OK;
    RAT3D_REQUIRE(ws_bytes >= need, RAT3D_EWORKSPACE, "workspace needs %zu bytes, got %zu",
                  need, ws_bytes);
    RAT3D_ACT(ws, "workspace");
    return RAT3D_OK;
}

}  // namespace rat3d

using namespace rat3d;

extern "C" {

const char* rat3d_last_error(void) { return g_last_error.c_str(); }

const char* rat3d_version(void) { return "0.1.0"; }

size_t rat3d_conv3d_workspace_size(const rat3d_conv3d_desc* desc, int pass) {
    ConvGeom g;
    if (check_conv(desc, &g) != RAT3D_OK || pass < 0 || pass > 2) return (size_t)-1;
    return conv_ws_bytes(g, desc->dtype, pass);
}

rat3d_status rat3d_conv3d_fwd(const rat3d_conv3d_desc* desc, const void* x, const void* w,
                              const float* bias, void* y, void* ws, size_t ws_bytes,
                              void* stream) {
    ConvGeom g;
    rat3d_status s = check_conv(desc, &g);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(x, "x");
    RAT3D_ACT(y, "y");
    RAT3D_REQUIRE(w != nullptr, RAT3D_EINVAL, "w must not be NULL");
    RAT3D_REQUIRE(!desc->has_bias || bias != nullptr, RAT3D_EINVAL,
                  "bias required when has_bias");
    s = check_ws(ws, ws_bytes, conv_ws_bytes(g, desc->dtype, 0));
    if (s != RAT3D_OK) return s;
    return conv_fwd(g, desc->dtype, x, w, desc->has_bias ? bias : nullptr, y, ws, ws_bytes,
                    (hipStream_t)stream);
}

rat3d_status rat3d_conv3d_dgrad(const rat3d_conv3d_desc* desc, const void* dy, const void* w,
                                void* dx, int accumulate, void* ws, size_t ws_bytes,
                                void* stream) {
    ConvGeom g;
    rat3d_status s = check_conv(desc, &g);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(dy, "dy");
    RAT3D_ACT(dx, "dx");
    RAT3D_REQUIRE(w != nullptr, RAT3D_EINVAL, "w must not be NULL");
    s = check_ws(ws, ws_bytes, conv_ws_bytes(g, desc->dtype, 1));
    if (s != RAT3D_OK) return s;
    return conv_dgrad(g, desc->dtype, dy, w, dx, accumulate ? 1 : 0, ws, ws_bytes,
                      (hipStream_t)stream);
}

rat3d_status rat3d_conv3d_wgrad(const rat3d_conv3d_desc* desc, const void* x, const void* dy,
                                float* dw, float* dbias, int accumulate, void* ws,
                                size_t ws_bytes, void* stream) {
    ConvGeom g;
    rat3d_status s = check_conv(desc, &g);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(x, "x");
    RAT3D_ACT(dy, "dy");
    RAT3D_REQUIRE(dw != nullptr, RAT3D_EINVAL, "dw must not be NULL");
    s = check_ws(ws, ws_bytes, conv_ws_bytes(g, desc->dtype, 2));
    if (s != RAT3D_OK) return s;
    return conv_wgrad(g, desc->dtype, x, dy, dw, dbias, accumulate ? 1 : 0, ws, ws_bytes,
                      (hipStream_t)stream);
}

static rat3d_status check_bn(const rat3d_bn_desc* d, BnGeom* g) {
    RAT3D_REQUIRE(d != nullptr, RAT3D_EINVAL, "bn descriptor is NULL");
    RAT3D_REQUIRE(d->n >= 1 && d->c >= 1 && d->d >= 1 && d->h >= 1 && d->w >= 1, RAT3D_EINVAL,
                  "bn sizes must be >= 1");
    RAT3D_REQUIRE(d->eps > 0.f && d->momentum >= 0.f && d->momentum <= 1.f, RAT3D_EINVAL,
                  "bn needs eps > 0 and 0 <= momentum <= 1");
    RAT3D_REQUIRE(valid_dtype(d->dtype), RAT3D_EUNSUPPORTED, "unsupported dtype %d",
                  (int)d->dtype);
    *g = BnGeom{d->n, d->c, (int64_t)d->d * d->h * d->w};
    return RAT3D_OK;
}

size_t rat3d_bn_workspace_size(const rat3d_bn_desc* desc) {
    BnGeom g;
    if (check_bn(desc, &g) != RAT3D_OK) return (size_t)-1;
    return bn_ws_bytes(g);
}

rat3d_status rat3d_bn_relu_fwd(const rat3d_bn_desc* desc, const void* x, const void* residual,
                               const float* gamma, const float* beta, void* y,
                               float* save_mean, float* save_invstd, float* run_mean,
                               float* run_var, void* ws, size_t ws_bytes, void* stream) {
    BnGeom g;
    rat3d_status s = check_bn(desc, &g);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(x, "x");
    RAT3D_ACT(y, "y");
    if (residual) RAT3D_ACT(residual, "residual");
    RAT3D_REQUIRE(gamma && beta && save_mean && save_invstd, RAT3D_EINVAL,
                  "gamma, beta, save_mean and save_invstd are required");
    s = check_ws(ws, ws_bytes, bn_ws_bytes(g));
    if (s != RAT3D_OK) return s;
    return bn_fwd(g, desc->dtype, desc->relu, desc->eps, desc->momentum, x, residual, gamma, beta,
                  y, save_mean, save_invstd, run_mean, run_var, nullptr, nullptr, ws,
                  (hipStream_t)stream);
}

rat3d_status rat3d_bn_relu_bwd(const rat3d_bn_desc* desc, const void* dy, const void* x,
                               const void* y, const float* gamma, const float* save_mean,
                               const float* save_invstd, void* dx, void* dresidual,
                               float* dgamma, float* dbeta, int accumulate, void* ws,
                               size_t ws_bytes, void* stream) {
    BnGeom g;
    rat3d_status s = check_bn(desc, &g);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(dy, "dy");
    RAT3D_ACT(x, "x");
    RAT3D_ACT(dx, "dx");
    if (desc->relu) RAT3D_ACT(y, "y");
    if (dresidual) RAT3D_ACT(dresidual, "dresidual");
    RAT3D_REQUIRE(gamma && save_mean && save_invstd && dgamma && dbeta, RAT3D_EINVAL,
                  "gamma, save_mean, save_invstd, dgamma and dbeta are required");
    s = check_ws(ws, ws_bytes, bn_ws_bytes(g));
    if (s != RAT3D_OK) return s;
    return bn_bwd(g, desc->dtype, desc->relu, dy, x, y, nullptr, gamma, save_mean, save_invstd,
                  nullptr,
                  dx, dresidual, 0, dgamma, dbeta, accumulate ? 1 : 0, ws, (hipStream_t)stream);
}

static rat3d_status check_pool(const rat3d_pool_desc* d) {
    RAT3D_REQUIRE(d != nullptr, RAT3D_EINVAL, "pool descriptor is NULL");
    RAT3D_REQUIRE(d->n >= 1 && d->c >= 1 && d->d >= 1 && d->h >= 1 && d->w >= 1, RAT3D_EINVAL,
                  "pool sizes must be >= 1");
    RAT3D_REQUIRE(d->k >= 1 && d->stride >= 1 && d->pad >= 0 && d->pad < d->k, RAT3D_EINVAL,
                  "pool needs k >= 1, stride >= 1, 0 <= pad < k");
    RAT3D_REQUIRE(d->k * d->k * d->k <= 256, RAT3D_EUNSUPPORTED,
                  "pool window above 256 taps does not fit the uint8 argmax");
    RAT3D_REQUIRE(valid_dtype(d->dtype), RAT3D_EUNSUPPORTED, "unsupported dtype");
    RAT3D_REQUIRE(out_dim(d->d, d->k, d->stride, d->pad) >= 1 &&
                      out_dim(d->h, d->k, d->stride, d->pad) >= 1 &&
                      out_dim(d->w, d->k, d->stride, d->pad) >= 1,
                  RAT3D_EINVAL, "pool output would be empty");
    return RAT3D_OK;
}

rat3d_status rat3d_softmask_down_fwd(const rat3d_pool_desc* desc, const void* x, void* y,
                                     uint8_t* argmax, void* stream) {
    rat3d_status s = check_pool(desc);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(x, "x");
    RAT3D_ACT(y, "y");
    RAT3D_REQUIRE(argmax != nullptr, RAT3D_EINVAL, "argmax must not be NULL");
    return pool_fwd(desc->n, desc->c, desc->d, desc->h, desc->w, desc->k, desc->stride, desc->pad,
                    desc->dtype, x, y, argmax, (hipStream_t)stream);
}

rat3d_status rat3d_softmask_down_bwd(const rat3d_pool_desc* desc, const void* dy,
                                     const uint8_t* argmax, void* dx, int accumulate,
                                     void* stream) {
    rat3d_status s = check_pool(desc);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(dy, "dy");
    RAT3D_ACT(dx, "dx");
    RAT3D_REQUIRE(argmax != nullptr, RAT3D_EINVAL, "argmax must not be NULL");
    return pool_bwd(desc->n, desc->c, desc->d, desc->h, desc->w, desc->k, desc->stride, desc->pad,
                    desc->dtype, dy, argmax, dx, accumulate ? 1 : 0, (hipStream_t)stream);
}

static rat3d_status check_up(const rat3d_up_desc* d) {
    RAT3D_REQUIRE(d != nullptr, RAT3D_EINVAL, "up descriptor is NULL");
    RAT3D_REQUIRE(d->n >= 1 && d->c >= 1 && d->d_in >= 1 && d->h_in >= 1 && d->w_in >= 1 &&
                      d->d_out >= 1 && d->h_out >= 1 && d->w_out >= 1,
                  RAT3D_EINVAL, "up sizes must be >= 1");
    RAT3D_REQUIRE(d->d_out <= 3 * d->d_in && d->h_out <= 3 * d->h_in && d->w_out <= 3 * d->w_in,
                  RAT3D_EUNSUPPORTED, "up ratio above 3 per axis is not built");
    RAT3D_REQUIRE(valid_dtype(d->dtype), RAT3D_EUNSUPPORTED, "unsupported dtype");
    return RAT3D_OK;
}

rat3d_status rat3d_softmask_up_fwd(const rat3d_up_desc* desc, const void* x, void* y,
                                   void* stream) {
    rat3d_status s = check_up(desc);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(x, "x");
    RAT3D_ACT(y, "y");
    return up_fwd(desc->n, desc->c, desc->d_in, desc->h_in, desc->w_in, desc->d_out, desc->h_out,
                  desc->w_out, desc->dtype, x, y, (hipStream_t)stream);
}

rat3d_status rat3d_softmask_up_bwd(const rat3d_up_desc* desc, const void* dy, void* dx,
                                   int accumulate, void* stream) {
    rat3d_status s = check_up(desc);
    if (s != RAT3D_OK) return s;
    RAT3D_ACT(dy, "dy");
    RAT3D_ACT(dx, "dx");
    return up_bwd(desc->n, desc->c, desc->d_in, desc->h_in, desc->w_in, desc->d_out, desc->h_out,
                  desc->w_out, desc->dtype, dy, dx, accumulate ? 1 : 0, (hipStream_t)stream);
}

rat3d_status rat3d_softmask_fwd(int64_t count, rat3d_dtype dtype, const void* z, const void* t,
                                void* out, void* m, void* stream) {
    RAT3D_REQUIRE(count >= 1, RAT3D_EINVAL, "count must be >= 1");
    RAT3D_REQUIRE(valid_dtype(dtype), RAT3D_EUNSUPPORTED, "unsupported dtype");
    RAT3D_ACT(z, "z");
    RAT3D_ACT(t, "t");
    RAT3D_ACT(out, "out");
    if (m) RAT3D_ACT(m, "m");
    return softmask_fwd(count, dtype, z, t, out, m, (hipStream_t)stream);
}

rat3d_status rat3d_softmask_bwd(int64_t count, rat3d_dtype dtype, const void* dout,
                                const void* t, const void* m, void* dt, int accumulate_dt,
                                void* dz, void* stream) {
    RAT3D_REQUIRE(count >= 1, RAT3D_EINVAL, "count must be >= 1");
    RAT3D_REQUIRE(valid_dtype(dtype), RAT3D_EUNSUPPORTED, "unsupported dtype");
    RAT3D_ACT(dout, "dout");
    RAT3D_ACT(t, "t");
    RAT3D_ACT(m, "m");
    RAT3D_ACT(dt, "dt");
    RAT3D_ACT(dz, "dz");
    return softmask_bwd(count, dtype, dout, t, m, dt, accumulate_dt ? 1 : 0, dz,
                        (hipStream_t)stream);
}

size_t rat3d_head_workspace_size(int n, int c, int classes) {
    if (n < 1 || c < 1 || classes < 1) return (size_t)-1;
    return head_ws_bytes(n, c, classes);
}

rat3d_status rat3d_head_fwd_bwd(int n, int c, int64_t v, int classes, rat3d_dtype dtype,
                                const void* x, const float* fc_w, const float* fc_b,
                                const int32_t* labels, float* logits, float* loss, void* dx,
                                float* dfc_w, float* dfc_b, int accumulate, void* ws,
                                size_t ws_bytes, void* stream) {
    RAT3D_REQUIRE(n >= 1 && c >= 1 && v >= 1 && classes >= 1, RAT3D_EINVAL,
                  "head sizes must be >= 1");
    RAT3D_REQUIRE(classes <= 8 && n * classes <= 256, RAT3D_EUNSUPPORTED,
                  "head supports classes <= 8 and n*classes <= 256");
    RAT3D_REQUIRE(valid_dtype(dtype), RAT3D_EUNSUPPORTED, "unsupported dtype");
    RAT3D_ACT(x, "x");
    RAT3D_ACT(dx, "dx");
    RAT3D_REQUIRE(fc_w && fc_b && labels && logits && loss && dfc_w && dfc_b, RAT3D_EINVAL,
                  "head pointers must not be NULL");
    rat3d_status s = check_ws(ws, ws_bytes, head_ws_bytes(n, c, classes));
    if (s != RAT3D_OK) return s;
    return head_fwd_bwd(n, c, v, classes, dtype, x, fc_w, fc_b, labels, logits, loss, dx, dfc_w,
                        dfc_b, accumulate ? 1 : 0, ws, (hipStream_t)stream);
}

rat3d_status rat3d_sgd(int64_t count, float lr, float* params, const float* grads,
                       void* stream) {
    RAT3D_REQUIRE(count >= 0, RAT3D_EINVAL, "count must be >= 0");
    if (count == 0) return RAT3D_OK;
    RAT3D_REQUIRE(params && grads, RAT3D_EINVAL, "params and grads must not be NULL");
    return sgd_update(count, lr, params, grads, (hipStream_t)stream);
}

}  // extern "C"
