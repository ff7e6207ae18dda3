// Convolution dispatch: picks the kernel family for a shape and sizes its
// workspace.  bf16 stride-1 convolutions with kernel 3 (pad 1) or 1 (pad 0)
// and suitable channel counts take the LDS-brick kernels (1^3 weight
// gradients a direct GEMM); the single-channel 7^3 stride-2 stem has its own
// kernels; every other shape is served by the generic gather implicit GEMM.
#include "kernels.hpp"

namespace rat3d {

static size_t wgrad_ws(const ConvGeom& g, rat3d_dtype dt) {
    if (stem_wgrad_ok(g, dt)) return stem_wgrad_ws(g);
    if (brick_wgrad_ok(g, dt)) return brick_wgrad_ws(g);
    if (pw_wgrad_ok(g, dt)) return pw_wgrad_ws(g);
    return wgrad_gather_ws(g);
}

size_t conv_ws_bytes(const ConvGeom& g, rat3d_dtype dt, int pass) {
    if (pass == 0) {
        if (stem_ok(g, dt)) return stem_fwd_ws();
        return brick_fd_ok(g, dt, false) ? brick_fd_ws(g, false) : 0;
    }
    if (pass == 1) return brick_fd_ok(g, dt, true) ? brick_fd_ws(g, true) : 0;
    // weight-gradient partials, then the bias-gradient slice sums
    const size_t wb = wgrad_ws(g, dt);
    return ((wb + 255) & ~(size_t)255) + bias_grad_ws(g);
}

rat3d_status conv_fwd(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* w,
                      const float* bias, void* y, void* ws, size_t ws_bytes, hipStream_t st) {
    (void)ws_bytes;
    if (stem_ok(g, dt) && !bias) return conv_fwd_stem(g, x, w, y, ws, st);
    if (brick_fd_ok(g, dt, false)) return conv_fd_brick(g, false, x, w, bias, y, 0, ws, st);
    return conv_fwd_gather(g, dt, x, w, bias, y, st);
}

rat3d_status conv_dgrad(const ConvGeom& g, rat3d_dtype dt, const void* dy, const void* w,
                        void* dx, int accumulate, void* ws, size_t ws_bytes, hipStream_t st) {
    (void)ws_bytes;
    if (brick_fd_ok(g, dt, true))
        return conv_fd_brick(g, true, dy, w, nullptr, dx, accumulate, ws, st);
    return conv_dgrad_gather(g, dt, dy, w, dx, accumulate, st);
}

bool conv_uses_prepared(const ConvGeom& g, rat3d_dtype dt, int pass) {
    if (pass == 0) return !(stem_ok(g, dt)) && brick_fd_ok(g, dt, false);
    if (pass == 1) return brick_fd_ok(g, dt, true);
    return false;
}

size_t conv_prepared_bytes(const ConvGeom& g) {
    return (size_t)g.Co * g.Ci * g.k * g.k * g.k * 2;
}

rat3d_status conv_prepare(const ConvGeom& g, rat3d_dtype dt, int pass, const void* w, void* wt,
                          hipStream_t st) {
    if (!conv_uses_prepared(g, dt, pass)) return RAT3D_OK;
    return brick_prep_weights(g, pass == 1, w, wt, st);
}

rat3d_status conv_fwd_prepared(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* w,
                               const void* wt, const float* bias, void* y, void* ws,
                               size_t ws_bytes, hipStream_t st) {
    if (wt && conv_uses_prepared(g, dt, 0))
        return conv_fd_brick(g, false, x, wt, bias, y, 0, ws, st, true);
    return conv_fwd(g, dt, x, w, bias, y, ws, ws_bytes, st);
}

rat3d_status conv_dgrad_prepared(const ConvGeom& g, rat3d_dtype dt, const void* dy,
                                 const void* w, const void* wt, void* dx, int accumulate,
                                 void* ws, size_t ws_bytes, hipStream_t st) {
    if (wt && conv_uses_prepared(g, dt, 1))
        return conv_fd_brick(g, true, dy, wt, nullptr, dx, accumulate, ws, st, true);
    return conv_dgrad(g, dt, dy, w, dx, accumulate, ws, ws_bytes, st);
}

rat3d_status conv_wgrad(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* dy,
                        float* dw, float* db, int accumulate, void* ws, size_t ws_bytes,
                        hipStream_t st) {
    (void)ws_bytes;
    rat3d_status s;
    if (stem_wgrad_ok(g, dt)) s = conv_wgrad_stem(g, x, dy, dw, accumulate, ws, st);
    else if (brick_wgrad_ok(g, dt)) s = conv_wgrad_brick(g, x, dy, dw, accumulate, ws, st);
    else if (pw_wgrad_ok(g, dt)) s = conv_wgrad_pw(g, x, dy, dw, accumulate, ws, st);
    else s = conv_wgrad_gather(g, dt, x, dy, dw, accumulate, ws, st);
    if (s != RAT3D_OK) return s;
    if (db) {
        const size_t wb = wgrad_ws(g, dt);
        return conv_bias_grad(g, dt, dy, db, accumulate,
                              (char*)ws + ((wb + 255) & ~(size_t)255), st);
    }
    return RAT3D_OK;
}

}  // namespace rat3d
