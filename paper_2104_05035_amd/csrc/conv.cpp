// Convolution dispatch: picks the kernel family for a shape and sizes its
// workspace.  Every shape is served by the generic gather implicit GEMM;
// 3x3x3 and 1x1x1 stride-1 convolutions with suitable channel counts take the
// LDS-brick kernels.
#include "kernels.hpp"

namespace rat3d {

size_t conv_ws_bytes(const ConvGeom& g, rat3d_dtype dt, int pass) {
    (void)dt;
    if (pass == 2) return wgrad_gather_ws(g);
    return 0;
}

rat3d_status conv_fwd(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* w,
                      const float* bias, void* y, void* ws, size_t ws_bytes, hipStream_t st) {
    (void)ws;
    (void)ws_bytes;
    return conv_fwd_gather(g, dt, x, w, bias, y, st);
}

rat3d_status conv_dgrad(const ConvGeom& g, rat3d_dtype dt, const void* dy, const void* w,
                        void* dx, int accumulate, void* ws, size_t ws_bytes, hipStream_t st) {
    (void)ws;
    (void)ws_bytes;
    return conv_dgrad_gather(g, dt, dy, w, dx, accumulate, st);
}

rat3d_status conv_wgrad(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* dy,
                        float* dw, float* db, int accumulate, void* ws, size_t ws_bytes,
                        hipStream_t st) {
    (void)ws_bytes;
    rat3d_status s = conv_wgrad_gather(g, dt, x, dy, dw, accumulate, ws, st);
    if (s != RAT3D_OK) return s;
    if (db) return conv_bias_grad(g, dt, dy, db, accumulate, st);
    return RAT3D_OK;
}

}  // namespace rat3d
