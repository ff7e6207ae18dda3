// Host-side launchers of the librat3d kernels.  Every launcher enqueues on the
// given stream, checks the launch and returns a rat3d_status; shapes have been
// validated by the caller.
#pragma once

#include "common.hpp"

namespace rat3d {

// Geometry of one convolution (input N x Ci x D x H x W, cubic kernel k).
struct ConvGeom {
    int N, Ci, Co, D, H, W, k, s, p;
    int Do, Ho, Wo;
};

inline ConvGeom make_geom(int N, int Ci, int Co, int D, int H, int W, int k, int s, int p) {
    ConvGeom g{N, Ci, Co, D, H, W, k, s, p, 0, 0, 0};
    g.Do = out_dim(D, k, s, p);
    g.Ho = out_dim(H, k, s, p);
    g.Wo = out_dim(W, k, s, p);
    return g;
}

// ---- argument validation shared by the C entry points (api.cpp) --------
// The descriptor checks of the conv calls (sizes, k/stride/pad, dtype,
// non-empty output), filling g; and the NULL / 16-byte alignment check of an
// activation pointer.  Both set the thread's error message on failure.
rat3d_status check_conv_desc(const rat3d_conv3d_desc* d, ConvGeom* g);
rat3d_status check_act(const void* p, const char* name);

// ---- convolution: dispatch (conv.cpp) ----------------------------------
// Workspace bytes of a pass (0 fwd, 1 dgrad, 2 wgrad).
size_t conv_ws_bytes(const ConvGeom& g, rat3d_dtype dt, int pass);
// Public-layout entry points: w is [Co][Ci][k^3] in dtype dt.
rat3d_status conv_fwd(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* w,
                      const float* bias, void* y, void* ws, size_t ws_bytes, hipStream_t st);
rat3d_status conv_dgrad(const ConvGeom& g, rat3d_dtype dt, const void* dy, const void* w,
                        void* dx, int accumulate, void* ws, size_t ws_bytes, hipStream_t st);
rat3d_status conv_wgrad(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* dy,
                        float* dw, float* db, int accumulate, void* ws, size_t ws_bytes,
                        hipStream_t st);
// Prepared weights: whether the forward (pass 0) or input-gradient (pass 1)
// kernel of a shape reads a prepared weight layout; the layout's bytes; the
// preparation; and the two passes taking already prepared weights wt (other
// shapes ignore wt and use w).
bool conv_uses_prepared(const ConvGeom& g, rat3d_dtype dt, int pass);
size_t conv_prepared_bytes(const ConvGeom& g);
rat3d_status conv_prepare(const ConvGeom& g, rat3d_dtype dt, int pass, const void* w, void* wt,
                          hipStream_t st);
rat3d_status conv_fwd_prepared(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* w,
                               const void* wt, const float* bias, void* y, void* ws,
                               size_t ws_bytes, hipStream_t st);
rat3d_status conv_dgrad_prepared(const ConvGeom& g, rat3d_dtype dt, const void* dy,
                                 const void* w, const void* wt, void* dx, int accumulate,
                                 void* ws, size_t ws_bytes, hipStream_t st);

// Algorithmic work of one conv pass: 2 * N * Co * Ci * k^3 * Vout flops, and
// one read of the input and weights plus one write of the output.
double conv_flops(const ConvGeom& g);
double conv_bytes(const ConvGeom& g, size_t esz);

// ---- generic gather implicit GEMM (conv_gather.hip) --------------------
rat3d_status conv_fwd_gather(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* w,
                             const float* bias, void* y, hipStream_t st);
rat3d_status conv_dgrad_gather(const ConvGeom& g, rat3d_dtype dt, const void* dy, const void* w,
                               void* dx, int accumulate, hipStream_t st);
size_t wgrad_gather_ws(const ConvGeom& g);
rat3d_status conv_wgrad_gather(const ConvGeom& g, rat3d_dtype dt, const void* x, const void* dy,
                               float* dw, int accumulate, void* ws, hipStream_t st);
size_t bias_grad_ws(const ConvGeom& g);
rat3d_status conv_bias_grad(const ConvGeom& g, rat3d_dtype dt, const void* dy, float* db,
                            int accumulate, void* ws, hipStream_t st);
// dw (+)= sum over `splits` partial slabs of `count` floats, in slab order.
rat3d_status wgrad_reduce_launch(const float* part, int splits, int64_t count, float* dw,
                                 int accumulate, hipStream_t st);

// ---- LDS-brick kernels for bf16, stride 1, k in {1, 3} (conv_brick.hip) ---
bool brick_fd_ok(const ConvGeom& g, rat3d_dtype dt, bool dgrad);
bool brick_wgrad_ok(const ConvGeom& g, rat3d_dtype dt);
size_t brick_fd_ws(const ConvGeom& g, bool dgrad);  // prepared weights (+ split partials)
size_t brick_wgrad_ws(const ConvGeom& g);
// w_prepared: w already holds the layout brick_prep_weights writes for this
// pass (the workspace is then unused); otherwise it is prepared into ws.
rat3d_status conv_fd_brick(const ConvGeom& g, bool dgrad, const void* src, const void* w,
                           const float* bias, void* dst, int accumulate, void* ws,
                           hipStream_t st, bool w_prepared = false);
// Writes the brick kernels' weight layout of the forward or input-gradient
// pass (Co * Ci * k^3 bf16 elements) from w [Co][Ci][k^3].
rat3d_status brick_prep_weights(const ConvGeom& g, bool dgrad, const void* w, void* wt,
                                hipStream_t st);
// The same for several convolutions, kPrepJobs per launch.
constexpr int kPrepJobs = 24;
struct PrepJob {
    ConvGeom g;
    bool dgrad;
    const void* w;
    void* wt;
};
rat3d_status brick_prep_weights_batch(const PrepJob* jobs, int n, hipStream_t st);
rat3d_status conv_wgrad_brick(const ConvGeom& g, const void* x, const void* dy, float* dw,
                              int accumulate, void* ws, hipStream_t st);

// ---- stem: one input channel, 7^3, stride 2, pad 3 (conv_stem.hip) -------
bool stem_ok(const ConvGeom& g, rat3d_dtype dt);
bool stem_wgrad_ok(const ConvGeom& g, rat3d_dtype dt);
size_t stem_fwd_ws();
size_t stem_wgrad_ws(const ConvGeom& g);
rat3d_status conv_fwd_stem(const ConvGeom& g, const void* x, const void* w, void* y, void* ws,
                           hipStream_t st);
rat3d_status conv_wgrad_stem(const ConvGeom& g, const void* x, const void* dy, float* dw,
                             int accumulate, void* ws, hipStream_t st);

// ---- 1x1x1 weight gradient as a direct GEMM (conv_pw.hip) ---------------
bool pw_wgrad_ok(const ConvGeom& g, rat3d_dtype dt);
// forward / input gradient with at most 64 source and target channels; wt is
// the brick kernels' prepared weight layout for k = 1
bool pw_fd_ok(const ConvGeom& g, rat3d_dtype dt, bool dgrad);
rat3d_status conv_fd_pw(const ConvGeom& g, bool dgrad, const void* src, const void* wt,
                        const float* bias, void* dst, int accumulate, hipStream_t st);
size_t pw_wgrad_ws(const ConvGeom& g);
rat3d_status conv_wgrad_pw(const ConvGeom& g, const void* x, const void* dy, float* dw,
                           int accumulate, void* ws, hipStream_t st);

// db (+)= the per-channel sums of `part` ([C][S] floats, summed in order)
rat3d_status bias_grad_from_partials(const float* part, int C, int S, float* db, int accumulate,
                                     hipStream_t st);

// ---- batch norm (bn.hip) -----------------------------------------------
struct BnGeom {
    int N, C;
    int64_t V;  // voxels per (n, c) plane
};
size_t bn_ws_bytes(const BnGeom& g);
// save_coef (may be null): receives the apply's float scale [C] and shift [C].
// ybits (may be null; bf16 with V % 8 == 0 and relu only): receives y > 0 of
// the stored y, one bit per element (byte i/8, bit i%8).
bool bn_bits_ok(const BnGeom& g, rat3d_dtype dt);
rat3d_status bn_fwd(const BnGeom& g, rat3d_dtype dt, int relu, float eps, float momentum,
                    const void* x, const void* residual, const float* gamma, const float* beta,
                    void* y, float* save_mean, float* save_invstd, float* run_mean,
                    float* run_var, float* save_coef, uint8_t* ybits, void* ws, hipStream_t st);
// fwd_coef (may be null): the forward's scale/shift of a BN + ReLU without a
// residual; the ReLU mask is then recomputed from x and y is not read.
// ybits (may be null): the forward's y > 0 bits; read instead of y.
// dres_acc: the residual gradient is added to dres (one rounding) instead of
// stored.
rat3d_status bn_bwd(const BnGeom& g, rat3d_dtype dt, int relu, const void* dy, const void* x,
                    const void* y, const uint8_t* ybits, const float* gamma,
                    const float* save_mean, const float* save_invstd, const float* fwd_coef,
                    void* dx, void* dres, int dres_acc, float* dgamma, float* dbeta,
                    int accumulate, void* ws, hipStream_t st);

// Pieces for the fused passes of the soft-mask branch (bf16, V % 8 == 0).
struct BnBwdStats;
rat3d_status bn_bwd_stats_x(const BnGeom& g, const void* dy, const void* x, const float* gamma,
                            const float* save_mean, const float* save_invstd,
                            const float* fwd_coef, float* dgamma, float* dbeta, int accumulate,
                            void* ws, hipStream_t st, BnBwdStats* bs);
size_t bn_max_slices(const BnGeom& g);
// relu(BN(x) + BN_r(r)) with the residual's BN applied inside (ws, rws: one
// bn_ws_bytes workspace each)
rat3d_status bn_fwd_res_bn(const BnGeom& g, float eps, float momentum, const void* x,
                           const float* gamma, const float* beta, void* y, float* save_mean,
                           float* save_invstd, float* run_mean, float* run_var,
                           uint8_t* ybits, void* ws, const void* r, const float* rgamma,
                           const float* rbeta, float* rsave_mean, float* rsave_invstd,
                           float* rrun_mean, float* rrun_var, void* rws, hipStream_t st);
rat3d_status bn_fwd_apply_from(const BnGeom& g, float eps, float momentum, const void* x,
                               const float* gamma, const float* beta, void* y,
                               float* save_mean, float* save_invstd, float* run_mean,
                               float* run_var, float* save_coef, const float* part, int slices,
                               hipStream_t st);

// ---- soft-mask branch (softmask.hip) -----------------------------------
rat3d_status pool_fwd(int N, int C, int D, int H, int W, int k, int s, int p, rat3d_dtype dt,
                      const void* x, void* y, uint8_t* argmax, hipStream_t st);
rat3d_status pool_bwd(int N, int C, int D, int H, int W, int k, int s, int p, rat3d_dtype dt,
                      const void* dy, const uint8_t* argmax, void* dx, int accumulate,
                      hipStream_t st);
rat3d_status up_fwd(int N, int C, int Di, int Hi, int Wi, int Do, int Ho, int Wo,
                    rat3d_dtype dt, const void* x, void* y, hipStream_t st);
rat3d_status up_bwd(int N, int C, int Di, int Hi, int Wi, int Do, int Ho, int Wo,
                    rat3d_dtype dt, const void* dy, void* dx, int accumulate, hipStream_t st);
rat3d_status softmask_fwd(int64_t count, rat3d_dtype dt, const void* z, const void* t,
                          void* out, void* m, hipStream_t st);
// m_is_z: `m` holds z (m was not stored) and m is recomputed and rounded as a
// store of it would be.  bias_part (bf16, count = N * C * V, V a multiple of
// 2048): per-block sums of the stored dz, [C][N * V / 2048], for
// bias_grad_from_partials.
rat3d_status softmask_bwd(int64_t count, rat3d_dtype dt, const void* dout, const void* t,
                          const void* m, void* dt_out, int accumulate_dt, void* dz,
                          hipStream_t st, int m_is_z = 0,
                          float* bias_part = nullptr, int N = 0, int C = 0, int64_t V = 0);
// relu(BN(up(xc))) with an exact x2 upsampling (bf16): the upsampling pass
// also yields the BN statistics (h = up(xc) is written for the backward);
// the backward forms h's gradient inside the upsampling transpose.
bool up2_bn_ok(int N, int C, int Di, int Hi, int Wi, rat3d_dtype dt);
rat3d_status up2_bn_relu_fwd(int N, int C, int Di, int Hi, int Wi, const void* xc, void* h,
                             float eps, float momentum, const float* gamma, const float* beta,
                             void* y, float* save_mean, float* save_invstd, float* run_mean,
                             float* run_var, float* save_coef, void* bn_ws, hipStream_t st);
rat3d_status bn_relu_bwd_up2(int N, int C, int Di, int Hi, int Wi, const void* dy, const void* h,
                             const float* gamma, const float* save_mean,
                             const float* save_invstd, const float* fwd_coef, float* dgamma,
                             float* dbeta, int accumulate, void* bn_ws, void* dxc,
                             hipStream_t st);

// ---- inference mode and Grad-CAM (gradcam.hip) --------------------------
// BN with the running statistics: y = act(x * s + t [+ residual]),
// s = gamma / sqrt(run_var + eps), t = beta - run_mean * s.
rat3d_status bn_eval_fwd(const BnGeom& g, rat3d_dtype dt, int relu, float eps, const void* x,
                         const void* residual, const float* gamma, const float* beta,
                         const float* run_mean, const float* run_var, void* y, hipStream_t st);
// Its gradients: dx = s * g (dx may be null), dres = g or dres += g (one
// rounding; dres may be null), g = dy masked by y > 0 under ReLU.
rat3d_status bn_eval_bwd(const BnGeom& g, rat3d_dtype dt, int relu, float eps, const void* dy,
                         const void* y, const float* gamma, const float* run_var, void* dx,
                         void* dres, int dres_acc, hipStream_t st);
// dtop[n, c, v] = fc_w[classes[n], c] / V (classes clamped into range).
rat3d_status gradcam_seed(int N, int C, int64_t V, int classes_n, rat3d_dtype dt,
                          const float* fc_w, const int32_t* classes, void* dtop, hipStream_t st);
// logits[n, k] = fc_w[k] . mean_v top[n, :, v] + fc_b[k] (classes_n <= 8).
rat3d_status gradcam_logits(int N, int C, int64_t V, int classes_n, rat3d_dtype dt,
                            const void* top, const float* fc_w, const float* fc_b,
                            float* logits, hipStream_t st);
// alpha[n, c] = voxel mean of dA; cam[n, v] = max(0, sum_c alpha A); cam_up
// (nullable) = cam resampled trilinearly to D0 x H0 x W0.
rat3d_status gradcam_maps(int N, int C, int Dt, int Ht, int Wt, rat3d_dtype dt, const void* A,
                          const void* dA, float* alpha, float* cam, int D0, int H0, int W0,
                          float* cam_up, hipStream_t st);

// ---- head, update, casts (head.hip) ------------------------------------
size_t head_ws_bytes(int N, int C, int classes);
rat3d_status head_fwd_bwd(int N, int C, int64_t V, int classes, rat3d_dtype dt, const void* x,
                          const float* fc_w, const float* fc_b, const int32_t* labels,
                          float* logits, float* loss, void* dx, float* dfc_w, float* dfc_b,
                          int accumulate, void* ws, hipStream_t st);
rat3d_status sgd_update(int64_t count, float lr, float* params, const float* grads,
                        hipStream_t st);
// dst[i] = bf16(src[i]) for i < count.
rat3d_status cast_f32_bf16(int64_t count, const float* src, bf16* dst, hipStream_t st);
// dst[i] = value.
rat3d_status fill_f32(int64_t count, float value, float* dst, hipStream_t st);
// dst[i] (+)= a[i] + b[i] in dtype (one rounding).
rat3d_status add_tensors(int64_t count, rat3d_dtype dt, const void* a, const void* b, void* dst,
                         hipStream_t st);

}  // namespace rat3d
