/*
 * rat3d.h -- C ABI of librat3d, the MI355X (gfx950) training step of a 3D
 * residual attention network (3D-ResAttNet), as used by the hybrid
 * model/data-parallel method of arXiv 2104.05035.
 *
 * What is computed, and where the paper defines it:
 *   - conv blocks: 3x3x3 3D convolution -> 3D batch normalisation -> ReLU;
 *     residual layers of two conv blocks; a self-attention layer inside the
 *     residual self-attention block (use-case section, description of the
 *     3D-ResAttNet blocks);
 *   - the cost of a conv layer, O(C_o C_i T H W K_T K_H K_W) (same passage);
 *   - batch-mean loss and mean-of-samples gradient (data-parallelisation
 *     section, the objective f(w;V) and its derivative, one GPU: m = 1);
 *   - cross-entropy loss and SGD at learning rate 1e-4 (experiments section);
 *   - w <- w - gamma_t * g after the gradient of a partition, and gradient
 *     accumulation over micro-batches of a partition before the update
 *     (model-parallelisation section, network partitioning).
 * The paper leaves the attention layer, the stage layout and the numeric
 * formats open; the readings implemented are listed with each call below.
 *
 * Conventions for every call:
 *   - Tensors are contiguous NCDHW; conv weights are [C_out][C_in][k][k][k].
 *   - Every pointer is device memory owned by the caller; the library never
 *     allocates device memory and never frees caller memory.  Activation
 *     tensors (x, y, dx, dy, residual, z, t, out, m) and workspaces must be
 *     16-byte aligned (RAT3D_EALIGN otherwise); weights and per-channel
 *     float32 vectors need only their natural alignment.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *     enqueue work; they return before it runs.  Argument errors are detected
 *     on the host and returned before anything is enqueued.
 *   - RAT3D_BF16 means bfloat16 storage of activations, activation gradients
 *     and weights, with float32 accumulation; every value stored to a bf16
 *     tensor is rounded to nearest-even.  Weight gradients, BN parameters and
 *     statistics, logits and the loss are always float32.
 *   - No call throws across the ABI.  On error the status is negative and
 *     rat3d_last_error() returns a message (thread-local, valid until the
 *     next call on the same thread).
 *   - All work of one call is enqueued on its stream only; results are
 *     deterministic (no atomics in any reduction).
 */
#ifndef RAT3D_H
#define RAT3D_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RAT3D_OK = 0,
    RAT3D_EINVAL = -1,       /* a size, count or pointer argument is invalid */
    RAT3D_EUNSUPPORTED = -2, /* valid, but this shape/dtype combination is not built */
    RAT3D_EALIGN = -3,       /* a device pointer is not 16-byte aligned */
    RAT3D_EWORKSPACE = -4,   /* workspace smaller than the *_workspace_size query */
    RAT3D_EHIP = -5          /* the HIP runtime reported an error at launch */
} rat3d_status;

typedef enum {
    RAT3D_F32 = 0,
    RAT3D_BF16 = 1,
    RAT3D_U8 = 2 /* only reported by rat3d_net_tensor_info (pooling argmax maps) */
} rat3d_dtype;

/* Message describing the last error on this thread ("" if none). */
const char* rat3d_last_error(void);

/* Library version, e.g. "0.1.0". */
const char* rat3d_version(void);

/* ------------------------------------------------------------------------
 * 3D convolution (use-case section: the conv block's 3x3x3 convolution and
 * the O(C_o C_i T H W K_T K_H K_W) cost).  Zero padding `pad` on every side,
 * stride `stride` on every axis, cubic kernel k.  Output size per axis:
 * floor((in + 2*pad - k) / stride) + 1.
 *   n, c_in, c_out, d, h, w : input batch, channels and volume (all >= 1)
 *   k >= 1, stride >= 1, 0 <= pad < k
 *   has_bias : forward adds bias[c_out]; wgrad then also produces dbias
 *   dtype    : storage type of x, y, w, dx, dy
 * Invalid geometry -> RAT3D_EINVAL.
 * ------------------------------------------------------------------------ */
typedef struct {
    int n, c_in, c_out, d, h, w, k, stride, pad, has_bias;
    rat3d_dtype dtype;
} rat3d_conv3d_desc;

/* Bytes of workspace `pass` needs (0 = fwd, 1 = dgrad, 2 = wgrad); 0 if
 * none.  (size_t)-1 if the descriptor is invalid. */
size_t rat3d_conv3d_workspace_size(const rat3d_conv3d_desc* desc, int pass);

/* y = conv(x, w) (+ bias).  x [n][c_in][d][h][w], w [c_out][c_in][k^3],
 * bias float32 [c_out] (device, required iff has_bias), y [n][c_out][out^3]. */
rat3d_status rat3d_conv3d_fwd(const rat3d_conv3d_desc* desc, const void* x, const void* w,
                              const float* bias, void* y, void* ws, size_t ws_bytes,
                              void* stream);

/* dx = conv^T(dy, w): dx[i] = sum over (co, t) with (i + pad - t) divisible by
 * stride of w[co][ci][t] * dy[(i + pad - t)/stride].  accumulate != 0 adds the
 * result to the existing dx (one rounding of the sum). */
rat3d_status rat3d_conv3d_dgrad(const rat3d_conv3d_desc* desc, const void* dy, const void* w,
                                void* dx, int accumulate, void* ws, size_t ws_bytes,
                                void* stream);

/* dw[co][ci][t] (+)= sum_{n,o} dy[n][co][o] * x[n][ci][o*stride - pad + t];
 * dbias[co] (+)= sum_{n,o} dy[n][co][o] (dbias may be NULL).  dw, dbias are
 * float32 device buffers; accumulate != 0 adds to their contents (used for
 * micro-batch accumulation). */
rat3d_status rat3d_conv3d_wgrad(const rat3d_conv3d_desc* desc, const void* x, const void* dy,
                                float* dw, float* dbias, int accumulate, void* ws,
                                size_t ws_bytes, void* stream);

/* rat3d_conv3d_wgrad without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * rat3d_conv3d_wgrad, except: the split partial sums live in a scratch array
 * built into the library (rat3d_conv3d_wgrad_noalloc_max_bytes() bytes, 32
 * MiB, held on each GPU the library runs on until the process ends); a shape
 * whose rat3d_conv3d_workspace_size(desc, 2) exceeds it returns
 * RAT3D_EWORKSPACE before anything is enqueued.  The call allocates nothing.
 * All calls on one GPU share that GPU's scratch array: calls that may run at
 * the same time on one GPU (different streams) race and must be ordered by
 * the caller.  The first call on a device looks the array's address up (a
 * HIP symbol query, no allocation). */
size_t rat3d_conv3d_wgrad_noalloc_max_bytes(void);
rat3d_status rat3d_conv3d_wgrad_noalloc(const rat3d_conv3d_desc* desc, const void* x,
                                        const void* dy, float* dw, float* dbias, int accumulate,
                                        void* stream);

/* ------------------------------------------------------------------------
 * 3D batch normalisation, training mode, fused with the ReLU of the conv
 * block and the residual add of the residual layer (use-case section).
 * Statistics are per channel over n*d*h*w; the variance used to normalise is
 * the biased one, the running variance the unbiased one.
 *   y = act(gamma * (x - mean) * invstd + beta [+ residual]),
 *   invstd = 1/sqrt(var + eps), act = ReLU if relu else identity.
 * ------------------------------------------------------------------------ */
typedef struct {
    int n, c, d, h, w, relu;
    float eps, momentum;
    rat3d_dtype dtype;
} rat3d_bn_desc;

size_t rat3d_bn_workspace_size(const rat3d_bn_desc* desc);

/* x, residual (nullable), y: [n][c][d][h][w] in dtype.  gamma, beta [c] f32.
 * save_mean, save_invstd [c] f32 outputs.  run_mean / run_var [c] f32 are
 * updated as r = (1 - momentum) r + momentum * batch value when non-NULL. */
rat3d_status rat3d_bn_relu_fwd(const rat3d_bn_desc* desc, const void* x, const void* residual,
                               const float* gamma, const float* beta, void* y,
                               float* save_mean, float* save_invstd, float* run_mean,
                               float* run_var, void* ws, size_t ws_bytes, void* stream);

/* Backward of rat3d_bn_relu_fwd.  dy is the gradient of y; y is the forward
 * output (its sign is the ReLU mask: gradient passes where y > 0).
 *   g = dy * [y > 0] (or dy if !relu);  dresidual = g (nullable);
 *   dbeta = sum g;  dgamma = sum g * xhat;
 *   dx = gamma * invstd * (g - dbeta/M - xhat * dgamma/M),  M = n*d*h*w.
 * dgamma, dbeta [c] f32: written, or added to when accumulate != 0. */
rat3d_status rat3d_bn_relu_bwd(const rat3d_bn_desc* desc, const void* dy, const void* x,
                               const void* y, const float* gamma, const float* save_mean,
                               const float* save_invstd, void* dx, void* dresidual,
                               float* dgamma, float* dbeta, int accumulate, void* ws,
                               size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Soft-mask branch of the attention layer.  The paper names a self-attention
 * layer inside its residual self-attention block (use-case section) without
 * giving its form; the reading built here is a soft mask: max-pool down,
 * trilinear up, sigmoid, and output (1 + M) * T.
 * ------------------------------------------------------------------------ */
typedef struct {
    int n, c, d, h, w, k, stride, pad;
    rat3d_dtype dtype;
} rat3d_pool_desc;

typedef struct {
    int n, c, d_in, h_in, w_in, d_out, h_out, w_out;
    rat3d_dtype dtype;
} rat3d_up_desc;

/* Max pooling over k^3 windows (padding never wins).  argmax (uint8, same
 * shape as y) is the window offset (kd*k + kh)*k + kw of the first maximum in
 * scan order.  Requires k^3 <= 256. */
rat3d_status rat3d_softmask_down_fwd(const rat3d_pool_desc* desc, const void* x, void* y,
                                     uint8_t* argmax, void* stream);

/* dx[i] (+)= sum of dy over the windows whose argmax names voxel i. */
rat3d_status rat3d_softmask_down_bwd(const rat3d_pool_desc* desc, const void* dy,
                                     const uint8_t* argmax, void* dx, int accumulate,
                                     void* stream);

/* Trilinear resampling to (d_out, h_out, w_out), half-pixel centres:
 * src = (o + 1/2) * in/out - 1/2 clamped at 0, i0 = floor(src),
 * i1 = min(i0 + 1, in - 1).  Each output size must be at most 3x its input
 * size (RAT3D_EUNSUPPORTED otherwise). */
rat3d_status rat3d_softmask_up_fwd(const rat3d_up_desc* desc, const void* x, void* y,
                                   void* stream);

/* Exact transpose of rat3d_softmask_up_fwd; accumulate != 0 adds to dx. */
rat3d_status rat3d_softmask_up_bwd(const rat3d_up_desc* desc, const void* dy, void* dx,
                                   int accumulate, void* stream);

/* m = sigmoid(z); out = (1 + m) * t.  z, t, out, m: `count` elements of dtype;
 * m may be NULL. */
rat3d_status rat3d_softmask_fwd(int64_t count, rat3d_dtype dtype, const void* z, const void* t,
                                void* out, void* m, void* stream);

/* dt (+)= (1 + m) * dout;  dz = dout * t * m * (1 - m), m as stored by the
 * forward.  accumulate_dt != 0 adds to dt. */
rat3d_status rat3d_softmask_bwd(int64_t count, rat3d_dtype dtype, const void* dout,
                                const void* t, const void* m, void* dt, int accumulate_dt,
                                void* dz, void* stream);

/* ------------------------------------------------------------------------
 * Classifier head and update (experiments section: cross-entropy, SGD).
 * ------------------------------------------------------------------------ */

/* Bytes of workspace rat3d_head_fwd_bwd needs. */
size_t rat3d_head_workspace_size(int n, int c, int classes);

/* Global average pool of x [n][c][v] (dtype) -> FC (fc_w [classes][c],
 * fc_b [classes], f32) -> logits [n][classes] f32 -> mean softmax
 * cross-entropy with int32 labels in [0, classes) (values outside are
 * clamped into range) -> *loss (f32, device).
 * Backward in the same call: dfc_w, dfc_b (f32, written or accumulated) and
 * dx [n][c][v] (dtype; gradient of x).  1 <= n*classes <= 256, classes <= 8. */
rat3d_status rat3d_head_fwd_bwd(int n, int c, int64_t v, int classes, rat3d_dtype dtype,
                                const void* x, const float* fc_w, const float* fc_b,
                                const int32_t* labels, float* logits, float* loss, void* dx,
                                float* dfc_w, float* dfc_b, int accumulate, void* ws,
                                size_t ws_bytes, void* stream);

/* params[i] -= lr * grads[i] for i < count (float32). */
rat3d_status rat3d_sgd(int64_t count, float lr, float* params, const float* grads,
                       void* stream);

/* ------------------------------------------------------------------------
 * Composite blocks and the training step.
 *   RAT3D_NET_RESUNIT    residual unit c_in -> c, stride 1: conv3 -> BN ->
 *                        ReLU -> conv3 -> BN, + skip (identity, or 1^3 conv +
 *                        BN when c_in != c), then ReLU.
 *   RAT3D_NET_ATTN       residual attention module on c channels: trunk = 2
 *                        residual units; mask = maxpool -> RU -> maxpool ->
 *                        RU -> RU -> up -> RU -> up -> 1^3 conv -> BN -> ReLU
 *                        -> 1^3 conv (+bias) -> sigmoid; out = (1 + M) * T.
 *                        (maxpool 3^3 stride 2 pad 1; up = trilinear back to
 *                        the pre-pool size.)
 *   RAT3D_NET_RESATTNET  single-channel input -> 7^3 stride-2 conv to 32 ch
 *                        -> BN -> ReLU -> maxpool -> three stages (64, 128,
 *                        256 ch; residual unit with stride 1, 2, 2, then an
 *                        attention module) -> global average pool -> FC to 2
 *                        classes -> cross-entropy -> SGD.
 *   RAT3D_NET_PARTITION1 first partition of the model-parallel split: stem
 *                        (7^3 s2 conv to 32 ch, BN, ReLU) -> residual unit
 *                        32 -> c -> attention module on c channels; driven by
 *                        the gradient received at its output; weight
 *                        gradients are summed over `micro_batches` micro-
 *                        batches of n volumes each, then one SGD step.
 * Parameter arena (float32, `rat3d_net_param_count` elements): for each conv
 * its weight then its bias if any, for each BN gamma then beta, the FC
 * weight and bias last; residual unit order conv1, bn1, conv2, bn2, then the
 * projection conv and its BN; attention module order: trunk units 1-2, mask
 * units 1-4, first 1^3 conv, its BN, second 1^3 conv.  The gradient arena has
 * the same layout.  Caller owns both arenas and the workspace.
 * ------------------------------------------------------------------------ */
typedef enum {
    RAT3D_NET_RESUNIT = 1,
    RAT3D_NET_ATTN = 2,
    RAT3D_NET_RESATTNET = 3,
    RAT3D_NET_PARTITION1 = 4
} rat3d_net_kind;

typedef struct {
    rat3d_net_kind kind;
    int n;               /* volumes per (micro-)batch */
    int c_in;            /* input channels (1 for RESATTNET / PARTITION1) */
    int c;               /* block channels (RESUNIT, ATTN, PARTITION1) */
    int d, h, w;         /* input volume */
    int micro_batches;   /* PARTITION1: micro-batches per step (>= 1); else 1 */
    float lr;            /* SGD learning rate */
    float bn_eps;        /* BN epsilon */
    float bn_momentum;   /* BN running-statistics momentum */
    rat3d_dtype dtype;
} rat3d_net_desc;

typedef struct rat3d_net rat3d_net;

/* Host-side plan of the network (shapes, arena and workspace layout). */
rat3d_status rat3d_net_create(const rat3d_net_desc* desc, rat3d_net** out);
void rat3d_net_destroy(rat3d_net* net);

/* float32 elements of the parameter (and gradient) arena. */
size_t rat3d_net_param_count(const rat3d_net* net);

/* Bytes of workspace: saved activations, activation gradients, bf16 weight
 * copies, BN statistics and scratch (PARTITION1 with several micro-batches:
 * two copies of the per-micro-batch part, see rat3d_train_step). */
size_t rat3d_net_workspace_size(const rat3d_net* net);

/* Number of parameter tensors, and the i-th one's name, arena offset
 * (elements) and shape (unused trailing dims are 1; *ndim set). */
int rat3d_net_num_params(const rat3d_net* net);
rat3d_status rat3d_net_param_info(const rat3d_net* net, int i, const char** name,
                                  size_t* offset, int* ndim, int shape[5]);

/* Tensors kept in the workspace (activations, statistics, logits, loss),
 * for inspection: name, byte offset, dtype, shape [n, c, d, h, w]. */
int rat3d_net_num_tensors(const rat3d_net* net);
rat3d_status rat3d_net_tensor_info(const rat3d_net* net, int i, const char** name,
                                   size_t* byte_offset, rat3d_dtype* dtype, int shape[5]);

/* Binds the caller's device buffers: params and grads (float32 arenas) and
 * the workspace.  Also resets BN running statistics (mean 0, var 1) when the
 * kernels next run: the reset is enqueued by the next call that takes a
 * stream.  PARTITION1 with several micro-batches, RESATTNET and ATTN: the
 * first bind also creates the network's streams (default priority) and
 * events, released by rat3d_net_destroy; RAT3D_EHIP if the runtime refuses
 * them. */
rat3d_status rat3d_net_bind(rat3d_net* net, float* params, float* grads, void* ws,
                            size_t ws_bytes);

/* Whether rat3d_train_step and rat3d_block_fwd_bwd run independent work
 * concurrently (enable != 0, the default) or every kernel on the caller's
 * stream in order (enable == 0, for per-kernel timing).  Concurrent:
 * PARTITION1 overlaps micro-batches, every attention module runs its mask
 * branch on a stream of the network's own next to its trunk, and RESATTNET
 * and ATTN run their weight gradients on another.  Both give bit-identical
 * results. */
rat3d_status rat3d_net_set_overlap(rat3d_net* net, int enable);

/* RESUNIT / ATTN: forward on x (input shape), backward from dy (output
 * shape); writes y, dx and the gradient arena (overwritten).  No update. */
rat3d_status rat3d_block_fwd_bwd(rat3d_net* net, const void* x, const void* dy, void* y,
                                 void* dx, void* stream);

/* RESATTNET: x [n][1][d][h][w], labels int32 [n]; dy_upstream unused.
 * PARTITION1: x [micro_batches*n][1][d][h][w], dy_upstream [micro_batches*n]
 * [c][d/2][h/2][w/2]; labels unused.
 * One training step: gradients (overwritten, then summed over micro-batches
 * in order) and params -= lr * grads.  loss_dev (nullable, RESATTNET)
 * receives the loss.  PARTITION1 with overlap on: micro-batch k + 1's forward
 * runs on the network's own stream while micro-batch k's backward runs on
 * `stream`, in two alternating copies of the saved activations (the last
 * micro-batch in the copy rat3d_net_tensor_info describes); the caller's
 * stream waits for all of it, so work enqueued after the call sees the
 * update.  The call enqueues kernels, stream-ordered copies and event
 * waits only, and every stream it forks joins `stream` again before it
 * returns, so a caller may capture it into a HIP graph from `stream` and
 * replay that graph (the buffers bound at rat3d_net_bind stay fixed).  While
 * `stream` is capturing, PARTITION1 enqueues its micro-batches one after
 * another (the two-stream overlap is not captured); the mask-branch and
 * weight-gradient streams are captured as forked work. */
rat3d_status rat3d_train_step(rat3d_net* net, const void* x, const int32_t* labels,
                              const void* dy_upstream, float* loss_dev, void* stream);

/* RESATTNET: 3D Grad-CAM, the explainable block of the use-case section
 * (gradient-weighted class activation mapping), in inference mode: every BN
 * applies the running statistics held in the workspace (mean 0 / var 1 after
 * rat3d_net_bind, updated by rat3d_train_step or set by
 * rat3d_net_running_load), no parameter or its gradient is changed.
 *   x        [n][1][d][h][w] in the network dtype (device);
 *   classes  int32 [n] (device): the class k whose logit is explained for
 *            each volume (clamped into [0, 1]);
 *   target   the explained map A: 0 = the stem's pooled output, s = 1..3 =
 *            the output of stage s's attention module;
 *   logits   float32 [n][2] (device, nullable): the inference-mode logits;
 *   cam      float32 [n][D_t][H_t][W_t] (device): ReLU(sum_c alpha_c A_c),
 *            alpha_c = mean over voxels of d logit_k / d A_c, at the target's
 *            resolution (rat3d_gradcam_shape gives C_t, D_t, H_t, W_t);
 *   cam_up   float32 [n][d][h][w] (device, nullable): cam resampled
 *            trilinearly (half-pixel centres) to the input's size.
 * Uses the network's workspace (the saved activations and gradients are
 * overwritten). */
rat3d_status rat3d_gradcam_shape(const rat3d_net* net, int target, int shape[4]);
rat3d_status rat3d_gradcam(rat3d_net* net, const void* x, const int32_t* classes, int target,
                           float* logits, float* cam, float* cam_up, void* stream);

/* PARTITION1, one micro-batch at a time (model-parallelisation section: a
 * partition processes micro-batches one after another, computing its weight
 * gradients from the gradient received at its output and accumulating them
 * before the update).  x [n][1][d][h][w] is one micro-batch, dy_upstream
 * [n][c][d/2][h/2][w/2] its output gradient.  Forward and backward of the
 * micro-batch; the gradient arena is overwritten (accumulate == 0) or added
 * to (accumulate != 0).  No update: rat3d_net_update applies it.  The saved
 * activations and gradients in the workspace are those of this micro-batch.
 * rat3d_train_step computes exactly these calls (accumulate = 0 for the
 * first micro-batch, 1 after), then rat3d_net_update. */
rat3d_status rat3d_partition_micro_batch(rat3d_net* net, const void* x, const void* dy_upstream,
                                         int accumulate, void* stream);

/* params -= lr * grads over the whole arena (the network's SGD step). */
rat3d_status rat3d_net_update(rat3d_net* net, void* stream);

/* Checkpointing of the BN running statistics, which live in the workspace
 * (the parameter arena is the caller's and is saved by the caller).
 * rat3d_net_running_count: number of BN channels in the network, R.
 * rat3d_net_running_save copies [means R][variances R] (float32, device) to
 * dst; it fails (RAT3D_EINVAL) if no step has run since rat3d_net_bind.
 * rat3d_net_running_load copies them from src into the workspace and cancels
 * the reset that rat3d_net_bind scheduled.  Both enqueue device-to-device
 * copies on `stream`. */
size_t rat3d_net_running_count(const rat3d_net* net);
rat3d_status rat3d_net_running_save(const rat3d_net* net, float* dst, void* stream);
rat3d_status rat3d_net_running_load(rat3d_net* net, const float* src, void* stream);

/* ------------------------------------------------------------------------
 * GABRA: allocation of the partitions of a model-parallel split to GPUs by
 * a genetic algorithm (model-parallelisation section, "Genetic Algorithm
 * Based Resource Allocation": eqs. 3-10, Algorithms 1-3).  Host-only: every
 * pointer here is HOST memory, nothing is enqueued.
 *   loads[n] (p_i > 0): computation load of each partition;
 *   capacities[m] (d_j > 0): capacity of each GPU, in the loads' unit;
 *   profit of running partition i on GPU j: c_ij = p_i / d_j;
 *   maximise sum of c over the allocation (eq. 7) subject to no GPU's load
 *   exceeding its capacity (eq. 8) and each partition on exactly one GPU
 *   (eq. 9); with every_gpu != 0, also every GPU runs a partition (the
 *   paper's stated assumption).
 * Chromosome: gene i = GPU of partition i.  Initial population: each
 * partition in turn to a GPU drawn uniformly among those with room left (a
 * stuck chromosome is redrawn, at most init_tries times).  Loop: two
 * roulette-wheel parents (probability fitness / total), midpoint crossover
 * with probability crossover_p (paper: 0.8; offspring keep genes at their
 * positions: first half of one parent, second half of the other; one of the
 * two offspring by a fair draw, else a copy of the first parent), inversion
 * mutation of a random segment; an offspring equal to a population member or
 * infeasible is dropped (selection starts over); otherwise it replaces the
 * worst member and becomes the best if strictly fitter.  Stops after
 * `generations` accepted offspring or max_attempts offspring in all.
 * Random numbers: SplitMix64 seeded with `seed` (deterministic for a seed).
 * Output: assignment[n] (GPU index of each partition, 0-based) and *profit of
 * the best allocation found; stats (nullable) receives the counters.
 * RAT3D_EINVAL on invalid arguments or when no feasible initial chromosome
 * is found (e.g. total capacity below total load). */
typedef struct {
    int population;       /* chromosomes, >= 2 */
    int generations;      /* t_max: offspring accepted into the population */
    double crossover_p;   /* in [0, 1] */
    uint64_t seed;        /* SplitMix64 seed */
    int every_gpu;        /* nonzero: every GPU must run at least one partition */
    int64_t max_attempts; /* offspring drawn in all; 0 = 50 * generations */
    int init_tries;       /* redraws of a stuck initial chromosome; 0 = 1000 */
} rat3d_gabra_params;

typedef struct {
    int64_t generations, duplicates, infeasible, attempts;
} rat3d_gabra_stats;

rat3d_status rat3d_gabra(int n, const double* loads, int m, const double* capacities,
                         const rat3d_gabra_params* params, int32_t* assignment, double* profit,
                         rat3d_gabra_stats* stats);

/* ------------------------------------------------------------------------
 * Measurement (off by default).  While enabled, every launch of a hot kernel
 * is bracketed by two hipEvents recorded on the stream it is launched on, and
 * the operation's algorithmic work is added to its tag: convolutions count
 * 2 * N * C_out * C_in * k^3 * (output voxels) flops per pass (the cost
 * formula of the use-case section, two flops per multiply-add), elementwise
 * kernels the bytes they must read and write once.  Reading a tag waits for
 * its pending events.  Not for use while another thread launches work.
 * ------------------------------------------------------------------------ */
rat3d_status rat3d_profile_enable(int enable);
/* Restricts the brackets to launches whose tag equals `tag` (a copy is kept);
 * NULL or "" brackets every tagged launch again.  Other launches record no
 * events and add nothing, so one kernel can be timed inside a region without
 * an event pair around every other launch. */
rat3d_status rat3d_profile_filter(const char* tag);
rat3d_status rat3d_profile_reset(void);
int rat3d_profile_count(void);
rat3d_status rat3d_profile_read(int i, const char** name, int64_t* launches, double* total_ms,
                                double* alg_flops, double* alg_bytes);

/* Achievable-peak probes (measurement only; they touch no training data).
 * rat3d_probe_mfma: `blocks` workgroups of 4 waves, each wave issuing `iters`
 * iterations of 4 independent bf16 MFMAs (16x16x32); sink [blocks * 256]
 * float32 (device) receives per-lane sums.  rat3d_probe_mfma_flops gives the
 * flops of such a launch.  rat3d_probe_copy: dst = src over `bytes` (a
 * multiple of 16; both 16-byte aligned) with 16-byte accesses. */
double rat3d_probe_mfma_flops(int blocks, int iters);
rat3d_status rat3d_probe_mfma(int blocks, int iters, float* sink, void* stream);
rat3d_status rat3d_probe_copy(const void* src, void* dst, size_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RAT3D_H */
