"""Oracle operations in float64 (TEST INFRASTRUCTURE ONLY).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this module.  It shares nothing with the HIP path: the convolution,
pooling and resampling loops live in ``oracle/primitives.c`` (called through
ctypes), the rest are plain numpy expressions of the textbook definitions.

Paper anchors (arXiv 2104.05035):
  * conv block = 3x3x3 3D convolution, 3D batch normalisation, ReLU
    (use-case section, description of the conv blocks and the residual layer);
  * a conv layer costs O(C_o C_i T H W K_T K_H K_W) (same passage);
  * the objective is the mean loss over the batch and its gradient is the mean
    of per-sample gradients (data-parallelisation section, the objective
    f(w;V) and its derivative; with one GPU, m = 1);
  * cross-entropy loss, SGD with initial learning rate 1e-4 (experiments
    section, training parameters);
  * SGD step w <- w - gamma_t * g (model-parallelisation section, the update
    after the per-partition gradient).
Readings where the paper is silent (soft-mask branch, pooling, resampling,
rounding points) are listed in the repository's design notes; each function
below states the reading it implements.
"""
import ctypes
import math

import numpy as np

from . import _build

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = _build.build()
        lib = ctypes.CDLL(path)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        i = ctypes.c_int
        lib.orc_conv3d_fwd.argtypes = [i] * 9 + [dp, dp, dp, dp]
        lib.orc_conv3d_dgrad.argtypes = [i] * 9 + [dp, dp, dp, i]
        lib.orc_conv3d_wgrad.argtypes = [i] * 9 + [dp, dp, dp, dp, i]
        lib.orc_maxpool3d_fwd.argtypes = [i] * 8 + [dp, dp, ip]
        lib.orc_maxpool3d_bwd.argtypes = [i] * 8 + [dp, ip, dp, i]
        lib.orc_trilinear_fwd.argtypes = [i] * 8 + [dp, dp]
        lib.orc_trilinear_bwd.argtypes = [i] * 8 + [dp, dp, i]
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = ctypes.c_int
        lib.orc_conv3d_fwd_points.argtypes = [i] * 9 + [dp, dp, dp, i, ip, dp]
        lib.orc_conv3d_dgrad_points.argtypes = [i] * 9 + [dp, dp, i, ip, dp]
        lib.orc_conv3d_wgrad_points.argtypes = [i] * 9 + [dp, dp, i, ip, dp]
        for f in ("orc_conv3d_fwd", "orc_conv3d_dgrad", "orc_conv3d_wgrad",
                  "orc_conv3d_fwd_points", "orc_conv3d_dgrad_points",
                  "orc_conv3d_wgrad_points",
                  "orc_maxpool3d_fwd", "orc_maxpool3d_bwd",
                  "orc_trilinear_fwd", "orc_trilinear_bwd"):
            getattr(lib, f).restype = None
        _LIB = lib
    return _LIB


def _dptr(a):
    if a is None:
        return None
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _iptr(a):
    assert a.dtype == np.int32 and a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def num_threads():
    """Threads used by the oracle's parallel loops."""
    return _lib().orc_num_threads()


def out_size(i, k, s, p):
    """Output length of a k-tap window with stride s and zero padding p."""
    return (i + 2 * p - k) // s + 1


# --------------------------------------------------------------------------
# Rounding to the storage type
# --------------------------------------------------------------------------
def round_bf16(a):
    """Value of `a` after storage in bfloat16.

    The GPU path accumulates in float32 and stores bfloat16, so the value is
    first rounded to float32 (round-to-nearest-even, numpy's cast) and then to
    the 8-bit-mantissa bfloat16 by round-to-nearest-even on the float32 bit
    pattern: add 0x7FFF plus the lowest kept bit, then clear the low 16 bits.
    NaN stays NaN.
    """
    f = np.ascontiguousarray(a, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = np.nan
    return out


def identity(a):
    return a


# --------------------------------------------------------------------------
# Convolution (zero padding, no dilation, no groups)
# --------------------------------------------------------------------------
def conv3d_fwd(x, w, bias, s, p):
    """y[n,co,o] = bias[co] + sum_{ci,t} w[co,ci,t] x[n,ci,o*s-p+t]."""
    x, w = _f64(x), _f64(w)
    N, Ci, D, H, W = x.shape
    Co, Ci2, k, k2, k3 = w.shape
    assert Ci == Ci2 and k == k2 == k3
    y = np.empty((N, Co, out_size(D, k, s, p), out_size(H, k, s, p),
                  out_size(W, k, s, p)))
    b = None if bias is None else _f64(bias)
    _lib().orc_conv3d_fwd(N, Ci, Co, D, H, W, k, s, p, _dptr(x), _dptr(w),
                          _dptr(b), _dptr(y))
    return y


def conv3d_dgrad(dy, w, in_shape, s, p, out=None):
    """Input gradient of conv3d_fwd; adds into `out` when given."""
    dy, w = _f64(dy), _f64(w)
    N, Ci, D, H, W = in_shape
    Co, _, k, _, _ = w.shape
    acc = out is not None
    dx = out if acc else np.empty(in_shape)
    assert dx.dtype == np.float64 and dx.flags.c_contiguous
    _lib().orc_conv3d_dgrad(N, Ci, Co, D, H, W, k, s, p, _dptr(dy), _dptr(w),
                            _dptr(dx), int(acc))
    return dx


def conv3d_wgrad(x, dy, k, s, p, with_bias):
    """Weight (and bias) gradients of conv3d_fwd."""
    x, dy = _f64(x), _f64(dy)
    N, Ci, D, H, W = x.shape
    Co = dy.shape[1]
    dw = np.empty((Co, Ci, k, k, k))
    db = np.empty(Co) if with_bias else None
    _lib().orc_conv3d_wgrad(N, Ci, Co, D, H, W, k, s, p, _dptr(x), _dptr(dy),
                            _dptr(dw), _dptr(db), 0)
    return dw, db


def _pts(points):
    pts = np.ascontiguousarray(points, dtype=np.int32).reshape(-1, 5)
    return pts, np.empty(pts.shape[0])


def conv3d_fwd_points(x, w, bias, s, p, points):
    """conv3d_fwd evaluated only at `points` = rows (n, co, od, oh, ow)."""
    x, w = _f64(x), _f64(w)
    N, Ci, D, H, W = x.shape
    Co, _, k, _, _ = w.shape
    pts, out = _pts(points)
    b = None if bias is None else _f64(bias)
    _lib().orc_conv3d_fwd_points(N, Ci, Co, D, H, W, k, s, p, _dptr(x), _dptr(w),
                                 _dptr(b), pts.shape[0], _iptr(pts), _dptr(out))
    return out


def conv3d_dgrad_points(dy, w, in_shape, s, p, points):
    """conv3d_dgrad evaluated only at `points` = rows (n, ci, id, ih, iw)."""
    dy, w = _f64(dy), _f64(w)
    N, Ci, D, H, W = in_shape
    Co, _, k, _, _ = w.shape
    pts, out = _pts(points)
    _lib().orc_conv3d_dgrad_points(N, Ci, Co, D, H, W, k, s, p, _dptr(dy), _dptr(w),
                                   pts.shape[0], _iptr(pts), _dptr(out))
    return out


def conv3d_wgrad_points(x, dy, k, s, p, points):
    """conv3d_wgrad weight entries at `points` = rows (co, ci, kd, kh, kw)."""
    x, dy = _f64(x), _f64(dy)
    N, Ci, D, H, W = x.shape
    Co = dy.shape[1]
    pts, out = _pts(points)
    _lib().orc_conv3d_wgrad_points(N, Ci, Co, D, H, W, k, s, p, _dptr(x), _dptr(dy),
                                   pts.shape[0], _iptr(pts), _dptr(out))
    return out


# --------------------------------------------------------------------------
# Soft-mask branch: pooling down, trilinear up, sigmoid fuse
# --------------------------------------------------------------------------
def maxpool3d_fwd(x, k=3, s=2, p=1):
    """Max over each k^3 window (padding never wins); argmax = window offset of
    the first maximum in scan order."""
    x = _f64(x)
    N, C, D, H, W = x.shape
    shp = (N, C, out_size(D, k, s, p), out_size(H, k, s, p), out_size(W, k, s, p))
    y = np.empty(shp)
    am = np.empty(shp, dtype=np.int32)
    _lib().orc_maxpool3d_fwd(N, C, D, H, W, k, s, p, _dptr(x), _dptr(y), _iptr(am))
    return y, am


def maxpool3d_bwd(dy, argmax, in_shape, k=3, s=2, p=1, out=None):
    dy = _f64(dy)
    am = np.ascontiguousarray(argmax, dtype=np.int32)
    N, C, D, H, W = in_shape
    acc = out is not None
    dx = out if acc else np.empty(in_shape)
    _lib().orc_maxpool3d_bwd(N, C, D, H, W, k, s, p, _dptr(dy), _iptr(am),
                             _dptr(dx), int(acc))
    return dx


def trilinear_fwd(x, size):
    """Trilinear resampling to `size` = (D, H, W), half-pixel centres."""
    x = _f64(x)
    N, C, Di, Hi, Wi = x.shape
    Do, Ho, Wo = size
    y = np.empty((N, C, Do, Ho, Wo))
    _lib().orc_trilinear_fwd(N, C, Di, Hi, Wi, Do, Ho, Wo, _dptr(x), _dptr(y))
    return y


def trilinear_bwd(dy, in_size, out=None):
    dy = _f64(dy)
    N, C, Do, Ho, Wo = dy.shape
    Di, Hi, Wi = in_size
    acc = out is not None
    dx = out if acc else np.empty((N, C, Di, Hi, Wi))
    _lib().orc_trilinear_bwd(N, C, Di, Hi, Wi, Do, Ho, Wo, _dptr(dy), _dptr(dx),
                             int(acc))
    return dx


def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def softmask_fwd(z, t, rnd=identity):
    """Attention output (1 + M) * T with M = sigmoid(z).

    Returns (out, m) as stored: both rounded by `rnd`; `out` is formed from the
    unrounded M (the GPU keeps M in a register when it forms the product).
    """
    m = sigmoid(z)
    return rnd((1.0 + m) * t), rnd(m)


def softmask_bwd(dout, t, m, rnd=identity):
    """dT = (1 + M) dout ;  dz = dout * T * M (1 - M), from the stored M."""
    return rnd((1.0 + m) * dout), rnd(dout * t * m * (1.0 - m))


# --------------------------------------------------------------------------
# Batch normalisation (training mode) and ReLU
# --------------------------------------------------------------------------
_AX = (0, 2, 3, 4)


def _bc(v):
    return v[None, :, None, None, None]


def bn_stats(x):
    """Per-channel batch mean and biased variance over N, D, H, W."""
    mean = x.mean(axis=_AX)
    var = ((x - _bc(mean)) ** 2).mean(axis=_AX)
    return mean, var


def bn_fwd(x, gamma, beta, eps, relu, residual=None):
    """y = act(gamma * (x - mean)/sqrt(var + eps) + beta [+ residual]).

    act is ReLU when `relu`, else identity.  Returns (y, mean, var, invstd).
    """
    mean, var = bn_stats(x)
    invstd = 1.0 / np.sqrt(var + eps)
    y = _bc(gamma) * (x - _bc(mean)) * _bc(invstd) + _bc(beta)
    if residual is not None:
        y = y + residual
    if relu:
        y = np.maximum(y, 0.0)
    return y, mean, var, invstd


def bn_bwd(dy, x, y, gamma, mean, invstd, relu):
    """Gradients of bn_fwd.

    g = dy masked by (y > 0) when `relu` (ReLU passes gradient only where its
    output is positive); g is also the gradient of the residual input.
      dbeta  = sum g,   dgamma = sum g * xhat,
      dx     = gamma * invstd * (g - mean(g) - xhat * mean(g * xhat)).
    Returns (dx, dresidual, dgamma, dbeta).
    """
    g = dy * (y > 0.0) if relu else dy.copy()
    xhat = (x - _bc(mean)) * _bc(invstd)
    cnt = x.shape[0] * x.shape[2] * x.shape[3] * x.shape[4]
    dbeta = g.sum(axis=_AX)
    dgamma = (g * xhat).sum(axis=_AX)
    dx = _bc(gamma * invstd) * (g - _bc(dbeta / cnt) - xhat * _bc(dgamma / cnt))
    return dx, g, dgamma, dbeta


def bn_eval_fwd(x, gamma, beta, run_mean, run_var, eps, relu, residual=None):
    """Inference-mode BN: y = act(gamma * (x - run_mean) / sqrt(run_var + eps)
    + beta [+ residual]) with the running statistics in place of the batch's."""
    s = gamma / np.sqrt(run_var + eps)
    y = _bc(s) * (x - _bc(run_mean)) + _bc(beta)
    if residual is not None:
        y = y + residual
    return np.maximum(y, 0.0) if relu else y


def bn_eval_bwd(dy, y, gamma, run_var, eps, relu):
    """Gradients of bn_eval_fwd with respect to x and the residual: the map is
    affine per channel, so dx = g * gamma / sqrt(run_var + eps) with
    g = dy masked by (y > 0) under ReLU; the residual's gradient is g.
    Returns (dx, g)."""
    g = dy * (y > 0.0) if relu else dy.copy()
    return _bc(gamma / np.sqrt(run_var + eps)) * g, g


def bn_running_update(run_mean, run_var, mean, var, count, momentum):
    """Running statistics: r <- (1 - m) r + m * batch value, with the unbiased
    variance var * count / (count - 1)."""
    unb = var * count / max(count - 1, 1)
    return ((1.0 - momentum) * run_mean + momentum * mean,
            (1.0 - momentum) * run_var + momentum * unb)


# --------------------------------------------------------------------------
# Classifier head and loss
# --------------------------------------------------------------------------
def gap_fwd(x):
    """Global average pool over D, H, W: (N, C, D, H, W) -> (N, C)."""
    return x.mean(axis=(2, 3, 4))


def gap_bwd(dg, spatial):
    D, H, W = spatial
    return np.broadcast_to(dg[:, :, None, None, None] / (D * H * W),
                           dg.shape + (D, H, W)).copy()


def fc_fwd(g, w, b):
    """logits[n, j] = sum_c w[j, c] g[n, c] + b[j]."""
    return g @ w.T + b


def fc_bwd(dl, g, w):
    """Returns (dg, dw, db)."""
    return dl @ w, dl.T @ g, dl.sum(axis=0)


def ce_fwd_bwd(logits, labels):
    """Mean softmax cross-entropy over the batch and its logit gradient.

    loss = (1/N) sum_n [log sum_j exp(l_nj) - l_n,label_n]
    dl   = (softmax(l) - onehot(label)) / N
    """
    N = logits.shape[0]
    mx = logits.max(axis=1, keepdims=True)
    lse = mx[:, 0] + np.log(np.exp(logits - mx).sum(axis=1))
    loss = float(np.mean(lse - logits[np.arange(N), labels]))
    sm = np.exp(logits - lse[:, None])
    onehot = np.zeros_like(logits)
    onehot[np.arange(N), labels] = 1.0
    return loss, (sm - onehot) / N


def sgd(w, g, lr):
    """Plain SGD step w <- w - lr * g (no momentum, no weight decay)."""
    return w - lr * g


def conv_flops(n, c_in, c_out, out_spatial, k):
    """Multiply-adds of one conv pass, counted as 2 flops each:
    2 * N * C_o * C_i * T*H*W (output) * K_T*K_H*K_W."""
    return 2 * n * c_out * c_in * int(np.prod(out_spatial)) * k ** 3


def ln2():
    return math.log(2.0)
