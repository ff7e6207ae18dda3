"""ctypes binding of librat3d (include/rat3d.h): argument marshalling only.

Each function has the name of the C entry point it calls and takes torch
tensors for device buffers (their data pointers are passed through) and the
current torch stream.  Every step of the computation runs in the library's
HIP kernels; there is no fallback: if the library is missing or a call fails,
an exception is raised.
"""
import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_build", "librat3d.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "rat3d.h")

OK, EINVAL, EUNSUPPORTED, EALIGN, EWORKSPACE, EHIP = 0, -1, -2, -3, -4, -5
F32, BF16, U8 = 0, 1, 2
NET_RESUNIT, NET_ATTN, NET_RESATTNET, NET_PARTITION1 = 1, 2, 3, 4


class Rat3dError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("rat3d status %d: %s" % (status, msg))
        self.status = status


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("n", "c_in", "c_out", "d", "h", "w", "k", "stride", "pad", "has_bias")] + \
               [("dtype", ctypes.c_int)]


class BnDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("n", "c", "d", "h", "w", "relu")] + \
               [("eps", ctypes.c_float), ("momentum", ctypes.c_float), ("dtype", ctypes.c_int)]


class PoolDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("n", "c", "d", "h", "w", "k", "stride", "pad")] + \
               [("dtype", ctypes.c_int)]


class UpDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("n", "c", "d_in", "h_in", "w_in", "d_out", "h_out", "w_out")] + \
               [("dtype", ctypes.c_int)]


class NetDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("kind", "n", "c_in", "c", "d", "h", "w",
                                            "micro_batches")] + \
               [("lr", ctypes.c_float), ("bn_eps", ctypes.c_float),
                ("bn_momentum", ctypes.c_float), ("dtype", ctypes.c_int)]


class GabraParams(ctypes.Structure):
    _fields_ = [("population", ctypes.c_int), ("generations", ctypes.c_int),
                ("crossover_p", ctypes.c_double), ("seed", ctypes.c_uint64),
                ("every_gpu", ctypes.c_int), ("max_attempts", ctypes.c_int64),
                ("init_tries", ctypes.c_int)]


class GabraStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("generations", "duplicates", "infeasible",
                                              "attempts")]


_lib = None
_VP = ctypes.c_void_p
_I = ctypes.c_int
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_F = ctypes.c_float

_SIGS = {
    "rat3d_last_error": (ctypes.c_char_p, []),
    "rat3d_version": (ctypes.c_char_p, []),
    "rat3d_conv3d_workspace_size": (_SZ, [ctypes.POINTER(ConvDesc), _I]),
    "rat3d_conv3d_fwd": (_I, [ctypes.POINTER(ConvDesc), _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    "rat3d_conv3d_dgrad": (_I, [ctypes.POINTER(ConvDesc), _VP, _VP, _VP, _I, _VP, _SZ, _VP]),
    "rat3d_conv3d_wgrad": (_I, [ctypes.POINTER(ConvDesc), _VP, _VP, _VP, _VP, _I, _VP, _SZ,
                                _VP]),
    "rat3d_conv3d_wgrad_noalloc_max_bytes": (_SZ, []),
    "rat3d_conv3d_wgrad_noalloc": (_I, [ctypes.POINTER(ConvDesc), _VP, _VP, _VP, _VP, _I, _VP]),
    "rat3d_bn_workspace_size": (_SZ, [ctypes.POINTER(BnDesc)]),
    "rat3d_bn_relu_fwd": (_I, [ctypes.POINTER(BnDesc)] + [_VP] * 9 + [_VP, _SZ, _VP]),
    "rat3d_bn_relu_bwd": (_I, [ctypes.POINTER(BnDesc)] + [_VP] * 10 + [_I, _VP, _SZ, _VP]),
    "rat3d_softmask_down_fwd": (_I, [ctypes.POINTER(PoolDesc), _VP, _VP, _VP, _VP]),
    "rat3d_softmask_down_bwd": (_I, [ctypes.POINTER(PoolDesc), _VP, _VP, _VP, _I, _VP]),
    "rat3d_softmask_up_fwd": (_I, [ctypes.POINTER(UpDesc), _VP, _VP, _VP]),
    "rat3d_softmask_up_bwd": (_I, [ctypes.POINTER(UpDesc), _VP, _VP, _I, _VP]),
    "rat3d_softmask_fwd": (_I, [_I64, _I, _VP, _VP, _VP, _VP, _VP]),
    "rat3d_softmask_bwd": (_I, [_I64, _I, _VP, _VP, _VP, _VP, _I, _VP, _VP]),
    "rat3d_head_workspace_size": (_SZ, [_I, _I, _I]),
    "rat3d_head_fwd_bwd": (_I, [_I, _I, _I64, _I, _I] + [_VP] * 9 + [_I, _VP, _SZ, _VP]),
    "rat3d_sgd": (_I, [_I64, _F, _VP, _VP, _VP]),
    "rat3d_net_create": (_I, [ctypes.POINTER(NetDesc), ctypes.POINTER(_VP)]),
    "rat3d_net_destroy": (None, [_VP]),
    "rat3d_net_param_count": (_SZ, [_VP]),
    "rat3d_net_workspace_size": (_SZ, [_VP]),
    "rat3d_net_num_params": (_I, [_VP]),
    "rat3d_net_param_info": (_I, [_VP, _I, ctypes.POINTER(ctypes.c_char_p),
                                  ctypes.POINTER(_SZ), ctypes.POINTER(_I),
                                  ctypes.POINTER(_I * 5)]),
    "rat3d_net_num_tensors": (_I, [_VP]),
    "rat3d_net_tensor_info": (_I, [_VP, _I, ctypes.POINTER(ctypes.c_char_p),
                                   ctypes.POINTER(_SZ), ctypes.POINTER(_I),
                                   ctypes.POINTER(_I * 5)]),
    "rat3d_net_bind": (_I, [_VP, _VP, _VP, _VP, _SZ]),
    "rat3d_net_set_overlap": (_I, [_VP, _I]),
    "rat3d_block_fwd_bwd": (_I, [_VP] * 6),
    "rat3d_train_step": (_I, [_VP] * 6),
    "rat3d_partition_micro_batch": (_I, [_VP, _VP, _VP, _I, _VP]),
    "rat3d_gradcam_shape": (_I, [_VP, _I, ctypes.POINTER(_I * 4)]),
    "rat3d_gradcam": (_I, [_VP, _VP, _VP, _I, _VP, _VP, _VP, _VP]),
    "rat3d_net_update": (_I, [_VP, _VP]),
    "rat3d_net_running_count": (_SZ, [_VP]),
    "rat3d_net_running_save": (_I, [_VP, _VP, _VP]),
    "rat3d_net_running_load": (_I, [_VP, _VP, _VP]),
    "rat3d_gabra": (_I, [_I, _VP, _I, _VP, ctypes.POINTER(GabraParams), _VP, _VP,
                         ctypes.POINTER(GabraStats)]),
    "rat3d_probe_mfma_flops": (ctypes.c_double, [_I, _I]),
    "rat3d_probe_mfma": (_I, [_I, _I, _VP, _VP]),
    "rat3d_probe_copy": (_I, [_VP, _VP, _SZ, _VP]),
    "rat3d_profile_enable": (_I, [_I]),
    "rat3d_profile_filter": (_I, [ctypes.c_char_p]),
    "rat3d_profile_reset": (_I, []),
    "rat3d_profile_count": (_I, []),
    "rat3d_profile_read": (_I, [_I, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(_I64),
                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                ctypes.POINTER(ctypes.c_double)]),
}


def header_symbols():
    """Names of the functions declared in include/rat3d.h."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(rat3d_\w+)\s*\(", txt)))


def lib():
    """The loaded library (built first if no build exists)."""
    global _lib
    if _lib is None:
        # torch supplies the device memory and streams every call uses; it is
        # imported before the library is loaded so that its HIP runtime is
        # loaded first (a HIP call through the library before torch was
        # imported left torch without a visible GPU)
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def last_error():
    return lib().rat3d_last_error().decode()


def _check(status):
    if status != OK:
        raise Rat3dError(status, last_error())


def _p(t):
    """Device pointer of a tensor (None passes NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def dtype_code(torch_dtype):
    import torch
    if torch_dtype == torch.float32:
        return F32
    if torch_dtype == torch.bfloat16:
        return BF16
    raise ValueError("unsupported dtype %s" % torch_dtype)


# ---------------------------------------------------------------- conv
def conv_desc(n, c_in, c_out, d, h, w, k, stride, pad, has_bias, dtype):
    return ConvDesc(n, c_in, c_out, d, h, w, k, stride, pad, int(has_bias), dtype)


def rat3d_conv3d_workspace_size(desc, pass_):
    return lib().rat3d_conv3d_workspace_size(ctypes.byref(desc), pass_)


def rat3d_conv3d_fwd(desc, x, w, bias, y, ws, ws_bytes, stream=None):
    _check(lib().rat3d_conv3d_fwd(ctypes.byref(desc), _p(x), _p(w), _p(bias), _p(y), _p(ws),
                                  ws_bytes, _stream(stream)))


def rat3d_conv3d_dgrad(desc, dy, w, dx, accumulate, ws, ws_bytes, stream=None):
    _check(lib().rat3d_conv3d_dgrad(ctypes.byref(desc), _p(dy), _p(w), _p(dx), int(accumulate),
                                    _p(ws), ws_bytes, _stream(stream)))


def rat3d_conv3d_wgrad(desc, x, dy, dw, dbias, accumulate, ws, ws_bytes, stream=None):
    _check(lib().rat3d_conv3d_wgrad(ctypes.byref(desc), _p(x), _p(dy), _p(dw), _p(dbias),
                                    int(accumulate), _p(ws), ws_bytes, _stream(stream)))


def rat3d_conv3d_wgrad_noalloc_max_bytes():
    return lib().rat3d_conv3d_wgrad_noalloc_max_bytes()


def rat3d_conv3d_wgrad_noalloc(desc, x, dy, dw, dbias, accumulate, stream=None):
    _check(lib().rat3d_conv3d_wgrad_noalloc(ctypes.byref(desc), _p(x), _p(dy), _p(dw),
                                            _p(dbias), int(accumulate), _stream(stream)))


# ---------------------------------------------------------------- batch norm
def rat3d_bn_workspace_size(desc):
    return lib().rat3d_bn_workspace_size(ctypes.byref(desc))


def rat3d_bn_relu_fwd(desc, x, residual, gamma, beta, y, save_mean, save_invstd, run_mean,
                      run_var, ws, ws_bytes, stream=None):
    _check(lib().rat3d_bn_relu_fwd(ctypes.byref(desc), _p(x), _p(residual), _p(gamma),
                                   _p(beta), _p(y), _p(save_mean), _p(save_invstd),
                                   _p(run_mean), _p(run_var), _p(ws), ws_bytes,
                                   _stream(stream)))


def rat3d_bn_relu_bwd(desc, dy, x, y, gamma, save_mean, save_invstd, dx, dresidual, dgamma,
                      dbeta, accumulate, ws, ws_bytes, stream=None):
    _check(lib().rat3d_bn_relu_bwd(ctypes.byref(desc), _p(dy), _p(x), _p(y), _p(gamma),
                                   _p(save_mean), _p(save_invstd), _p(dx), _p(dresidual),
                                   _p(dgamma), _p(dbeta), int(accumulate), _p(ws), ws_bytes,
                                   _stream(stream)))


# ---------------------------------------------------------------- soft mask
def rat3d_softmask_down_fwd(desc, x, y, argmax, stream=None):
    _check(lib().rat3d_softmask_down_fwd(ctypes.byref(desc), _p(x), _p(y), _p(argmax),
                                         _stream(stream)))


def rat3d_softmask_down_bwd(desc, dy, argmax, dx, accumulate, stream=None):
    _check(lib().rat3d_softmask_down_bwd(ctypes.byref(desc), _p(dy), _p(argmax), _p(dx),
                                         int(accumulate), _stream(stream)))


def rat3d_softmask_up_fwd(desc, x, y, stream=None):
    _check(lib().rat3d_softmask_up_fwd(ctypes.byref(desc), _p(x), _p(y), _stream(stream)))


def rat3d_softmask_up_bwd(desc, dy, dx, accumulate, stream=None):
    _check(lib().rat3d_softmask_up_bwd(ctypes.byref(desc), _p(dy), _p(dx), int(accumulate),
                                       _stream(stream)))


def rat3d_softmask_fwd(count, dtype, z, t, out, m, stream=None):
    _check(lib().rat3d_softmask_fwd(count, dtype, _p(z), _p(t), _p(out), _p(m),
                                    _stream(stream)))


def rat3d_softmask_bwd(count, dtype, dout, t, m, dt, accumulate_dt, dz, stream=None):
    _check(lib().rat3d_softmask_bwd(count, dtype, _p(dout), _p(t), _p(m), _p(dt),
                                    int(accumulate_dt), _p(dz), _stream(stream)))


# ---------------------------------------------------------------- head, sgd
def rat3d_head_workspace_size(n, c, classes):
    return lib().rat3d_head_workspace_size(n, c, classes)


def rat3d_head_fwd_bwd(n, c, v, classes, dtype, x, fc_w, fc_b, labels, logits, loss, dx,
                       dfc_w, dfc_b, accumulate, ws, ws_bytes, stream=None):
    _check(lib().rat3d_head_fwd_bwd(n, c, v, classes, dtype, _p(x), _p(fc_w), _p(fc_b),
                                    _p(labels), _p(logits), _p(loss), _p(dx), _p(dfc_w),
                                    _p(dfc_b), int(accumulate), _p(ws), ws_bytes,
                                    _stream(stream)))


def rat3d_sgd(count, lr, params, grads, stream=None):
    _check(lib().rat3d_sgd(count, lr, _p(params), _p(grads), _stream(stream)))


# ---------------------------------------------------------------- GABRA (host)
def rat3d_gabra(loads, capacities, population=20, generations=200, crossover_p=0.8, seed=0,
                every_gpu=False, max_attempts=0, init_tries=0):
    """Host-side GPU allocation; returns (assignment list, profit, stats dict)."""
    import numpy as np
    p = np.ascontiguousarray(loads, dtype=np.float64)
    d = np.ascontiguousarray(capacities, dtype=np.float64)
    out = np.zeros(len(p), dtype=np.int32)
    prof = ctypes.c_double()
    st = GabraStats()
    prm = GabraParams(population, generations, crossover_p, seed & ((1 << 64) - 1),
                      int(every_gpu), max_attempts, init_tries)
    _check(lib().rat3d_gabra(len(p), p.ctypes.data, len(d), d.ctypes.data, ctypes.byref(prm),
                             out.ctypes.data, ctypes.byref(prof), ctypes.byref(st)))
    return ([int(v) for v in out], prof.value,
            {k: getattr(st, k) for k, _ in GabraStats._fields_})


# ---------------------------------------------------------------- measurement
def rat3d_probe_mfma_flops(blocks, iters):
    return lib().rat3d_probe_mfma_flops(blocks, iters)


def rat3d_probe_mfma(blocks, iters, sink, stream=None):
    _check(lib().rat3d_probe_mfma(blocks, iters, _p(sink), _stream(stream)))


def rat3d_probe_copy(src, dst, nbytes, stream=None):
    _check(lib().rat3d_probe_copy(_p(src), _p(dst), nbytes, _stream(stream)))


def rat3d_profile_enable(enable):
    _check(lib().rat3d_profile_enable(int(enable)))


def rat3d_profile_filter(tag=None):
    _check(lib().rat3d_profile_filter(tag.encode() if tag else None))


def rat3d_profile_reset():
    _check(lib().rat3d_profile_reset())


def rat3d_profile_count():
    return lib().rat3d_profile_count()


def rat3d_profile_read(i):
    """(tag, launches, total_ms, alg_flops, alg_bytes) of tag i (waits for its events)."""
    name, n = ctypes.c_char_p(), _I64()
    ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib().rat3d_profile_read(i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms),
                                    ctypes.byref(fl), ctypes.byref(by)))
    return name.value.decode(), n.value, ms.value, fl.value, by.value


# ---------------------------------------------------------------- network
class Net:
    """Owns one rat3d_net handle (host plan); buffers are bound separately."""

    def __init__(self, kind, n, c_in, c, d, h, w, dtype, micro_batches=1, lr=1e-4,
                 bn_eps=1e-5, bn_momentum=0.1):
        desc = NetDesc(kind, n, c_in, c, d, h, w, micro_batches, lr, bn_eps, bn_momentum, dtype)
        h_ = _VP()
        _check(lib().rat3d_net_create(ctypes.byref(desc), ctypes.byref(h_)))
        self.h = h_
        self.desc = desc

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and _lib is not None:
            _lib.rat3d_net_destroy(h)
            self.h = None

    @property
    def param_count(self):
        return lib().rat3d_net_param_count(self.h)

    @property
    def workspace_size(self):
        return lib().rat3d_net_workspace_size(self.h)

    def params(self):
        """[(name, offset, shape)] in arena order."""
        out = []
        for i in range(lib().rat3d_net_num_params(self.h)):
            name, off, nd, shp = ctypes.c_char_p(), _SZ(), _I(), (_I * 5)()
            _check(lib().rat3d_net_param_info(self.h, i, ctypes.byref(name), ctypes.byref(off),
                                              ctypes.byref(nd), ctypes.byref(shp)))
            out.append((name.value.decode(), off.value, tuple(shp[:nd.value])))
        return out

    def tensors(self):
        """{name: (byte_offset, dtype_code, shape)} of workspace tensors."""
        out = {}
        for i in range(lib().rat3d_net_num_tensors(self.h)):
            name, off, dt, shp = ctypes.c_char_p(), _SZ(), _I(), (_I * 5)()
            _check(lib().rat3d_net_tensor_info(self.h, i, ctypes.byref(name), ctypes.byref(off),
                                               ctypes.byref(dt), ctypes.byref(shp)))
            out[name.value.decode()] = (off.value, dt.value, tuple(shp))
        return out

    def rat3d_net_bind(self, params, grads, ws, ws_bytes):
        _check(lib().rat3d_net_bind(self.h, _p(params), _p(grads), _p(ws), ws_bytes))

    def rat3d_net_set_overlap(self, enable):
        _check(lib().rat3d_net_set_overlap(self.h, int(enable)))

    def rat3d_block_fwd_bwd(self, x, dy, y, dx, stream=None):
        _check(lib().rat3d_block_fwd_bwd(self.h, _p(x), _p(dy), _p(y), _p(dx), _stream(stream)))

    def rat3d_train_step(self, x, labels, dy_upstream, loss_dev, stream=None):
        _check(lib().rat3d_train_step(self.h, _p(x), _p(labels), _p(dy_upstream), _p(loss_dev),
                                      _stream(stream)))

    def rat3d_partition_micro_batch(self, x, dy_upstream, accumulate, stream=None):
        _check(lib().rat3d_partition_micro_batch(self.h, _p(x), _p(dy_upstream), int(accumulate),
                                                 _stream(stream)))

    def rat3d_net_update(self, stream=None):
        _check(lib().rat3d_net_update(self.h, _stream(stream)))

    @property
    def running_count(self):
        return lib().rat3d_net_running_count(self.h)

    def rat3d_net_running_save(self, dst, stream=None):
        _check(lib().rat3d_net_running_save(self.h, _p(dst), _stream(stream)))

    def rat3d_net_running_load(self, src, stream=None):
        _check(lib().rat3d_net_running_load(self.h, _p(src), _stream(stream)))

    def rat3d_gradcam_shape(self, target):
        """(C, D, H, W) of the map Grad-CAM explains at `target`."""
        shp = (_I * 4)()
        _check(lib().rat3d_gradcam_shape(self.h, int(target), ctypes.byref(shp)))
        return tuple(shp)

    def rat3d_gradcam(self, x, classes, target, logits, cam, cam_up, stream=None):
        _check(lib().rat3d_gradcam(self.h, _p(x), _p(classes), int(target), _p(logits), _p(cam),
                                   _p(cam_up), _stream(stream)))
