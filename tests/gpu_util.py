"""Helpers for the GPU parity tests: seeded host inputs, transfers, and the
comparison gates.

Tolerances (the stated ones): float32 paths must match the oracle within a
norm-wise relative error of 1e-4 (and max-abs error within 1e-4 * max|ref|);
bfloat16-storage paths (float32 accumulation) within 2e-2 norm-wise.

On top of the norm-wise gate every element is bounded (`check`), for results
whose oracle sees the very inputs the GPU saw:
  * stored outputs (kind "out"): |g - o| <= 2 ulp(|o|) + extra + 2^-16 S,
    where o is the oracle's value rounded to the storage type, ulp is that
    type's spacing at |o| (the two sides may round a float32 sum to
    neighbouring values), S = sum of |terms| of the defining sum (the float32
    accumulation error of K <= 64k terms stays below 2^-16 S: sqrt(K) 2^-24),
    and `extra` is the propagated bound of an intermediate that the GPU
    overwrites (a chain of two stores); plus 2^-126, since float32 results
    below the normal range may be flushed to zero;
  * float32 sums over voxels (kind "sum": weight, bias and BN-parameter
    gradients, BN means): |g - o| <= extra + min(2^-12, tol) S, where S is
    the sum of |terms| (float32 sums of up to 16 M terms: sqrt(K) 2^-24 <=
    2^-12).  Per-channel BN sums that cancel by construction are gated this
    way only (norm=False).
S >= |o| always, so elements within the bound taken with S = |o| pass without
evaluating S; S is computed (fully, or by a callable at the remaining element
indices) only for the others."""
import numpy as np

TOL = {"f32": 1e-4, "bf16": 2e-2}


def torch_mod():
    import torch
    return torch


def tdtype(dt):
    torch = torch_mod()
    return torch.float32 if dt == "f32" else torch.bfloat16


def code(dt):
    from paper_2104_05035_amd import rat3d as R
    return R.F32 if dt == "f32" else R.BF16


def host_tensor(a, dt):
    """CPU torch tensor in the storage dtype, and the exact float64 values it holds."""
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(tdtype(dt))
    return t, t.to(torch.float64).numpy()


def to_dev(t):
    return t.contiguous().to("cuda:0")


def dev_input(a, dt):
    """(device tensor, float64 copy of its exact values)."""
    t, ref = host_tensor(a, dt)
    return to_dev(t), ref


def f64(t):
    torch = torch_mod()
    return t.detach().to("cpu").to(torch.float64).numpy()


def empty(shape, dt):
    torch = torch_mod()
    return torch.empty(shape, dtype=tdtype(dt), device="cuda:0")


def zeros_f32(shape):
    torch = torch_mod()
    return torch.zeros(shape, dtype=torch.float32, device="cuda:0")


def workspace(nbytes):
    torch = torch_mod()
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda:0")


def rel(got, ref):
    d = np.linalg.norm(np.asarray(got, np.float64) - ref)
    n = np.linalg.norm(ref)
    return d / n if n > 0 else d


C_OUT = 2.0 ** -16  # float32 accumulation error of a stored output, per unit of sum|terms|
C_SUM = 2.0 ** -12  # the same for float32 sums over up to 16 M voxels
FLUSH = 2.0 ** -126  # smallest normal float32: results below it may be flushed to zero

LAST = {}  # statistics of the last check: rel, n_above_1ulp, n_terms_evaluated, worst


def ulp(a, dt):
    """Spacing of the storage type at |a| (bfloat16: 8 significant bits)."""
    f = np.abs(np.asarray(a, dtype=np.float64)).astype(np.float32)
    s = np.spacing(f).astype(np.float64)
    return s * 65536.0 if dt == "bf16" else s


def check(got, ref, dt, what="", terms=None, extra=None, kind="out", norm=True):
    """Norm-wise gate at the stated tolerance plus the element-wise bound of
    the module docstring.  `terms`: sum|terms| as an array of ref's shape, or
    a callable taking (P, ndim) integer indices of elements and returning
    their sum|terms|.  Returns the norm-wise relative error."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), what
    r = rel(got, ref)
    if norm:
        assert r <= TOL[dt], "%s: relative error %.3e > %.1e" % (what, r, TOL[dt])
    if dt == "f32" and kind == "out":
        mx = np.max(np.abs(got - ref)) if got.size else 0.0
        assert mx <= 1e-4 * max(np.max(np.abs(ref)) if ref.size else 0.0, 1e-30), \
            "%s: max abs %.3e" % (what, mx)
    d = np.abs(got - ref)
    ex = 0.0 if extra is None else np.broadcast_to(np.asarray(extra, np.float64), ref.shape)
    # FLUSH: float32 results below the normal range may be flushed to zero
    if kind == "out":
        lim = 2.0 * ulp(ref, dt) + ex + FLUSH
        c = C_OUT
    else:
        lim = np.broadcast_to(np.asarray(ex, np.float64), ref.shape) + FLUSH
        c = min(C_SUM, TOL[dt])
    bad = d > lim + c * np.abs(ref)
    nterms = int(bad.sum())
    worst = 0.0
    if nterms:
        assert terms is not None, "%s: %d elements beyond %s bound and no terms given (worst " \
            "|d| %.3e at ref %.3e)" % (what, nterms, kind, d[bad].max(), ref[bad][np.argmax(d[bad])])
        if callable(terms):
            S = np.asarray(terms(np.argwhere(bad)), dtype=np.float64)
        else:
            S = np.broadcast_to(np.asarray(terms, np.float64), ref.shape)[bad]
        allow = lim[bad] + c * S
        ok = d[bad] <= allow
        worst = float(np.max(d[bad] / np.maximum(allow, 1e-300)))
        if not ok.all():
            i = np.argmax(d[bad] - allow)
            pos = np.argwhere(bad)[i]
            raise AssertionError("%s: %d of %d elements beyond the element-wise %s bound; worst "
                                 "at %s: got %.6e ref %.6e |d| %.3e allowed %.3e" % (
                                     what, int((~ok).sum()), got.size, kind, tuple(pos),
                                     got[tuple(pos)], ref[tuple(pos)], d[bad][i], allow[i]))
    n1 = int((d > ulp(ref, dt)).sum()) if kind == "out" else 0
    LAST.clear()
    LAST.update(rel=r, above_1ulp=n1, terms_evaluated=nterms, worst=worst, size=got.size)
    return r


def sync():
    torch_mod().cuda.synchronize()


GUARD = 4096      # bytes of sentinel on each side of a guarded output
SENTINEL = 0xA5


def guarded(shape, dt):
    """An output tensor placed between two 4 KiB sentinel bands: returns
    (tensor view, backing byte buffer).  dt: "f32", "bf16" or a torch dtype."""
    torch = torch_mod()
    tdt = dt if isinstance(dt, torch.dtype) else tdtype(dt)
    es = torch.empty(0, dtype=tdt).element_size()
    nb = int(np.prod(shape)) * es
    buf = torch.full((2 * GUARD + nb,), SENTINEL, dtype=torch.uint8, device="cuda:0")
    return buf[GUARD:GUARD + nb].view(tdt).reshape(shape), buf


def guard_intact(buf, what=""):
    """Both sentinel bands of a guarded buffer unchanged."""
    torch = torch_mod()
    for band, name in ((buf[:GUARD], "before"), (buf[buf.numel() - GUARD:], "after")):
        bad = (band != SENTINEL).nonzero()
        assert bad.numel() == 0, "%s: %d bytes written %s the output (first at offset %d)" % (
            what, bad.numel(), name, int(bad[0]))
    del torch
