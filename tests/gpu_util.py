"""Helpers for the GPU parity tests: seeded host inputs, transfers, and the
comparison gates.  Tolerances: float32 paths must match the oracle within a
norm-wise relative error of 1e-4 (and max-abs error within 1e-4 * max|ref|);
bfloat16-storage paths (float32 accumulation) within 2e-2 norm-wise."""
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


def check(got, ref, dt, what=""):
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), what
    r = rel(got, ref)
    assert r <= TOL[dt], "%s: relative error %.3e > %.1e" % (what, r, TOL[dt])
    if dt == "f32":
        mx = np.max(np.abs(got - ref))
        assert mx <= 1e-4 * max(np.max(np.abs(ref)), 1e-30), "%s: max abs %.3e" % (what, mx)
    return r


def sync():
    torch_mod().cuda.synchronize()
