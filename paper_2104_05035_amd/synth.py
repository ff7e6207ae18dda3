"""Seeded synthetic inputs for the five workloads.

This module is the only code that both the GPU path's harness and the oracle
tests use.  It draws random numbers and shapes inputs; it performs none of
the training step's arithmetic.

The paper trains on ADNI structural MRI (dataset section), which is
access-controlled and absent here; single-channel volumes of 96x112x96 built
from a Gaussian-blurred normal field inside a random ellipsoid "brain" mask,
z-scored, stand in for it.  Generators: numpy PCG64 seeded with
2104050350 + workload index, sub-streams spawned in a fixed order.
"""
import numpy as np

SEED_BASE = 2104050350

# Workload shapes (N, C_in, C, D, H, W) and options.  Index = position in the
# list of workloads: 0 single conv layer, 1 residual unit, 2 attention module,
# 3 full network step, 4 first-stage partition with 4 micro-batches.
WORKLOADS = {
    0: dict(name="conv3d_layer", n=1, c_in=4, c=8, d=16, h=16, w=16, k=3, stride=1,
            pad=1, bias=True, dtype="f32"),
    1: dict(name="resunit", n=2, c_in=32, c=32, d=32, h=32, w=32, dtype="f32"),
    2: dict(name="attn", n=4, c_in=64, c=64, d=48, h=48, w=48, dtype="bf16"),
    3: dict(name="resattnet", n=8, c_in=1, c=32, d=96, h=112, w=96, dtype="bf16",
            lr=1e-4),
    4: dict(name="partition1", n=16, c_in=1, c=64, d=96, h=112, w=96, dtype="bf16",
            lr=1e-4, micro_batches=4),
}


def streams(workload, count):
    """`count` independent generators for a workload, in a fixed order."""
    ss = np.random.SeedSequence(SEED_BASE + int(workload))
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(count)]


def mri_volumes(rng, n, shape, sigma=2.0):
    """`n` single-channel volumes (n, 1, D, H, W), float32.

    Each: iid N(0,1) field -> separable Gaussian blur (sigma voxels, radius
    4*sigma, reflecting borders) -> multiplied by an axis-aligned ellipsoid
    mask (centre at mid-volume +/- 5% per axis, semi-axes U(0.30, 0.45) of the
    axis length) -> z-scored over the whole volume.
    """
    from scipy.ndimage import gaussian_filter

    D, H, W = shape
    out = np.empty((n, 1, D, H, W), dtype=np.float32)
    grid = np.meshgrid(np.arange(D), np.arange(H), np.arange(W), indexing="ij")
    for i in range(n):
        f = rng.standard_normal((D, H, W))
        f = gaussian_filter(f, sigma=sigma, mode="reflect", truncate=4.0)
        cen = [L / 2.0 + rng.uniform(-0.05, 0.05) * L for L in (D, H, W)]
        ax = [rng.uniform(0.30, 0.45) * L for L in (D, H, W)]
        r2 = sum(((g - c) / a) ** 2 for g, c, a in zip(grid, cen, ax))
        v = f * (r2 <= 1.0)
        v = (v - v.mean()) / v.std()
        out[i, 0] = v.astype(np.float32)
    return out


def init_param(rng, name, shape, bias_std=0.0, perturb_bn=0.0):
    """Initial value of one parameter, by its role (read from its name).

    conv weights: He normal N(0, 2 / fan_in), fan_in = C_in * k^3;
    conv biases: N(0, bias_std) (0 by default); BN gamma 1 and beta 0, each
    plus N(0, perturb_bn) noise when perturb_bn > 0; FC weight N(0, 1/C),
    FC bias 0.
    """
    shape = tuple(shape)
    if name.startswith("fc.w"):
        return rng.normal(0.0, np.sqrt(1.0 / shape[1]), shape)
    if name.startswith("fc.b"):
        return np.zeros(shape)
    if name.endswith(".g"):
        return np.ones(shape) + (rng.normal(0.0, perturb_bn, shape) if perturb_bn else 0.0)
    if name.endswith(".b"):
        return rng.normal(0.0, perturb_bn, shape) if perturb_bn else np.zeros(shape)
    if name.endswith("bias"):
        return rng.normal(0.0, bias_std, shape) if bias_std else np.zeros(shape)
    fan_in = int(np.prod(shape[1:]))
    return rng.normal(0.0, np.sqrt(2.0 / fan_in), shape)


def init_params(rng, layout, **kw):
    """Dict name -> float64 array for an ordered (name, shape) layout."""
    return {name: np.asarray(init_param(rng, name, shape, **kw), dtype=np.float64)
            for name, shape in layout}
