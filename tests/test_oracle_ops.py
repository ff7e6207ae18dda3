"""Pins for the oracle's non-convolution operations: bfloat16 rounding, max
pooling, trilinear resampling, batch norm, the soft-mask fuse, the head and
SGD.  Each is checked against closed forms, invariants, finite differences or
an independent library (torch CPU, float64)."""
import math

import numpy as np
import pytest

from oracle import ops

RNG = np.random.default_rng(11)


def _rand(*shape):
    return RNG.standard_normal(shape)


# ---------------------------------------------------------------- rounding
def test_round_bf16_matches_torch_conversion():
    torch = pytest.importorskip("torch")
    vals = np.concatenate([
        RNG.standard_normal(20000).astype(np.float32) * 10.0 ** RNG.integers(-30, 30, 20000),
        # exact ties between two bf16 neighbours, both parities
        (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, 1e-40, np.inf, -np.inf], dtype=np.float32),
    ]).astype(np.float32)
    ref = torch.tensor(vals).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ops.round_bf16(vals.astype(np.float64)), ref)


def test_round_bf16_ties_to_even():
    one = 1.0
    ulp = 2.0 ** -7  # bfloat16 spacing at 1.0
    assert ops.round_bf16(np.array([one + ulp / 2]))[0] == one          # tie -> even
    assert ops.round_bf16(np.array([one + 1.5 * ulp]))[0] == one + 2 * ulp
    assert np.isnan(ops.round_bf16(np.array([np.nan]))[0])


# ---------------------------------------------------------------- max pool
def test_maxpool_constant_and_ramp():
    x = np.full((1, 2, 7, 6, 5), 3.25)
    y, am = ops.maxpool3d_fwd(x)
    assert y.shape == (1, 2, 4, 3, 3) and np.all(y == 3.25)
    # ties: first maximum in scan order -> the first in-bounds tap
    assert am[0, 0, 0, 0, 0] == 13 and am[0, 0, 1, 1, 1] == 0
    d, h, w = np.meshgrid(np.arange(7), np.arange(6), np.arange(5), indexing="ij")
    ramp = (100 * d + 10 * h + w).astype(np.float64)[None, None]
    y, am = ops.maxpool3d_fwd(ramp)
    for od in range(4):
        for oh in range(3):
            for ow in range(3):
                dd, hh, ww = min(2 * od + 1, 6), min(2 * oh + 1, 5), min(2 * ow + 1, 4)
                assert y[0, 0, od, oh, ow] == 100 * dd + 10 * hh + ww
                kd, kh, kw = dd - 2 * od + 1, hh - 2 * oh + 1, ww - 2 * ow + 1
                assert am[0, 0, od, oh, ow] == (kd * 3 + kh) * 3 + kw


def test_maxpool_against_torch():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    for shape in [(2, 3, 9, 8, 7), (1, 2, 6, 7, 6), (1, 1, 3, 4, 3), (1, 1, 2, 2, 2)]:
        x = _rand(*shape)
        xt = torch.tensor(x, requires_grad=True)
        yt, it = F.max_pool3d(xt, 3, 2, 1, return_indices=True)
        y, am = ops.maxpool3d_fwd(x)
        np.testing.assert_array_equal(y, yt.detach().numpy())
        # convert the window offset into torch's flat input index
        N, C, D, H, W = shape
        Do, Ho, Wo = y.shape[2:]
        od, oh, ow = np.meshgrid(np.arange(Do), np.arange(Ho), np.arange(Wo), indexing="ij")
        kd, kh, kw = am // 9, (am // 3) % 3, am % 3
        flat = ((2 * od - 1 + kd) * H + (2 * oh - 1 + kh)) * W + (2 * ow - 1 + kw)
        np.testing.assert_array_equal(flat, it.numpy())
        dy = _rand(*y.shape)
        yt.backward(torch.tensor(dy))
        np.testing.assert_allclose(ops.maxpool3d_bwd(dy, am, shape), xt.grad.numpy(),
                                   rtol=1e-14, atol=1e-14)


def test_maxpool_bwd_conserves_mass():
    x = _rand(2, 3, 8, 7, 6)
    y, am = ops.maxpool3d_fwd(x)
    dy = _rand(*y.shape)
    dx = ops.maxpool3d_bwd(dy, am, x.shape)
    np.testing.assert_allclose(dx.sum(axis=(2, 3, 4)), dy.sum(axis=(2, 3, 4)), atol=1e-12)
    base = _rand(*x.shape)
    acc = base.copy()
    ops.maxpool3d_bwd(dy, am, x.shape, out=acc)
    np.testing.assert_allclose(acc, base + dx, atol=1e-14)


# ---------------------------------------------------------------- trilinear
def test_trilinear_constant_and_affine():
    x = np.full((1, 2, 3, 4, 5), -1.5)
    np.testing.assert_array_equal(ops.trilinear_fwd(x, (6, 8, 10)), np.full((1, 2, 6, 8, 10), -1.5))
    # affine field a.(i) + b is reproduced exactly where no clamping happens
    Di, Hi, Wi, Do, Ho, Wo = 6, 7, 6, 12, 14, 12
    d, h, w = np.meshgrid(np.arange(Di), np.arange(Hi), np.arange(Wi), indexing="ij")
    f = (0.5 * d - 0.25 * h + 2.0 * w + 1.0)[None, None]
    y = ops.trilinear_fwd(f, (Do, Ho, Wo))
    src = lambda o, i, O: (o + 0.5) * i / O - 0.5
    for od in range(1, Do - 1):
        for oh in range(1, Ho - 1):
            for ow in range(1, Wo - 1):
                e = 0.5 * src(od, Di, Do) - 0.25 * src(oh, Hi, Ho) + 2.0 * src(ow, Wi, Wo) + 1.0
                assert abs(y[0, 0, od, oh, ow] - e) < 1e-12


def test_trilinear_axis_values_by_hand():
    # length 2 -> 4 along W: src = -0.25 (clamped to 0), 0.25, 0.75, 1.25 (i0 = i1 = 1)
    x = np.zeros((1, 1, 1, 1, 2))
    x[..., 1] = 1.0
    np.testing.assert_allclose(ops.trilinear_fwd(x, (1, 1, 4))[0, 0, 0, 0],
                               [0.0, 0.25, 0.75, 1.0], atol=0)


@pytest.mark.parametrize("sizes", [((6, 7, 6), (12, 14, 12)), ((3, 4, 3), (6, 7, 6)),
                                   ((2, 2, 2), (3, 4, 3)), ((12, 12, 12), (24, 24, 24)),
                                   ((5, 3, 4), (5, 9, 7))])
def test_trilinear_against_torch_and_adjoint(sizes):
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    (Di, Hi, Wi), (Do, Ho, Wo) = sizes
    x = _rand(2, 3, Di, Hi, Wi)
    xt = torch.tensor(x, requires_grad=True)
    yt = F.interpolate(xt, size=(Do, Ho, Wo), mode="trilinear", align_corners=False)
    y = ops.trilinear_fwd(x, (Do, Ho, Wo))
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-13, atol=1e-13)
    r = _rand(*y.shape)
    yt.backward(torch.tensor(r))
    dx = ops.trilinear_bwd(r, (Di, Hi, Wi))
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    assert abs(np.sum(y * r) - np.sum(x * dx)) < 1e-10
    np.testing.assert_allclose(dx.sum(axis=(2, 3, 4)), r.sum(axis=(2, 3, 4)), atol=1e-11)


# ---------------------------------------------------------------- batch norm
def test_bn_output_moments_closed_form():
    x = 3.0 + 2.0 * _rand(3, 4, 5, 6, 7)
    g, b, eps = _rand(4), _rand(4), 1e-5
    y, mean, var, invstd = ops.bn_fwd(x, g, b, eps, relu=False)
    ym, yv = ops.bn_stats(y)
    np.testing.assert_allclose(ym, b, atol=1e-12)
    np.testing.assert_allclose(yv, g ** 2 * var / (var + eps), rtol=1e-12)
    np.testing.assert_allclose(mean, x.mean(axis=(0, 2, 3, 4)), rtol=1e-13)


def test_bn_bwd_invariants():
    x = _rand(2, 3, 4, 5, 6) + 0.5
    g, b, eps = _rand(3), _rand(3), 1e-5
    y, mean, var, invstd = ops.bn_fwd(x, g, b, eps, relu=False)
    dy = _rand(*x.shape)
    dx, dres, dg, db = ops.bn_bwd(dy, x, y, g, mean, invstd, relu=False)
    np.testing.assert_allclose(dx.sum(axis=(0, 2, 3, 4)), 0.0, atol=1e-10)
    np.testing.assert_allclose(db, dy.sum(axis=(0, 2, 3, 4)), rtol=1e-13)
    xhat = (x - mean[None, :, None, None, None]) * invstd[None, :, None, None, None]
    lhs = (dx * xhat).sum(axis=(0, 2, 3, 4))
    rhs = g * invstd * (eps / (var + eps)) * (dy * xhat).sum(axis=(0, 2, 3, 4))
    np.testing.assert_allclose(lhs, rhs, atol=1e-9)
    np.testing.assert_array_equal(dres, dy)


@pytest.mark.parametrize("relu,resid", [(False, False), (True, False), (True, True)])
def test_bn_against_torch(relu, resid):
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    x = _rand(2, 3, 4, 5, 3)
    g, b, r = _rand(3), _rand(3), _rand(*x.shape)
    xt, gt, bt, rt = (torch.tensor(a, requires_grad=True) for a in (x, g, b, r))
    yt = F.batch_norm(xt, None, None, gt, bt, training=True, eps=1e-5)
    if resid:
        yt = yt + rt
    if relu:
        yt = torch.relu(yt)
    y, mean, var, invstd = ops.bn_fwd(x, g, b, 1e-5, relu, r if resid else None)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = _rand(*x.shape)
    yt.backward(torch.tensor(dy))
    dx, dres, dg, db = ops.bn_bwd(dy, x, y, g, mean, invstd, relu)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-10, atol=1e-10)
    if resid:
        np.testing.assert_allclose(dres, rt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_bn_running_update_closed_form():
    rm, rv = ops.bn_running_update(np.zeros(2), np.ones(2), np.array([1.0, 2.0]),
                                   np.array([4.0, 8.0]), 5, 0.1)
    np.testing.assert_allclose(rm, [0.1, 0.2])
    np.testing.assert_allclose(rv, [0.9 + 0.1 * 5.0, 0.9 + 0.1 * 10.0])


# ---------------------------------------------------------------- soft mask
def test_softmask_special_values():
    t = _rand(2, 3, 4)
    dout = _rand(2, 3, 4)
    out, m = ops.softmask_fwd(np.zeros_like(t), t)
    np.testing.assert_array_equal(out, 1.5 * t)
    dt, dz = ops.softmask_bwd(dout, t, m)
    np.testing.assert_array_equal(dz, 0.25 * dout * t)
    np.testing.assert_array_equal(dt, 1.5 * dout)
    out, m = ops.softmask_fwd(np.full_like(t, -80.0), t)
    np.testing.assert_array_equal(out, t)


def test_softmask_finite_differences():
    z, t, dout = _rand(50), _rand(50), _rand(50)
    out, m = ops.softmask_fwd(z, t)
    dt, dz = ops.softmask_bwd(dout, t, m)
    h = 1e-6
    f = lambda zz, tt: float(np.sum(ops.softmask_fwd(zz, tt)[0] * dout))
    for i in range(0, 50, 7):
        e = np.zeros(50)
        e[i] = h
        assert abs((f(z + e, t) - f(z - e, t)) / (2 * h) - dz[i]) < 1e-8
        assert abs((f(z, t + e) - f(z, t - e)) / (2 * h) - dt[i]) < 1e-8


# ---------------------------------------------------------------- head
def test_ce_uniform_logits_is_ln2():
    loss, dl = ops.ce_fwd_bwd(np.zeros((6, 2)), np.array([0, 1, 1, 0, 1, 0]))
    assert abs(loss - math.log(2.0)) < 1e-15
    np.testing.assert_allclose(dl.sum(axis=1), 0.0, atol=1e-16)
    np.testing.assert_allclose(np.abs(dl), 0.5 / 6)


def test_head_against_torch():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    x = _rand(4, 5, 3, 2, 3)
    w, b = _rand(2, 5), _rand(2)
    lab = np.array([0, 1, 1, 0])
    xt, wt, bt = (torch.tensor(a, requires_grad=True) for a in (x, w, b))
    lt = F.linear(xt.mean(dim=(2, 3, 4)), wt, bt)
    Lt = F.cross_entropy(lt, torch.tensor(lab))
    Lt.backward()
    g = ops.gap_fwd(x)
    logits = ops.fc_fwd(g, w, b)
    loss, dl = ops.ce_fwd_bwd(logits, lab)
    dg, dw, db = ops.fc_bwd(dl, g, w)
    assert abs(loss - Lt.item()) < 1e-13
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12)
    np.testing.assert_allclose(ops.gap_bwd(dg, x.shape[2:]), xt.grad.numpy(), rtol=1e-12)


def test_sgd_closed_form():
    w, g = np.array([1.0, -2.0, 0.5]), np.array([10.0, -20.0, 0.0])
    np.testing.assert_array_equal(ops.sgd(w, g, 0.5), [-4.0, 8.0, 0.5])
