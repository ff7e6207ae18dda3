"""Pins for the oracle's 3D convolution (forward, input gradient, weight
gradient) against facts fixed by mathematics, hand-derived closed forms and an
independent library (torch CPU, float64)."""
import itertools

import numpy as np
import pytest

from oracle import ops

RNG = np.random.default_rng(7)

SHAPES = [  # (N, Ci, Co, D, H, W, k, s, p)
    (2, 3, 4, 5, 6, 7, 3, 1, 1),
    (1, 2, 3, 9, 8, 7, 3, 2, 1),
    (2, 1, 4, 13, 11, 12, 7, 2, 3),
    (1, 3, 2, 6, 5, 7, 1, 2, 0),
    (2, 4, 3, 4, 5, 3, 1, 1, 0),
    (1, 2, 2, 5, 5, 5, 3, 1, 0),
    (1, 2, 3, 6, 7, 5, 2, 2, 1),
]


def _rand(*shape):
    return RNG.standard_normal(shape)


def test_delta_kernel_identity():
    # centred delta: w[c, c, 1, 1, 1] = 1 with k=3, p=1, s=1 reproduces x exactly
    x = _rand(2, 3, 5, 6, 7)
    w = np.zeros((3, 3, 3, 3, 3))
    for c in range(3):
        w[c, c, 1, 1, 1] = 1.0
    assert np.array_equal(ops.conv3d_fwd(x, w, None, 1, 1), x)


def test_shifted_delta_shifts_with_zero_fill():
    x = _rand(1, 2, 4, 5, 6)
    w = np.zeros((2, 2, 3, 3, 3))
    w[0, 0, 0, 1, 2] = 1.0   # reads x[d-1, h, w+1]
    w[1, 1, 2, 0, 1] = 1.0   # reads x[d+1, h-1, w]
    y = ops.conv3d_fwd(x, w, None, 1, 1)
    e0 = np.zeros((4, 5, 6))
    e0[1:, :, :-1] = x[0, 0, :-1, :, 1:]
    e1 = np.zeros((4, 5, 6))
    e1[:-1, 1:, :] = x[0, 1, 1:, :-1, :]
    assert np.array_equal(y[0, 0], e0)
    assert np.array_equal(y[0, 1], e1)


def test_stride2_delta_subsamples():
    x = _rand(2, 2, 7, 8, 9)
    w = np.zeros((2, 2, 3, 3, 3))
    w[0, 0, 1, 1, 1] = w[1, 1, 1, 1, 1] = 1.0
    y = ops.conv3d_fwd(x, w, None, 2, 1)
    assert np.array_equal(y, x[:, :, ::2, ::2, ::2])


def _valid_count(L):
    # taps of a 3-wide, pad-1 window that land inside a length-L axis
    c = np.full(L, 3.0)
    c[0] -= 1
    c[-1] -= 1
    return c


@pytest.mark.parametrize("L", [(4, 5, 6), (1, 3, 2)])
def test_all_ones_closed_form(L):
    Ci, Co = 3, 2
    x = np.ones((2, Ci) + L)
    w = np.ones((Co, Ci, 3, 3, 3))
    y = ops.conv3d_fwd(x, w, None, 1, 1)
    cnt = (_valid_count(L[0])[:, None, None] * _valid_count(L[1])[None, :, None]
           * _valid_count(L[2])[None, None, :])
    if min(L) >= 3:
        # 27*Ci interior, 18*Ci face, 12*Ci edge, 8*Ci corner
        assert cnt[1, 1, 1] == 27 and cnt[0, 1, 1] == 18 and cnt[0, 0, 1] == 12
        assert cnt[0, 0, 0] == 8
    assert np.array_equal(y, np.broadcast_to(Ci * cnt, y.shape))


def test_zero_weight_gives_bias():
    x = _rand(1, 2, 4, 4, 4)
    b = _rand(3)
    y = ops.conv3d_fwd(x, np.zeros((3, 2, 3, 3, 3)), b, 1, 1)
    assert np.array_equal(y, np.broadcast_to(b[None, :, None, None, None], y.shape))


@pytest.mark.parametrize("shape", SHAPES)
def test_adjoint_input(shape):
    N, Ci, Co, D, H, W, k, s, p = shape
    x = _rand(N, Ci, D, H, W)
    w = _rand(Co, Ci, k, k, k)
    y = ops.conv3d_fwd(x, w, None, s, p)
    r = _rand(*y.shape)
    lhs = float(np.sum(y * r))
    rhs = float(np.sum(x * ops.conv3d_dgrad(r, w, x.shape, s, p)))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)) * 10


@pytest.mark.parametrize("shape", SHAPES)
def test_adjoint_weight(shape):
    N, Ci, Co, D, H, W, k, s, p = shape
    x = _rand(N, Ci, D, H, W)
    w = _rand(Co, Ci, k, k, k)
    y = ops.conv3d_fwd(x, w, None, s, p)
    r = _rand(*y.shape)
    dw, db = ops.conv3d_wgrad(x, r, k, s, p, True)
    lhs = float(np.sum(y * r))
    assert abs(lhs - float(np.sum(w * dw))) <= 1e-11 * max(1.0, abs(lhs))
    assert np.allclose(db, r.sum(axis=(0, 2, 3, 4)), rtol=1e-13, atol=1e-12)


def test_wgrad_all_ones_closed_form():
    N, Ci, Co, L = 2, 2, 3, (5, 4, 6)
    x = np.ones((N, Ci) + L)
    dy = np.ones((N, Co) + L)
    dw, _ = ops.conv3d_wgrad(x, dy, 3, 1, 1, False)
    for kd, kh, kw in itertools.product(range(3), repeat=3):
        expect = N * (L[0] - abs(kd - 1)) * (L[1] - abs(kh - 1)) * (L[2] - abs(kw - 1))
        assert np.all(dw[:, :, kd, kh, kw] == expect)


def test_dgrad_all_ones_closed_form():
    Ci, Co, L = 2, 3, (4, 5, 6)
    dy = np.ones((1, Co) + L)
    w = np.ones((Co, Ci, 3, 3, 3))
    dx = ops.conv3d_dgrad(dy, w, (1, Ci) + L, 1, 1)
    cnt = (_valid_count(L[0])[:, None, None] * _valid_count(L[1])[None, :, None]
           * _valid_count(L[2])[None, None, :])
    assert np.array_equal(dx, np.broadcast_to(Co * cnt, dx.shape))


def test_dgrad_accumulates():
    x_shape = (1, 2, 4, 5, 3)
    w = _rand(3, 2, 3, 3, 3)
    dy = _rand(1, 3, 4, 5, 3)
    base = _rand(*x_shape)
    out = base.copy()
    ops.conv3d_dgrad(dy, w, x_shape, 1, 1, out=out)
    assert np.allclose(out, base + ops.conv3d_dgrad(dy, w, x_shape, 1, 1), atol=1e-13)


@pytest.mark.parametrize("shape", SHAPES)
def test_against_torch_float64(shape):
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    N, Ci, Co, D, H, W, k, s, p = shape
    x = _rand(N, Ci, D, H, W)
    w = _rand(Co, Ci, k, k, k)
    b = _rand(Co)
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.conv3d(xt, wt, bt, stride=s, padding=p)
    y = ops.conv3d_fwd(x, w, b, s, p)
    assert y.shape == tuple(yt.shape)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    r = _rand(*y.shape)
    yt.backward(torch.tensor(r))
    np.testing.assert_allclose(ops.conv3d_dgrad(r, w, x.shape, s, p), xt.grad.numpy(),
                               rtol=1e-11, atol=1e-11)
    dw, db = ops.conv3d_wgrad(x, r, k, s, p, True)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-11, atol=1e-11)


def test_finite_differences():
    N, Ci, Co, D, H, W, k, s, p = 1, 2, 2, 4, 3, 5, 3, 2, 1
    x = _rand(N, Ci, D, H, W)
    w = _rand(Co, Ci, k, k, k)
    r = _rand(*ops.conv3d_fwd(x, w, None, s, p).shape)
    f = lambda xx, ww: float(np.sum(ops.conv3d_fwd(xx, ww, None, s, p) * r))
    dx = ops.conv3d_dgrad(r, w, x.shape, s, p)
    dw, _ = ops.conv3d_wgrad(x, r, k, s, p, False)
    h = 1e-6
    for idx in [(0, 0, 0, 0, 0), (0, 1, 3, 2, 4), (0, 1, 1, 1, 2)]:
        e = np.zeros_like(x)
        e[idx] = h
        assert abs((f(x + e, w) - f(x - e, w)) / (2 * h) - dx[idx]) < 1e-7
    for idx in [(0, 0, 0, 0, 0), (1, 1, 2, 2, 2), (1, 0, 1, 2, 0)]:
        e = np.zeros_like(w)
        e[idx] = h
        assert abs((f(x, w + e) - f(x, w - e)) / (2 * h) - dw[idx]) < 1e-7


@pytest.mark.parametrize("shape", SHAPES[:4])
def test_points_agree_with_full(shape):
    N, Ci, Co, D, H, W, k, s, p = shape
    x = _rand(N, Ci, D, H, W)
    w = _rand(Co, Ci, k, k, k)
    b = _rand(Co)
    y = ops.conv3d_fwd(x, w, b, s, p)
    r = _rand(*y.shape)
    pts = np.stack([RNG.integers(0, m, 20) for m in y.shape], axis=1)
    np.testing.assert_allclose(ops.conv3d_fwd_points(x, w, b, s, p, pts),
                               y[tuple(pts.T)], rtol=1e-13, atol=1e-13)
    dx = ops.conv3d_dgrad(r, w, x.shape, s, p)
    pts = np.stack([RNG.integers(0, m, 20) for m in x.shape], axis=1)
    np.testing.assert_allclose(ops.conv3d_dgrad_points(r, w, x.shape, s, p, pts),
                               dx[tuple(pts.T)], rtol=1e-13, atol=1e-13)
    dw, _ = ops.conv3d_wgrad(x, r, k, s, p, False)
    pts = np.stack([RNG.integers(0, m, 20) for m in w.shape], axis=1)
    np.testing.assert_allclose(ops.conv3d_wgrad_points(x, r, k, s, p, pts),
                               dw[tuple(pts.T)], rtol=1e-12, atol=1e-12)


def test_flop_count_follows_cost_formula():
    # O(C_o C_i T H W K_T K_H K_W) multiply-adds, 2 flops each
    assert ops.conv_flops(16, 64, 64, (48, 56, 48), 3) == 2 * 16 * 64 * 64 * 129024 * 27
