"""GPU parity of each C-ABI operation against the oracle, element by element,
at sizes the oracle finishes in seconds: several tiles, ragged tails, odd
volumes, both storage types, and the degenerate cases (one voxel, one
channel).  Gates: see tests/gpu_util.py."""
import zlib

import numpy as np
import pytest

from oracle import ops
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

CONV_CASES = [
    # N, Ci, Co, D, H, W, k, s, p, bias, dtype
    (1, 4, 8, 16, 16, 16, 3, 1, 1, True, "f32"),
    (2, 3, 5, 7, 9, 11, 3, 1, 1, False, "f32"),
    (2, 32, 32, 9, 10, 13, 3, 1, 1, False, "f32"),
    (2, 32, 64, 9, 10, 13, 3, 1, 1, False, "bf16"),
    (2, 64, 64, 12, 14, 12, 3, 1, 1, False, "bf16"),
    (1, 64, 64, 5, 16, 48, 3, 1, 1, False, "bf16"),
    (1, 1, 32, 20, 22, 18, 7, 2, 3, False, "bf16"),
    (2, 64, 128, 12, 14, 12, 3, 2, 1, False, "bf16"),
    (2, 32, 64, 10, 9, 8, 1, 1, 0, False, "bf16"),
    (2, 64, 128, 12, 14, 12, 1, 2, 0, False, "bf16"),
    # pipelined strided forward: ragged rows and output channels, bias
    (3, 32, 40, 9, 11, 7, 3, 2, 1, True, "bf16"),
    # pipelined strided input gradient: ragged rows and input channels
    (2, 40, 64, 9, 11, 7, 3, 2, 1, False, "bf16"),
    (2, 64, 64, 6, 7, 6, 1, 1, 0, True, "bf16"),
    (1, 1, 1, 1, 1, 1, 1, 1, 0, True, "f32"),
    (1, 2, 3, 2, 2, 2, 3, 1, 1, False, "bf16"),
    (3, 5, 70, 5, 3, 4, 3, 1, 1, True, "bf16"),
    (2, 128, 256, 6, 7, 6, 3, 2, 1, False, "bf16"),
    # LDS-brick paths: full and ragged tiles, 32- and 64-channel output tiles,
    # 1^3 kernels, weight-gradient row bands (W multiple of 8)
    (2, 64, 64, 6, 10, 32, 3, 1, 1, False, "bf16"),
    (1, 32, 64, 5, 9, 24, 3, 1, 1, False, "bf16"),
    (2, 64, 32, 4, 8, 16, 3, 1, 1, False, "bf16"),
    (1, 64, 128, 7, 5, 40, 3, 1, 1, True, "bf16"),
    (2, 64, 64, 5, 9, 24, 1, 1, 0, True, "bf16"),
    (1, 32, 64, 3, 3, 8, 1, 1, 0, False, "bf16"),
    (1, 96, 64, 9, 17, 48, 3, 1, 1, False, "bf16"),
    # 64-channel output tiles (128 spatial tiles or more), ragged in d and h:
    # the input gradient's accumulating drain in two column groups
    (4, 64, 64, 14, 30, 32, 3, 1, 1, False, "bf16"),
    # weight gradient over row bands (W a multiple of 8, at most 56): the widest
    # band, one-row-per-group widths, a single plane, ragged last bands
    (1, 32, 64, 4, 5, 56, 3, 1, 1, False, "bf16"),
    (2, 16, 64, 5, 20, 8, 3, 1, 1, False, "bf16"),
    (1, 64, 64, 1, 12, 16, 3, 1, 1, False, "bf16"),
    # many short step ranges over shallow volumes: with 256 workgroups a range
    # holds 3, 7 or 8 planes, so bands begin at every step position of a
    # range (the first step, the prefetched second and third, and later ones)
    (192, 16, 64, 4, 1, 4, 3, 1, 1, False, "bf16"),
    (448, 16, 64, 4, 1, 8, 3, 1, 1, False, "bf16"),
    (320, 16, 64, 6, 2, 16, 3, 1, 1, False, "bf16"),
    # weight-gradient bricks on maps wider than a band
    (1, 64, 64, 3, 9, 64, 3, 1, 1, False, "bf16"),
    # row bands on widths divisible by 4 but not 8 (half-filled last group of a row)
    (1, 64, 64, 5, 6, 20, 3, 1, 1, False, "bf16"),
    (1, 16, 64, 3, 9, 4, 3, 1, 1, False, "bf16"),
    (1, 32, 64, 3, 7, 52, 3, 1, 1, False, "bf16"),
    # the small deep-stage volumes of the full network (tiles mostly outside)
    (2, 64, 64, 12, 14, 12, 1, 1, 0, False, "bf16"),
    (2, 128, 128, 6, 7, 6, 3, 1, 1, False, "bf16"),
    (2, 256, 256, 3, 4, 3, 3, 1, 1, False, "bf16"),
    (2, 256, 256, 2, 2, 2, 3, 1, 1, False, "bf16"),
    (2, 256, 256, 1, 1, 1, 3, 1, 1, False, "bf16"),
    (2, 256, 256, 3, 4, 3, 1, 1, 0, True, "bf16"),
    # 1^3 weight gradient as a direct GEMM (voxels per volume a multiple of 32)
    (2, 64, 64, 4, 8, 16, 1, 1, 0, True, "bf16"),
    (1, 32, 64, 8, 8, 8, 1, 1, 0, False, "bf16"),
    (3, 80, 48, 4, 4, 8, 1, 1, 0, False, "bf16"),
    # strided input gradients by phase class: float32, stride 3, even kernels,
    # classes without taps (1^3 stride 2), ragged class grids
    (2, 3, 5, 9, 8, 7, 3, 2, 1, False, "f32"),
    (1, 4, 6, 7, 9, 8, 1, 2, 0, True, "f32"),
    (1, 2, 3, 8, 8, 8, 2, 2, 0, False, "f32"),
    (1, 2, 3, 10, 9, 8, 3, 3, 1, False, "bf16"),
    (3, 70, 65, 5, 6, 7, 3, 2, 1, False, "bf16"),
    # stem kernels (1 -> 32, 7^3, stride 2, pad 3): full and ragged tiles
    (2, 1, 32, 24, 30, 32, 7, 2, 3, False, "bf16"),
    (1, 1, 32, 13, 9, 21, 7, 2, 3, False, "bf16"),
    (2, 1, 32, 20, 34, 48, 7, 2, 3, False, "bf16"),
]


def _id(c):
    return "n%d_%dto%d_%dx%dx%d_k%ds%dp%d_%s%s" % (c[0], c[1], c[2], c[3], c[4], c[5], c[6], c[7],
                                                   c[8], c[10], "_bias" if c[9] else "")


@pytest.mark.parametrize("case", CONV_CASES, ids=_id)
def test_conv3d(case):
    """Forward, input gradient (plain and accumulating) and weight gradient
    (plain and accumulating, with the bias gradient) against the oracle; every
    output lies between two 4 KiB sentinel bands that must stay untouched."""
    from paper_2104_05035_amd import rat3d as R
    N, Ci, Co, D, H, W, k, s, p, has_bias, dt = case
    rng = np.random.default_rng(zlib.crc32(repr(case).encode()))
    rnd = ops.round_bf16 if dt == "bf16" else ops.identity
    x, xr = U.dev_input(rng.standard_normal((N, Ci, D, H, W)), dt)
    w, wr = U.dev_input(rng.normal(0, np.sqrt(2.0 / (Ci * k ** 3)), (Co, Ci, k, k, k)), dt)
    b32 = rng.normal(0, 0.1, Co).astype(np.float32)
    bias = U.to_dev(U.torch_mod().from_numpy(b32)) if has_bias else None
    br = b32.astype(np.float64) if has_bias else None
    desc = R.conv_desc(N, Ci, Co, D, H, W, k, s, p, has_bias, U.code(dt))
    Do, Ho, Wo = (ops.out_size(v, k, s, p) for v in (D, H, W))
    ws = U.workspace(max(R.rat3d_conv3d_workspace_size(desc, i) for i in range(3)))
    nbytes = ws.numel()
    # forward
    y, yb = U.guarded((N, Co, Do, Ho, Wo), dt)
    R.rat3d_conv3d_fwd(desc, x, w, bias, y, ws, nbytes)
    yref = rnd(ops.conv3d_fwd(xr, wr, br, s, p))
    # input gradient, plain and accumulated
    dy, dyr = U.dev_input(rng.standard_normal((N, Co, Do, Ho, Wo)), dt)
    dx, dxb = U.guarded((N, Ci, D, H, W), dt)
    R.rat3d_conv3d_dgrad(desc, dy, w, dx, 0, ws, nbytes)
    dxref = ops.conv3d_dgrad(dyr, wr, xr.shape, s, p)
    base0, baser = U.dev_input(rng.standard_normal((N, Ci, D, H, W)), dt)
    base, baseb = U.guarded((N, Ci, D, H, W), dt)
    base.copy_(base0)
    R.rat3d_conv3d_dgrad(desc, dy, w, base, 1, ws, nbytes)
    # weight gradient, plain and accumulated
    torch = U.torch_mod()
    dw, dwb = U.guarded((Co, Ci, k, k, k), torch.float32)
    dw.zero_()
    db, dbb = U.guarded((Co,), torch.float32) if has_bias else (None, None)
    R.rat3d_conv3d_wgrad(desc, x, dy, dw, db, 0, ws, nbytes)
    dw2, dw2b = U.guarded((Co, Ci, k, k, k), torch.float32)
    dw2.fill_(1.0)
    R.rat3d_conv3d_wgrad(desc, x, dy, dw2, None, 1, ws, nbytes)
    U.sync()
    for buf, nm in ((yb, "y"), (dxb, "dx"), (baseb, "dx accumulate"), (dwb, "dw"),
                    (dw2b, "dw accumulate"), (dbb, "db")):
        if buf is not None:
            U.guard_intact(buf, nm)
    dwref, dbref = ops.conv3d_wgrad(xr, dyr, k, s, p, has_bias)
    ax, aw, ady = np.abs(xr), np.abs(wr), np.abs(dyr)
    ty = ops.conv3d_fwd(ax, aw, None if br is None else np.abs(br), s, p)
    tdx = ops.conv3d_dgrad(ady, aw, xr.shape, s, p)
    tdw, tdb = ops.conv3d_wgrad(ax, ady, k, s, p, has_bias)
    U.check(U.f64(y), yref, dt, "y", terms=ty)
    U.check(U.f64(dx), rnd(dxref), dt, "dx", terms=tdx)
    U.check(U.f64(base), rnd(baser + dxref), dt, "dx accumulate", terms=tdx + np.abs(baser))
    U.check(U.f64(dw), dwref, dt, "dw", kind="sum", terms=tdw)
    U.check(U.f64(dw2), dwref + 1.0, dt, "dw accumulate", kind="sum", terms=tdw + 1.0)
    if has_bias:
        U.check(U.f64(db), dbref, dt, "db", kind="sum", norm=False, terms=tdb)


# Maps with fewer brick tiles than CUs split the 32-channel source chunks
# over workgroups (fp32 partials summed in order, then bias, old value and one
# rounding): a bias case, eight splits over 256 source channels, and an odd
# width (element-wise partial stores).
SPLIT_CASES = [
    (2, 64, 64, 12, 14, 12, 3, 1, 1, True, "bf16"),
    (1, 256, 64, 6, 7, 6, 3, 1, 1, False, "bf16"),
    (1, 64, 64, 5, 6, 7, 3, 1, 1, False, "bf16"),
]


@pytest.mark.parametrize("case", SPLIT_CASES, ids=_id)
def test_conv3d_source_split(case):
    """The split forward and input-gradient passes run (their measurement tags
    appear) and match the oracle like every other conv pass."""
    from paper_2104_05035_amd import rat3d as R
    R.rat3d_profile_reset()
    R.rat3d_profile_filter(None)
    R.rat3d_profile_enable(1)
    try:
        test_conv3d(case)
        U.sync()
    finally:
        R.rat3d_profile_enable(0)
    tags = {R.rat3d_profile_read(i)[0] for i in range(R.rat3d_profile_count())}
    for t in ("conv_brick3_fwd_c32_split", "conv_brick3_dgrad_c32_split",
              "conv_brick3_dgrad_acc_c32_split"):
        assert t in tags, "%s not launched (tags: %s)" % (t, sorted(tags))


BN_CASES = [
    (2, 3, 5, 6, 7, "f32"), (4, 16, 12, 14, 12, "bf16"), (2, 8, 6, 7, 6, "bf16"),
    (1, 2, 1, 1, 3, "f32"), (3, 4, 3, 4, 3, "bf16"),
]


@pytest.mark.parametrize("case", BN_CASES, ids=lambda c: "%dx%dx%dx%dx%d_%s" % c)
@pytest.mark.parametrize("relu,resid", [(1, False), (0, False), (1, True)])
def test_bn(case, relu, resid):
    from paper_2104_05035_amd import rat3d as R
    torch = U.torch_mod()
    N, C, D, H, W, dt = case
    rng = np.random.default_rng(N * 1000 + C * 10 + relu + 2 * resid)
    rnd = ops.round_bf16 if dt == "bf16" else ops.identity
    shp = (N, C, D, H, W)
    x, xr = U.dev_input(1.5 + 2.0 * rng.standard_normal(shp), dt)
    r, rr = U.dev_input(rng.standard_normal(shp), dt) if resid else (None, None)
    g32 = (1.0 + 0.3 * rng.standard_normal(C)).astype(np.float32)
    b32 = (0.2 * rng.standard_normal(C)).astype(np.float32)
    gamma, beta = U.to_dev(torch.from_numpy(g32)), U.to_dev(torch.from_numpy(b32))
    desc = R.BnDesc(N, C, D, H, W, relu, 1e-5, 0.1, U.code(dt))
    ws = U.workspace(R.rat3d_bn_workspace_size(desc))
    y = U.empty(shp, dt)
    mean, invstd = U.zeros_f32((C,)), U.zeros_f32((C,))
    rm, rv = U.zeros_f32((C,)), U.to_dev(torch.ones(C))
    R.rat3d_bn_relu_fwd(desc, x, r, gamma, beta, y, mean, invstd, rm, rv, ws, ws.numel())
    dy, dyr = U.dev_input(rng.standard_normal(shp), dt)
    dx = U.empty(shp, dt)
    dres = U.empty(shp, dt) if resid else None
    dg, dbt = U.zeros_f32((C,)), U.zeros_f32((C,))
    R.rat3d_bn_relu_bwd(desc, dy, x, y, gamma, mean, invstd, dx, dres, dg, dbt, 0, ws,
                        ws.numel())
    U.sync()
    g64, b64 = g32.astype(np.float64), b32.astype(np.float64)
    _, mref, vref, isref = ops.bn_fwd(xr, g64, b64, 1e-5, relu, rr)
    # the output with the statistics the GPU saved (checked just below)
    bc = lambda v: v[None, :, None, None, None]
    mg, ig = U.f64(mean), U.f64(invstd)
    yref = bc(g64 * ig) * (xr - bc(mg)) + bc(b64) + (0.0 if rr is None else rr)
    yref = rnd(np.maximum(yref, 0.0) if relu else yref)
    sc = g64 * ig
    ty = np.abs(xr) * bc(np.abs(sc)) + bc(np.abs(b64) + np.abs(mg * sc))
    if resid:
        ty = ty + np.abs(rr)
    U.check(U.f64(y), yref, dt, "y", terms=ty)
    U.check(U.f64(mean), mref, "f32", "mean", kind="sum", norm=False,
            terms=np.abs(xr).mean(axis=(0, 2, 3, 4)))
    U.check(U.f64(invstd), isref, "f32", "invstd",
            terms=isref * (xr * xr).mean(axis=(0, 2, 3, 4)) / (vref + 1e-5))
    cnt = N * D * H * W
    rmr, rvr = ops.bn_running_update(np.zeros(C), np.ones(C), mref, vref, cnt, 0.1)
    U.check(U.f64(rm), rmr, "f32", "running mean")
    U.check(U.f64(rv), rvr, "f32", "running var")
    # the ReLU mask is the GPU's stored y > 0 (decision-matched)
    dxr, gr, dgr, dbr = ops.bn_bwd(dyr, xr, U.f64(y), g64, mg, ig, relu)
    M = N * D * H * W
    xh = (xr - bc(mg)) * bc(ig)
    Sg = np.abs(gr).sum(axis=(0, 2, 3, 4))
    Sgx = np.abs(gr * xh).sum(axis=(0, 2, 3, 4))
    tdx = bc(np.abs(sc)) * (np.abs(gr) + bc(Sg / M) + (np.abs(xr) + bc(np.abs(mg)))
                            * bc(ig * Sgx / M))
    U.check(U.f64(dx), rnd(dxr), dt, "dx", terms=tdx)
    U.check(U.f64(dg), dgr, dt, "dgamma", kind="sum", norm=False, terms=Sgx)
    U.check(U.f64(dbt), dbr, dt, "dbeta", kind="sum", norm=False, terms=Sg)
    if resid:
        U.check(U.f64(dres), rnd(gr), dt, "dresidual", terms=np.abs(gr))


POOL_CASES = [(2, 3, 9, 8, 7, "bf16"), (2, 16, 24, 28, 24, "bf16"), (1, 2, 3, 4, 3, "f32"),
              (1, 1, 2, 2, 2, "bf16"), (2, 4, 6, 7, 6, "bf16"), (1, 1, 1, 1, 1, "f32"),
              (1, 2, 48, 56, 48, "bf16"), (1, 1, 5, 300, 7, "f32"),
              # plane-staged bf16 paths: odd depth/height, W a multiple of 8
              (1, 3, 7, 5, 16, "bf16"), (2, 2, 5, 3, 8, "bf16"),
              # the smallest maps of the W % 8 = 0 paths: one plane, one row
              (1, 2, 1, 1, 8, "bf16"), (1, 1, 2, 3, 8, "bf16"), (2, 2, 3, 2, 16, "bf16")]


@pytest.mark.parametrize("case", POOL_CASES, ids=lambda c: "%dx%dx%dx%dx%d_%s" % c)
def test_maxpool(case):
    from paper_2104_05035_amd import rat3d as R
    torch = U.torch_mod()
    N, C, D, H, W, dt = case
    rng = np.random.default_rng(D * 100 + H * 10 + W)
    rnd = ops.round_bf16 if dt == "bf16" else ops.identity
    x, xr = U.dev_input(rng.standard_normal((N, C, D, H, W)), dt)
    yref, amref = ops.maxpool3d_fwd(xr)
    desc = R.PoolDesc(N, C, D, H, W, 3, 2, 1, U.code(dt))
    y = U.empty(yref.shape, dt)
    am = torch.empty(yref.shape, dtype=torch.uint8, device="cuda:0")
    R.rat3d_softmask_down_fwd(desc, x, y, am)
    dy, dyr = U.dev_input(rng.standard_normal(yref.shape), dt)
    dx = U.empty((N, C, D, H, W), dt)
    R.rat3d_softmask_down_bwd(desc, dy, am, dx, 0)
    base, baser = U.dev_input(rng.standard_normal((N, C, D, H, W)), dt)
    R.rat3d_softmask_down_bwd(desc, dy, am, base, 1)
    U.sync()
    np.testing.assert_array_equal(U.f64(y), yref)                      # bit-exact
    np.testing.assert_array_equal(am.cpu().numpy().astype(np.int32), amref)
    dxr = ops.maxpool3d_bwd(dyr, amref, xr.shape)
    tdx = ops.maxpool3d_bwd(np.abs(dyr), amref, xr.shape)
    U.check(U.f64(dx), rnd(dxr), dt, "dx", terms=tdx)
    U.check(U.f64(base), rnd(baser + dxr), dt, "dx accumulate", terms=tdx + np.abs(baser))


# values from a five-element set: most windows hold ties, all-negative windows
# and both signed zeros, so the first-maximum rule decides most argmax bytes
TIE_CASES = [(2, 3, 10, 12, 16), (1, 2, 9, 7, 24), (2, 2, 6, 5, 6), (1, 4, 48, 56, 48)]


@pytest.mark.parametrize("case", TIE_CASES, ids=lambda c: "%dx%dx%dx%dx%d" % c)
def test_maxpool_ties(case):
    from paper_2104_05035_amd import rat3d as R
    torch = U.torch_mod()
    N, C, D, H, W = case
    rng = np.random.default_rng(7 * D + W)
    vals = np.array([-1.0, -0.0, 0.0, 0.5, -0.5])
    x, xr = U.dev_input(vals[rng.integers(0, len(vals), (N, C, D, H, W))], "bf16")
    yref, amref = ops.maxpool3d_fwd(xr)
    desc = R.PoolDesc(N, C, D, H, W, 3, 2, 1, U.code("bf16"))
    y = U.empty(yref.shape, "bf16")
    am = torch.empty(yref.shape, dtype=torch.uint8, device="cuda:0")
    R.rat3d_softmask_down_fwd(desc, x, y, am)
    U.sync()
    np.testing.assert_array_equal(U.f64(y), yref)  # -0 and +0 compare equal
    np.testing.assert_array_equal(am.cpu().numpy().astype(np.int32), amref)


UP_CASES =[((6, 7, 6), (12, 14, 12)), ((3, 4, 3), (6, 7, 6)), ((2, 2, 2), (3, 4, 3)),
            ((12, 12, 12), (24, 24, 24)), ((5, 3, 4), (5, 9, 7)), ((1, 1, 1), (2, 3, 1)),
            ((24, 28, 24), (48, 56, 48)), ((2, 130, 3), (4, 260, 5)),
            # exact x2 with a plane size that is not a multiple of 8, odd depth
            ((3, 5, 4), (6, 10, 8)), ((5, 3, 8), (10, 6, 16)),
            # fine planes of 256-512 groups of 8 (the whole-volume transpose):
            # one coarse plane, and an odd count
            ((1, 16, 32), (2, 32, 64)), ((3, 16, 32), (6, 32, 64))]


@pytest.mark.parametrize("sizes", UP_CASES, ids=lambda s: "%s_to_%s" % s)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_trilinear(sizes, dt):
    from paper_2104_05035_amd import rat3d as R
    (Di, Hi, Wi), (Do, Ho, Wo) = sizes
    rng = np.random.default_rng(Di * 7 + Do)
    rnd = ops.round_bf16 if dt == "bf16" else ops.identity
    N, C = 2, 3
    x, xr = U.dev_input(rng.standard_normal((N, C, Di, Hi, Wi)), dt)
    desc = R.UpDesc(N, C, Di, Hi, Wi, Do, Ho, Wo, U.code(dt))
    y = U.empty((N, C, Do, Ho, Wo), dt)
    R.rat3d_softmask_up_fwd(desc, x, y)
    dy, dyr = U.dev_input(rng.standard_normal((N, C, Do, Ho, Wo)), dt)
    dx = U.empty((N, C, Di, Hi, Wi), dt)
    R.rat3d_softmask_up_bwd(desc, dy, dx, 0)
    base, baser = U.dev_input(rng.standard_normal((N, C, Di, Hi, Wi)), dt)
    R.rat3d_softmask_up_bwd(desc, dy, base, 1)
    U.sync()
    U.check(U.f64(y), rnd(ops.trilinear_fwd(xr, (Do, Ho, Wo))), dt, "y",
            terms=ops.trilinear_fwd(np.abs(xr), (Do, Ho, Wo)))
    dxr = ops.trilinear_bwd(dyr, (Di, Hi, Wi))
    tdx = ops.trilinear_bwd(np.abs(dyr), (Di, Hi, Wi))
    U.check(U.f64(dx), rnd(dxr), dt, "dx", terms=tdx)
    U.check(U.f64(base), rnd(baser + dxr), dt, "dx accumulate", terms=tdx + np.abs(baser))


@pytest.mark.parametrize("count", [1, 1001, 4096, 131072 + 5])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_softmask_fuse(count, dt):
    from paper_2104_05035_amd import rat3d as R
    rng = np.random.default_rng(count)
    rnd = ops.round_bf16 if dt == "bf16" else ops.identity
    z, zr = U.dev_input(3 * rng.standard_normal(count), dt)
    t, tr = U.dev_input(rng.standard_normal(count), dt)
    out, m = U.empty((count,), dt), U.empty((count,), dt)
    R.rat3d_softmask_fwd(count, U.code(dt), z, t, out, m)
    dout, doutr = U.dev_input(rng.standard_normal(count), dt)
    dtt, dz = U.empty((count,), dt), U.empty((count,), dt)
    R.rat3d_softmask_bwd(count, U.code(dt), dout, t, m, dtt, 0, dz)
    acc, accr = U.dev_input(rng.standard_normal(count), dt)
    dz2 = U.empty((count,), dt)
    R.rat3d_softmask_bwd(count, U.code(dt), dout, t, m, acc, 1, dz2)
    U.sync()
    outr, mr = ops.softmask_fwd(zr, tr, rnd)
    mraw = ops.sigmoid(zr)
    U.check(U.f64(out), outr, dt, "out", terms=np.abs((1.0 + mraw) * tr))
    U.check(U.f64(m), mr, dt, "m", terms=mraw)
    # the backward reads the M the GPU stored
    mg = U.f64(m)
    dtr, dzr = ops.softmask_bwd(doutr, tr, mg, rnd)
    U.check(U.f64(dtt), dtr, dt, "dt", terms=np.abs(doutr) * (1.0 + np.abs(mg)))
    U.check(U.f64(dz), dzr, dt, "dz", terms=np.abs(doutr * tr * mg) * (1.0 + np.abs(mg)))
    U.check(U.f64(acc), rnd(accr + (1.0 + mg) * doutr), dt, "dt accumulate",
            terms=np.abs(accr) + np.abs((1.0 + mg) * doutr))


@pytest.mark.parametrize("N,C,V,dt", [(8, 256, 252, "bf16"), (3, 5, 7, "f32"), (1, 1, 1, "f32")])
def test_head(N, C, V, dt):
    from paper_2104_05035_amd import rat3d as R
    torch = U.torch_mod()
    rng = np.random.default_rng(N + C + V)
    rnd = ops.round_bf16 if dt == "bf16" else ops.identity
    x, xr = U.dev_input(rng.standard_normal((N, C, V)) + 0.3, dt)
    w32 = rng.normal(0, np.sqrt(1.0 / C), (2, C)).astype(np.float32)
    b32 = rng.normal(0, 0.1, 2).astype(np.float32)
    lab = rng.integers(0, 2, N).astype(np.int32)
    fw, fb = U.to_dev(torch.from_numpy(w32)), U.to_dev(torch.from_numpy(b32))
    labels = U.to_dev(torch.from_numpy(lab))
    logits, loss = U.zeros_f32((N, 2)), U.zeros_f32((1,))
    dx = U.empty((N, C, V), dt)
    dfw, dfb = U.zeros_f32((2, C)), U.zeros_f32((2,))
    ws = U.workspace(R.rat3d_head_workspace_size(N, C, 2))
    R.rat3d_head_fwd_bwd(N, C, V, 2, U.code(dt), x, fw, fb, labels, logits, loss, dx, dfw, dfb, 0,
                         ws, ws.numel())
    U.sync()
    g = xr.mean(axis=2)
    lref = ops.fc_fwd(g, w32.astype(np.float64), b32.astype(np.float64))
    lossr, dl = ops.ce_fwd_bwd(lref, lab)
    dg, dwr, dbr = ops.fc_bwd(dl, g, w32.astype(np.float64))
    w64 = w32.astype(np.float64)
    U.check(U.f64(logits), lref, "f32", "logits",
            terms=np.abs(g) @ np.abs(w64).T + np.abs(b32.astype(np.float64)))
    assert abs(float(U.f64(loss)[0]) - lossr) <= 1e-4 * max(1.0, abs(lossr))
    U.check(U.f64(dfw), dwr, "f32", "dfc_w", kind="sum", terms=np.abs(dl).T @ np.abs(g))
    U.check(U.f64(dfb), dbr, "f32", "dfc_b", kind="sum", norm=False,
            terms=np.abs(dl).sum(axis=0))
    tdx = np.repeat((np.abs(dl) @ np.abs(w64))[:, :, None] / V, V, axis=2)
    U.check(U.f64(dx), rnd(np.repeat(dg[:, :, None] / V, V, axis=2)), dt, "dx", terms=tdx)


def test_sgd_update_is_one_rounding():
    from paper_2104_05035_amd import rat3d as R
    torch = U.torch_mod()
    rng = np.random.default_rng(5)
    n = 1000003
    w32 = rng.standard_normal(n).astype(np.float32)
    g32 = rng.standard_normal(n).astype(np.float32)
    w = U.to_dev(torch.from_numpy(w32.copy()))
    g = U.to_dev(torch.from_numpy(g32))
    R.rat3d_sgd(n, 1e-4, w, g)
    U.sync()
    lr = np.float64(np.float32(1e-4))
    exact = w32.astype(np.float64) - lr * g32.astype(np.float64)
    got = w.cpu().numpy()
    # within one float32 rounding of the exact update
    ulp = np.spacing(np.abs(exact).astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(got.astype(np.float64) - exact) <= ulp)
