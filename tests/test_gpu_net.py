"""GPU parity of the composite blocks and training steps against the oracle:
the single conv layer, the residual unit, the attention module and the full
network at their full workload sizes, the first-stage partition at a reduced
volume (its full size is covered by tests/test_gpu_full.py), plus reduced and
ragged blocks.

Gates.  Every layer of every step is checked by the decision-matched replay
(tests/replay.py): the oracle applies the layer to the tensors the GPU stored
for it and each output -- activations, activation gradients, BN statistics,
and, summed over the step, every parameter gradient -- must match at the
stated tolerance (1e-4 float32, 2e-2 bfloat16, norm-wise) and within the
element-wise bound of tests/gpu_util.check.  The block and partition outputs
are also compared end to end with the oracle's own forward pass at the stated
tolerance (norm-wise: the oracle's pooling and ReLU decisions are its own).
The end-to-end gradients are printed as a diagnostic only.  The SGD update
is checked exactly (one float32 rounding of w - lr g)."""
import numpy as np
import pytest

from oracle import net as onet
from oracle import ops
from paper_2104_05035_amd import rat3d as R
from paper_2104_05035_amd import synth
from tests import gpu_util as U
from tests.net_util import Bound, check_sgd, end_to_end, partition_replayed
from tests.replay import Replay, Source

pytestmark = pytest.mark.gpu


def test_conv_layer_workload():
    """Single conv3d layer fwd + dgrad + wgrad, float32: N=1, 4 -> 8 channels,
    16^3, 3^3 kernel, stride 1, pad 1, bias; x U(-1,1), w and b N(0,0.1),
    upstream gradient N(0,1)."""
    cfg = synth.WORKLOADS[0]
    rx, rw, rb, rdy = synth.streams(0, 4)
    x, xr = U.dev_input(rx.uniform(-1, 1, (1, 4, 16, 16, 16)), "f32")
    w, wr = U.dev_input(rw.normal(0, 0.1, (8, 4, 3, 3, 3)), "f32")
    b, br = U.dev_input(rb.normal(0, 0.1, 8), "f32")
    dy, dyr = U.dev_input(rdy.standard_normal((1, 8, 16, 16, 16)), "f32")
    desc = R.conv_desc(1, 4, 8, 16, 16, 16, 3, 1, 1, True, R.F32)
    ws = U.workspace(max(R.rat3d_conv3d_workspace_size(desc, i) for i in range(3)))
    y, dx = U.empty((1, 8, 16, 16, 16), "f32"), U.empty((1, 4, 16, 16, 16), "f32")
    dw, db = U.zeros_f32((8, 4, 3, 3, 3)), U.zeros_f32((8,))
    R.rat3d_conv3d_fwd(desc, x, w, b, y, ws, ws.numel())
    R.rat3d_conv3d_dgrad(desc, dy, w, dx, 0, ws, ws.numel())
    R.rat3d_conv3d_wgrad(desc, x, dy, dw, db, 0, ws, ws.numel())
    U.sync()
    assert cfg["k"] == 3 and cfg["bias"]
    ax, aw, ady = np.abs(xr), np.abs(wr), np.abs(dyr)
    U.check(U.f64(y), ops.conv3d_fwd(xr, wr, br, 1, 1), "f32", "y",
            terms=ops.conv3d_fwd(ax, aw, np.abs(br), 1, 1))
    U.check(U.f64(dx), ops.conv3d_dgrad(dyr, wr, xr.shape, 1, 1), "f32", "dx",
            terms=ops.conv3d_dgrad(ady, aw, xr.shape, 1, 1))
    dwr, dbr = ops.conv3d_wgrad(xr, dyr, 3, 1, 1, True)
    tw, tb = ops.conv3d_wgrad(ax, ady, 3, 1, 1, True)
    U.check(U.f64(dw), dwr, "f32", "dw", kind="sum", terms=tw)
    U.check(U.f64(db), dbr, "f32", "db", kind="sum", terms=tb)


def _block(kind, code, n, c, d, h, w, dt, seed, perturb_bn=0.0):
    rng, rx, rdy = synth.streams(seed, 3)
    B = Bound(code, n, c, c, d, h, w, dt, rng, perturb_bn=perturb_bn, bias_std=0.1)
    x, xr = U.dev_input(rx.standard_normal((n, c, d, h, w)), dt)
    dy, dyr = U.dev_input(rdy.standard_normal((n, c, d, h, w)), dt)
    y, dx = U.empty((n, c, d, h, w), dt), U.empty((n, c, d, h, w), dt)
    print("%s %dx%dx%dx%dx%d %s: block step on the GPU" % (kind, n, c, d, h, w, dt), flush=True)
    B.net.rat3d_block_fwd_bwd(x, dy, y, dx)
    U.sync()
    yo = "y" if kind == "resunit" else "out"
    S = Source(B, {"x": xr, yo: U.f64(y), "d:" + yo: dyr, "d:x": U.f64(dx)})
    rep = Replay(B.params, dt)
    getattr(rep, kind)(S)
    rep.finish(B.grads())
    # end to end: the block output within the stated tolerance of the
    # oracle's own forward pass; gradients as a diagnostic
    bf = dt == "bf16"
    yref, dxref, Gref, _ = onet.block_fwd_bwd(kind, B.params, xr, dyr, bf16=bf)
    r = U.rel(U.f64(y), yref)
    print("end-to-end output rel %.3e, input gradient rel %.3e (diagnostic)" % (
        r, U.rel(U.f64(dx), dxref)))
    assert r <= U.TOL[dt], "block output: relative error %.3e" % r
    end_to_end(B.grads(), Gref)
    # the same call with every kernel on one stream: bit-identical outputs
    # and gradients (an attention module's mask branch otherwise runs on a
    # stream of its own)
    torch = U.torch_mod()
    y1, dx1, G1 = y.clone(), dx.clone(), B.G.clone()
    B.net.rat3d_net_set_overlap(0)
    B.net.rat3d_block_fwd_bwd(x, dy, y, dx)
    U.sync()
    B.net.rat3d_net_set_overlap(1)
    assert torch.equal(y, y1) and torch.equal(dx, dx1) and torch.equal(B.G, G1), \
        "serial block call differs from the concurrent one"


def test_resunit_workload():
    """Residual unit fwd+bwd, float32: N=2, C=32, 32^3, He weights, BN
    (batch statistics, eps 1e-5), identity skip."""
    _block("resunit", R.NET_RESUNIT, 2, 32, 32, 32, 32, "f32", 1)


def test_resunit_ragged_perturbed_bn():
    _block("resunit", R.NET_RESUNIT, 3, 16, 7, 9, 5, "f32", 11, perturb_bn=0.2)


def test_attn_reduced_bf16():
    _block("attn", R.NET_ATTN, 2, 16, 24, 24, 24, "bf16", 12, perturb_bn=0.1)


def test_attn_ragged_f32():
    _block("attn", R.NET_ATTN, 2, 8, 12, 14, 12, "f32", 13, perturb_bn=0.1)


@pytest.mark.timeout(900)
def test_attn_workload():
    """Attention module fwd+bwd, bf16 storage / fp32 accumulation: N=4, C=64,
    48^3 (trunk 2 RUs; mask pool-RU-pool-2RU-up-RU-up-1^3-1^3-sigmoid)."""
    _block("attn", R.NET_ATTN, 4, 64, 48, 48, 48, "bf16", 2)


def _resattnet(n, d, h, w, seed, dt="bf16"):
    rng, rx, rl = synth.streams(seed, 3)
    B = Bound(R.NET_RESATTNET, n, 1, 32, d, h, w, dt, rng)
    vol = synth.mri_volumes(rx, n, (d, h, w))
    x, xr = U.dev_input(vol, dt)
    lab = rl.integers(0, 2, n).astype(np.int32)
    torch = U.torch_mod()
    labels = U.to_dev(torch.from_numpy(lab))
    loss = U.zeros_f32((1,))
    old = {k: v.copy() for k, v in B.params.items()}
    print("resattnet %dx%dx%dx%d %s: train step on the GPU" % (n, d, h, w, dt), flush=True)
    B.net.rat3d_train_step(x, labels, None, loss)
    U.sync()
    G = B.grads()
    rep = Replay(B.params, dt)
    rep.resattnet(Source(B, {"x": xr}), lab)
    rep.finish(G)
    assert float(U.f64(loss)[0]) == float(B.tensor("loss").ravel()[0])
    check_sgd(old, B.new_params(), G, 1e-4)
    bf = dt == "bf16"
    _, Gref, info = onet.train_step("resattnet", B.params, 1e-4, bf, x=xr, labels=lab)
    print("end-to-end logits rel %.3e, loss %.6f vs %.6f (diagnostic)" % (
        U.rel(B.tensor("logits").reshape(n, 2), info["logits"]), float(U.f64(loss)[0]),
        info["loss"]))
    end_to_end(G, Gref)
    # the same step with every kernel on one stream (no mask-branch stream):
    # bit-identical gradients and parameters
    G1, P1 = B.G.clone(), B.P.clone()
    B.net.rat3d_net_set_overlap(0)
    B.reset_params()
    B.net.rat3d_train_step(x, labels, None, loss)
    U.sync()
    B.net.rat3d_net_set_overlap(1)
    assert torch.equal(B.G, G1) and torch.equal(B.P, P1), \
        "serial full-network step differs from the one with mask-branch streams"


def test_resattnet_reduced_f32():
    """Full network step on 2 volumes of 48x56x48 in float32 (same graph,
    smaller maps; the third stage's mask branch reaches 1x1x1)."""
    _resattnet(2, 48, 56, 48, 23, "f32")


def test_resattnet_reduced_bf16():
    """The same reduced network in bf16: its deepest mask level normalises
    over 2 values, where decisions are most fragile."""
    _resattnet(2, 48, 56, 48, 25, "bf16")


@pytest.mark.timeout(900)
def test_resattnet_workload():
    """Full network train step: 8 MRI-shaped volumes 96x112x96, bf16 storage,
    stem 7^3 s2 -> 32 ch, maxpool, stages 64/128/256 (RU + attention), GAP,
    FC to 2 classes, cross-entropy with random labels, SGD."""
    _resattnet(8, 96, 112, 96, 3)


def test_partition1_reduced():
    """First-stage partition, 2 micro-batches of 2 volumes of 48x56x48."""
    partition_replayed(2, 2, 48, 56, 48, 64, 24)


def test_partition1_reduced_bias_sums():
    """A partition whose 24x32x32 attention maps are a multiple of 2048
    voxels, so the soft-mask backward also sums dz for the c2 bias gradient
    (the path the measured workload takes), accumulated over 3 micro-batches."""
    partition_replayed(1, 3, 48, 64, 64, 32, 26)
