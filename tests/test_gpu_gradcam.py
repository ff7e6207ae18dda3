"""GPU parity of 3D Grad-CAM (rat3d_gradcam, the explainable block, inference
mode) against the oracle (oracle/net.py gradcam) on seeded running
statistics loaded with rat3d_net_running_load: the reduced full network in
float32 at every target stage, in bf16 at stages 1-3, and the full network
(8 volumes 96x112x96, bf16) at stages 2 and 3.

Gates: every layer of the inference pass is replayed by the oracle on the
tensors the GPU stored for it (tests/replay.py, inference mode: BN on the
running statistics; the forward, the logits, the seed d logit_k / d top and
the backward down to the target map, element-wise at the stated tolerance),
and the map kernels are checked element-wise on the GPU's own stored A and dA
(alpha, the ReLU of the weighted sum, the trilinear resampling).  The logits
must also match the oracle's own end-to-end inference pass at the stated
tolerance; its dA and maps, whose pooling decisions are its own (a near-tie
at the 1x1x1 mask level reroutes a whole channel's gradient), are printed as
a diagnostic.  The call must leave the parameter and gradient arenas
untouched."""
import numpy as np
import pytest

from oracle import net as onet
from oracle import ops
from paper_2104_05035_amd import rat3d as R
from paper_2104_05035_amd import synth
from tests import gpu_util as U
from tests.net_util import Bound
from tests.replay import Replay, Source

pytestmark = pytest.mark.gpu


def _case(n, d, h, w, dt, seed, targets):
    torch = U.torch_mod()
    rng, rx, rl = synth.streams(seed, 3)
    B = Bound(R.NET_RESATTNET, n, 1, 32, d, h, w, dt, rng)
    # running statistics, one (mean, var) per BN channel in arena order
    bns = [nm[:-2] for nm, _, _ in B.layout if nm.endswith(".g")]
    rr = np.random.default_rng(seed + 100)
    means = {b: rr.normal(0.0, 0.3, B.params[b + ".g"].shape).astype(np.float32) for b in bns}
    varis = {b: rr.uniform(0.5, 2.0, B.params[b + ".g"].shape).astype(np.float32) for b in bns}
    run = np.concatenate([means[b] for b in bns] + [varis[b] for b in bns])
    assert run.size == 2 * B.net.running_count
    B.net.rat3d_net_running_load(U.to_dev(torch.from_numpy(run)))
    running = {b: (means[b].astype(np.float64), varis[b].astype(np.float64)) for b in bns}
    vol = synth.mri_volumes(rx, n, (d, h, w))
    x, xr = U.dev_input(vol, dt)
    classes = rl.integers(0, 2, n).astype(np.int32)
    cls = U.to_dev(torch.from_numpy(classes))
    P0 = B.P.clone()
    for target in targets:
        C, Dt, Ht, Wt = B.net.rat3d_gradcam_shape(target)
        name = "stem.p" if target == 0 else "s%d.am.out" % target
        cam, up = U.zeros_f32((n, Dt, Ht, Wt)), U.zeros_f32((n, d, h, w))
        logits = U.zeros_f32((n, 2))
        print("gradcam %dx%dx%dx%d %s target %d" % (n, d, h, w, dt, target), flush=True)
        B.net.rat3d_gradcam(x, cls, target, logits, cam, up)
        U.sync()
        assert torch.equal(B.P, P0) and not torch.any(B.G != 0), "Grad-CAM changed the arenas"
        rep = Replay(B.params, dt, eval_stats=running, verbose=False)
        rep.gradcam(Source(B, {"x": xr, "logits": U.f64(logits)}), classes, target)
        print("   replay: %d checks, %d of %d stored elements differ by more than one ulp" % (
            rep.checks, rep.above_1ulp, rep.elements), flush=True)
        out = onet.gradcam(B.params, xr, classes, running, target, dt == "bf16")
        r = U.rel(U.f64(logits), out["logits"])
        print("   end to end logits rel %.3e" % r, flush=True)
        assert r <= U.TOL[dt], "logits: relative error %.3e" % r
        for what, got, ref in (("dA", B.tensor("d:" + name), out["dA"]),
                               ("cam", U.f64(cam), out["cam"]), ("cam_up", U.f64(up), out["up"])):
            print("   end to end %-8s rel %.3e (diagnostic)" % (what, U.rel(got, ref)), flush=True)
        # the map kernels on the GPU's own A and dA
        A, dA = B.tensor(name), B.tensor("d:" + name)
        alpha = dA.mean(axis=(2, 3, 4))
        ta = np.abs(dA).mean(axis=(2, 3, 4))
        camr = np.maximum((alpha[:, :, None, None, None] * A).sum(axis=1), 0.0)
        terms = ((np.abs(alpha) + ta)[:, :, None, None, None] * np.abs(A)).sum(axis=1)
        U.check(U.f64(cam), camr, "f32", "cam (GPU A, dA)", terms=terms)
        upr = ops.trilinear_fwd(U.f64(cam)[:, None], (d, h, w))[:, 0]
        U.check(U.f64(up), upr, "f32", "cam_up (GPU cam)",
                terms=ops.trilinear_fwd(np.abs(U.f64(cam))[:, None], (d, h, w))[:, 0])
        assert U.f64(cam).max() > 0.0


def test_gradcam_reduced_f32():
    _case(2, 48, 56, 48, "f32", 51, (0, 1, 2, 3))


def test_gradcam_reduced_bf16():
    _case(2, 48, 56, 48, "bf16", 52, (1, 2, 3))


@pytest.mark.timeout(900)
def test_gradcam_workload():
    """The full network's explainable block on 8 MRI-shaped volumes
    96x112x96 (bf16), maps at stages 2 and 3."""
    _case(8, 96, 112, 96, "bf16", 53, (2, 3))
