"""Drivers shared by the composite GPU tests: seeded parameters for a
library network, binding, one call, read-back of the gradient arena and
workspace tensors, the exact SGD check and the end-to-end diagnostics."""
import numpy as np

from oracle import net as onet
from oracle import ops
from paper_2104_05035_amd import rat3d as R
from paper_2104_05035_amd import synth
from tests import gpu_util as U
from tests.replay import Replay, Source


class Bound:
    """A rat3d network with seeded parameters and bound device buffers."""

    def __init__(self, kind, n, c_in, c, d, h, w, dt, rng, micro_batches=1, perturb_bn=0.0,
                 bias_std=0.0, lr=1e-4):
        torch = U.torch_mod()
        self.dt = dt
        self.net = R.Net(kind, n, c_in, c, d, h, w, U.code(dt), micro_batches=micro_batches,
                         lr=lr)
        self.layout = self.net.params()
        self.params = synth.init_params(rng, [(nm, shp) for nm, _, shp in self.layout],
                                        bias_std=bias_std, perturb_bn=perturb_bn)
        arena = np.concatenate([self.params[nm].astype(np.float32).ravel()
                                for nm, _, _ in self.layout])
        self.arena0 = torch.from_numpy(arena)
        self.P = U.to_dev(self.arena0)
        self.G = U.zeros_f32(arena.shape)
        self.ws = U.workspace(self.net.workspace_size)
        self.net.rat3d_net_bind(self.P, self.G, self.ws, self.ws.numel())
        # the oracle sees the float32 parameter values the GPU holds
        self.params = {nm: self.params[nm].astype(np.float32).astype(np.float64)
                       for nm, _, _ in self.layout}
        self.tinfo = self.net.tensors()

    def arena(self, t):
        a = t.detach().cpu().numpy().astype(np.float64)
        return {nm: a[off:off + int(np.prod(shp))].reshape(shp) for nm, off, shp in self.layout}

    def grads(self):
        return self.arena(self.G)

    def new_params(self):
        return self.arena(self.P)

    def reset_params(self):
        """Parameter arena back to its seeded values, gradient arena zero."""
        self.P.copy_(self.arena0.to(self.P.device))
        self.G.zero_()

    def tensor(self, name):
        torch = U.torch_mod()
        off, dt, shp = self.tinfo[name]
        if dt == R.U8:
            nb = int(np.prod(shp))
            return self.ws[off:off + nb].cpu().numpy().reshape(shp)
        es = 2 if dt == R.BF16 else 4
        nb = int(np.prod(shp)) * es
        raw = self.ws[off:off + nb]
        t = raw.view(torch.bfloat16 if dt == R.BF16 else torch.float32).reshape(shp)
        return t.to(torch.float64).cpu().numpy()


def check_sgd(old, new, G, lr):
    """new == fl32(old - lr*G) within one float32 rounding (GPU's own G)."""
    lr64 = np.float64(np.float32(lr))
    for k in old:
        exact = old[k] - lr64 * G[k]
        ulp = np.spacing(np.abs(exact).astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(new[k] - exact) <= ulp), k


def end_to_end(G, Gref, what="gradients"):
    """Diagnostic only (not a gate): norm-wise distance of the GPU's
    gradients from the oracle's own end-to-end run, whose ReLU and pooling
    decisions are its own.  The layer-by-layer replay is the gate."""
    rows = sorted(((U.rel(G[k], Gref[k]), k) for k in Gref), reverse=True)
    keys = list(Gref)
    cat = lambda D: np.concatenate([np.ravel(D[k]) for k in keys])
    print("end-to-end %s (diagnostic): whole vector rel %.3e; largest:" % (
        what, U.rel(cat(G), cat(Gref))))
    for err, k in rows[:5]:
        print("   %-26s %.3e" % (k, err))


def partition_replayed(n, mb, d, h, w, c, seed, verbose=True):
    """First-stage partition, micro-batch by micro-batch through the C ABI
    (rat3d_partition_micro_batch, then rat3d_net_update); every micro-batch
    is replayed layer by layer on a snapshot of its stored tensors and the
    accumulated gradient arena is compared with the summed oracle gradients.
    Then rat3d_train_step on the same inputs must give bit-identical
    gradients and parameters (it runs the same calls)."""
    torch = U.torch_mod()
    rng, rx, rdy = synth.streams(seed, 3)
    B = Bound(R.NET_PARTITION1, n, 1, c, d, h, w, "bf16", rng, micro_batches=mb)
    vol = synth.mri_volumes(rx, n * mb, (d, h, w))
    x, xr = U.dev_input(vol, "bf16")
    so = [ops.out_size(v, 7, 2, 3) for v in (d, h, w)]
    dy, dyr = U.dev_input(rdy.standard_normal((n * mb, c) + tuple(so)), "bf16")
    old = {k: v.copy() for k, v in B.params.items()}
    rep = Replay(B.params, "bf16", verbose=verbose)
    for m in range(mb):
        sl = slice(m * n, (m + 1) * n)
        print("partition micro-batch %d of %d (%d volumes %dx%dx%d)" % (m + 1, mb, n, d, h, w),
              flush=True)
        B.net.rat3d_partition_micro_batch(x[sl], dy[sl], m > 0)
        U.sync()
        rep.partition1(Source(B, {"x": xr[sl], "d:am.out": dyr[sl]}, snapshot=True))
    out_last = B.tensor("am.out")
    G = B.grads()
    rep.finish(G)
    B.net.rat3d_net_update()
    U.sync()
    new = B.new_params()
    check_sgd(old, new, G, 1e-4)
    # the same step through rat3d_train_step: bit-identical results, with
    # micro-batches overlapped (the default) and with every kernel on one
    # stream; the last micro-batch's tensors are where rat3d_net_tensor_info
    # says they are
    G1, P1 = B.G.clone(), B.P.clone()
    for overlap in (1, 0):
        B.net.rat3d_net_set_overlap(overlap)
        B.reset_params()
        B.net.rat3d_train_step(x, None, dy, None)
        U.sync()
        assert torch.equal(B.G, G1) and torch.equal(B.P, P1), \
            "rat3d_train_step (overlap %d) differs from its micro-batch calls" % overlap
        assert np.array_equal(B.tensor("am.out"), out_last), \
            "rat3d_train_step (overlap %d): last micro-batch output not in place" % overlap
    B.net.rat3d_net_set_overlap(1)
    _, Gref, info = onet.train_step("partition1", old, 1e-4, True, x=xr, dy=dyr,
                                    micro_batches=mb)
    r = U.rel(out_last, info["y"][-1])
    print("end-to-end partition output (last micro-batch) rel %.3e" % r)
    assert r <= U.TOL["bf16"], "partition output: relative error %.3e" % r
    end_to_end(G, Gref)
    return B
