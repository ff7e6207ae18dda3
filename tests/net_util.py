"""Drivers shared by the composite GPU tests: seeded parameters for a
library network, binding, one call, and read-back of the gradient arena and
workspace tensors."""
import numpy as np

from paper_2104_05035_amd import rat3d as R
from paper_2104_05035_amd import synth
from tests import gpu_util as U


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
        self.P = U.to_dev(torch.from_numpy(arena))
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


def compare_grads(G, Gref, dt, skip=()):
    worst = 0.0
    for k, ref in Gref.items():
        if k in skip:
            continue
        r = U.check(G[k], ref, dt, "grad " + k)
        worst = max(worst, r)
    return worst


def check_sgd(old, new, G, lr):
    """new == fl32(old - lr*G) within one float32 rounding (GPU's own G)."""
    lr64 = np.float64(np.float32(lr))
    for k in old:
        exact = old[k] - lr64 * G[k]
        ulp = np.spacing(np.abs(exact).astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(new[k] - exact) <= ulp), k


JITTER = 1e-6  # relative noise of float32 arithmetic at a store point


def floors(ref, jittered):
    """Per-key spread of the oracle under rounding-level jitter (max over runs)."""
    return {k: max(U.rel(j[k], ref[k]) for j in jittered) for k in ref}


def gate(got, ref, floor, dt, what):
    """Error must be within max(stated tolerance, 2 x the oracle's own spread)."""
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), what
    err = U.rel(got, ref)
    lim = max(U.TOL[dt], 2.0 * floor)
    assert err <= lim, "%s: relative error %.3e > %.3e (oracle spread %.3e)" % (
        what, err, lim, floor)
    return err, lim


def gate_grads(G, Gref, Gjit, dt):
    """Gate every parameter gradient and the whole gradient vector; returns
    the number of tensors within the stated tolerance outright."""
    fl = floors(Gref, Gjit)
    within = 0
    rows = sorted(((U.rel(G[k], Gref[k]), fl[k], k) for k in Gref), reverse=True)
    print("gradients: %d tensors; worst (error, oracle spread):" % len(rows))
    for err, f, k in rows[:6]:
        print("   %-24s %.3e  %.3e" % (k, err, f))
    for k in Gref:
        err, _ = gate(G[k], Gref[k], fl[k], dt, "grad " + k)
        within += err <= U.TOL[dt]
    keys = list(Gref)
    cat = lambda D: np.concatenate([np.ravel(D[k]) for k in keys])
    gfl = max(U.rel(cat(j), cat(Gref)) for j in Gjit)
    gate(cat(G), cat(Gref), gfl, dt, "gradient vector")
    return within
