"""Layer-by-layer parity of a library network's step against the oracle
(decision-matched replay).

The training step is only piecewise smooth: ReLU masks, first-maximum pooling
and BN over the few voxels of the deep mask levels turn rounding-level
differences into different decisions downstream, in any implementation whose
summation order differs from the oracle's.  An end-to-end comparison of the
gradients therefore measures the conditioning of the step more than the
kernels.  Here every layer is checked on its own, at the stated tolerance and
element by element (tests/gpu_util.check): the oracle applies the layer to
the inputs the GPU stored for it -- its activations, its incoming gradient,
the stored layer outputs whose sign is the ReLU mask, the pooling argmax maps
-- and the GPU's outputs of that layer must match.  The decisions (which
voxel passes a ReLU, which tap wins a pooling window) are thus the GPU's, and
each one is itself checked where it is made: pooling values and argmax
bit-exact on the GPU's pooling input, BN+ReLU outputs on the GPU's BN input.
BN statistics are recomputed by the oracle from the GPU's stored BN inputs and
compared with the GPU's saved statistics (float32); the BN outputs and
gradients are then compared with the oracle's BN evaluated with the statistics
the GPU applied.

Where the GPU overwrites an intermediate (an input gradient formed in two
stores: the skip or mask-branch part first, the conv part added onto it) the
oracle forms the intermediate from the GPU's stored inputs and carries its
element-wise bound into the final check (`extra`).

Parameter gradients of every layer are summed over the replays of a step's
micro-batches (each replay sees that micro-batch's stored tensors) and
compared with the GPU's gradient arena at the end (`finish`).

Graph and names follow the network plan of the library (rat3d_net_tensor_info
names; the readings are those of oracle/net.py): residual unit conv1 -> bn1
(ReLU) -> conv2 -> bn2 (+ skip, ReLU), projection skip = 1^3 conv + BN;
attention module trunk t1, t2, mask pool -> m1 -> pool -> m2 -> m3 -> up ->
m4 -> 1^3 conv c1 -> up -> BN + ReLU -> 1^3 conv c2 (+bias) -> sigmoid fuse.
The library runs the mask tail's bias-free c1 on the coarse map before the
last upsampling (the two linear maps commute); the replay checks the layers in
the library's order (conv on the coarse map, then the upsampling), and the
end-to-end comparisons of the block outputs cover the literal order.
"""
import numpy as np

from oracle import ops
from paper_2104_05035_amd import rat3d as R
from tests import gpu_util as U

AX = (0, 2, 3, 4)


def _bc(v):
    return v[None, :, None, None, None]


class Source:
    """Float64 views of a network's stored tensors: from the bound workspace
    (device) or a host snapshot of it, with external tensors (the caller's x,
    y, dx, dy) by name."""

    def __init__(self, B, ext=None, snapshot=False):
        self.tinfo = B.tinfo
        self.ws = B.ws.cpu() if snapshot else B.ws
        self.ext = dict(ext or {})

    def __contains__(self, name):
        return name in self.ext or name in self.tinfo

    def __call__(self, name):
        if name in self.ext:
            return np.asarray(self.ext[name], dtype=np.float64)
        torch = U.torch_mod()
        off, dt, shp = self.tinfo[name]
        if dt == R.U8:
            n = int(np.prod(shp))
            return self.ws[off:off + n].cpu().numpy().reshape(shp).astype(np.int32)
        es = 2 if dt == R.BF16 else 4
        raw = self.ws[off:off + int(np.prod(shp)) * es]
        t = raw.view(torch.bfloat16 if dt == R.BF16 else torch.float32).reshape(shp)
        return t.to(torch.float64).cpu().numpy()


class Replay:
    """Checks every layer of a step; accumulates the oracle's parameter
    gradients (and their sum|terms|) over micro-batches."""

    def __init__(self, params, dt, eps=1e-5, verbose=True, eval_stats=None):
        self.P = params
        # inference mode (Grad-CAM): BN on the running statistics
        # {name: (mean, var)}; no parameter gradients
        self.eval_stats = eval_stats
        self.dt = dt
        self.rnd = ops.round_bf16 if dt == "bf16" else ops.identity
        self.eps = eps
        self.G = {}
        self.T = {}   # name -> list of sum|terms| arrays or callables
        self.verbose = verbose
        self.checks = 0
        self.above_1ulp = 0
        self.elements = 0
        self.S = None

    # ------------------------------------------------------------ helpers
    def w(self, name):
        """Conv weight as the convolution sees it (bf16 working copy)."""
        return self.rnd(self.P[name])

    def chk(self, what, got, ref, dt=None, **kw):
        dt = dt or self.dt
        r = U.check(got, ref, dt, what, **kw)
        st = U.LAST
        self.checks += 1
        self.above_1ulp += st["above_1ulp"]
        self.elements += st["size"]
        if self.verbose:
            print("   %-30s rel %.2e  >1ulp %6d/%-9d terms@%d" % (
                what, r, st["above_1ulp"], st["size"], st["terms_evaluated"]), flush=True)
        return r

    def bound(self, ref, terms):
        """Element-wise bound of a stored value the GPU may round differently."""
        return 2.0 * U.ulp(ref, self.dt) + U.C_OUT * terms

    def add_grad(self, name, ref, terms):
        if name in self.G:
            self.G[name] = self.G[name] + ref
        else:
            self.G[name] = np.array(ref, dtype=np.float64)
        self.T.setdefault(name, []).append(terms)

    # ------------------------------------------------------------ layers
    def conv_fwd(self, oname, x, wname, bname, s, p):
        w = self.w(wname)
        b = self.P[bname] if bname else None
        ref = self.rnd(ops.conv3d_fwd(x, w, b, s, p))
        ax, aw = np.abs(x), np.abs(w)
        ab = None if b is None else np.abs(b)
        self.chk(oname, self.S(oname), ref,
                 terms=lambda idx: ops.conv3d_fwd_points(ax, aw, ab, s, p, idx))
        return self.S(oname)

    def conv_dgrad(self, dname, dy, wname, in_shape, s, p, base=None, base_extra=None):
        w = self.w(wname)
        raw = ops.conv3d_dgrad(dy, w, in_shape, s, p)
        ref = self.rnd(raw if base is None else base + raw)
        ady, aw = np.abs(dy), np.abs(w)

        def terms(idx):
            t = ops.conv3d_dgrad_points(ady, aw, in_shape, s, p, idx)
            if base is not None:
                t = t + np.abs(base[tuple(idx.T)])
            return t
        self.chk(dname, self.S(dname), ref, terms=terms, extra=base_extra)
        return self.S(dname)

    def conv_wgrad(self, wname, x, dy, k, s, p, bname=None):
        if self.eval_stats is not None:
            return
        dw, db = ops.conv3d_wgrad(x, dy, k, s, p, bname is not None)
        ax, ady = np.abs(x), np.abs(dy)
        self.add_grad(wname, dw, lambda idx: ops.conv3d_wgrad_points(ax, ady, k, s, p, idx))
        if bname:
            self.add_grad(bname, db, ady.sum(axis=AX))

    def bn_stats(self, name, h):
        """Checks the GPU's saved batch statistics against the oracle's, from
        the GPU's stored BN input, and returns the GPU's: the layer's outputs
        are then compared with the oracle's BN evaluated with the statistics
        the GPU applied."""
        mean, var = ops.bn_stats(h)
        invstd = 1.0 / np.sqrt(var + self.eps)
        gm, gi = self.S(name + ".mean").ravel(), self.S(name + ".invstd").ravel()
        self.chk(name + ".mean", gm, mean, dt="f32", kind="sum", norm=False,
                 terms=np.abs(h).mean(axis=AX))
        # float32 statistics: the variance's rounding error is at most that of
        # the unshifted moments, relative E[h^2] / (var + eps)
        self.chk(name + ".invstd", gi, invstd, dt="f32",
                 terms=invstd * (h * h).mean(axis=AX) / (var + self.eps))
        return gm, gi

    def bn_value(self, name, h, st, relu, residual=None):
        """BN (+ residual) (+ ReLU) of h with statistics st (inference mode:
        the running statistics); (unrounded value, sum|terms| of the float32
        evaluation x * scale + shift [+ r])."""
        g, b = self.P[name + ".g"], self.P[name + ".b"]
        if self.eval_stats is not None:
            rm, rv = self.eval_stats[name]
            mean, invstd = rm, 1.0 / np.sqrt(rv + self.eps)
        else:
            mean, invstd = st
        sc = g * invstd
        y = _bc(sc) * (h - _bc(mean)) + _bc(b)
        terms = np.abs(h) * _bc(np.abs(sc)) + _bc(np.abs(b) + np.abs(mean * sc))
        if residual is not None:
            y = y + residual
            terms = terms + np.abs(residual)
        if relu:
            y = np.maximum(y, 0.0)
        return y, terms

    def bn_fwd(self, name, h, yname, relu, residual=None, res_extra=None):
        st = self.bn_stats(name, h) if self.eval_stats is None else None
        y, terms = self.bn_value(name, h, st, relu, residual)
        self.chk(yname, self.S(yname), self.rnd(y), terms=terms, extra=res_extra)
        return st

    def bn_bwd(self, name, dy, h, y, relu, st, dxname=None):
        """Backward of a BN (+ReLU); the ReLU mask is y > 0 of the GPU's
        stored output.  Returns (rounded dx, gradient of the residual input,
        sum|terms| of dx)."""
        gam = self.P[name + ".g"]
        if self.eval_stats is not None:
            # inference mode: dx = g * gamma / sqrt(running var + eps)
            dx, gres = ops.bn_eval_bwd(dy, y, gam, self.eval_stats[name][1], self.eps, relu)
            terms = np.abs(dx)
            ref = self.rnd(dx)
            if dxname is not None:
                self.chk(dxname, self.S(dxname), ref, terms=terms)
            return ref, gres, terms
        mean, invstd = st
        dx, gres, dgam, dbet = ops.bn_bwd(dy, h, y, gam, mean, invstd, relu)
        M = h.shape[0] * h.shape[2] * h.shape[3] * h.shape[4]
        xh = (h - _bc(mean)) * _bc(invstd)
        ag = np.abs(gres)
        Sg = ag.sum(axis=AX)
        Sgx = np.abs(gres * xh).sum(axis=AX)
        terms = _bc(np.abs(gam * invstd)) * (
            ag + _bc(Sg / M) + (np.abs(h) + _bc(np.abs(mean))) * _bc(invstd * Sgx / M))
        ref = self.rnd(dx)
        if dxname is not None:
            self.chk(dxname, self.S(dxname), ref, terms=terms)
        self.add_grad(name + ".g", dgam, Sgx)
        self.add_grad(name + ".b", dbet, Sg)
        return ref, gres, terms

    def pool_fwd(self, x, yname):
        yref, amref = ops.maxpool3d_fwd(x)
        got, am = self.S(yname), self.S(yname + ".argmax")
        assert np.array_equal(got, yref), yname + ": pooled values differ"
        assert np.array_equal(am, amref), yname + ": argmax differs"
        self.checks += 2
        if self.verbose:
            print("   %-30s bit-exact (values and argmax, %d)" % (yname, got.size), flush=True)
        return got, am

    def pool_bwd_value(self, dy, am, in_shape):
        """rnd(pool gradient) and its element-wise bound (GPU sums in float32)."""
        raw = ops.maxpool3d_bwd(dy, am, in_shape)
        ref = self.rnd(raw)
        return ref, ops.maxpool3d_bwd(np.abs(dy), am, in_shape)

    # ------------------------------------------------------------ blocks
    def ru_fwd(self, pre, xname, stride):
        x = self.S(xname)
        proj = (pre + "proj.w") in self.P
        c = dict(x=x, xname=xname, stride=stride, proj=proj)
        c["h1"] = self.conv_fwd(pre + "h1", x, pre + "conv1.w", None, stride, 1)
        c["st1"] = self.bn_fwd(pre + "bn1", c["h1"], pre + "a1", relu=True)
        c["a1"] = self.S(pre + "a1")
        c["h2"] = self.conv_fwd(pre + "h2", c["a1"], pre + "conv2.w", None, 1, 1)
        extra = None
        if proj and self.eval_stats is not None:
            # inference mode: the projection BN's output is stored
            c["hp"] = self.conv_fwd(pre + "hp", x, pre + "proj.w", None, stride, 0)
            c["stp"] = None
            spv, spt = self.bn_value(pre + "projbn", c["hp"], None, relu=False)
            self.chk(pre + "sp", self.S(pre + "sp"), self.rnd(spv), terms=spt)
            skip = self.S(pre + "sp")
        elif proj:
            c["hp"] = self.conv_fwd(pre + "hp", x, pre + "proj.w", None, stride, 0)
            c["stp"] = self.bn_stats(pre + "projbn", c["hp"])
            spv, spt = self.bn_value(pre + "projbn", c["hp"], c["stp"], relu=False)
            skip = self.rnd(spv)
            # the GPU rounds its own BN_p(h_p) to bf16 before the add
            extra = self.bound(skip, spt)
        else:
            skip = x
        c["st2"] = self.bn_fwd(pre + "bn2", c["h2"], pre + "y", relu=True, residual=skip,
                               res_extra=extra)
        c["y"] = self.S(pre + "y")
        return c

    def ru_bwd(self, pre, c, dyname, dxname, dx_acc=None, acc_extra=None):
        """dx_acc: the partial input gradient already stored at dx (its
        oracle value and element-wise bound)."""
        x, s = c["x"], c["stride"]
        dy = self.S(dyname)
        _, gres, _ = self.bn_bwd(pre + "bn2", dy, c["h2"], c["y"], True, c["st2"],
                                 "d:" + pre + "h2")
        dh2 = self.S("d:" + pre + "h2")
        self.conv_dgrad("d:" + pre + "a1", dh2, pre + "conv2.w", c["a1"].shape, 1, 1)
        self.conv_wgrad(pre + "conv2.w", c["a1"], dh2, 3, 1, 1)
        da1 = self.S("d:" + pre + "a1")
        self.bn_bwd(pre + "bn1", da1, c["h1"], c["a1"], True, c["st1"], "d:" + pre + "h1")
        dh1 = self.S("d:" + pre + "h1")
        if c["proj"]:
            self.chk("d:" + pre + "skip", self.S("d:" + pre + "skip"), self.rnd(gres),
                     terms=np.abs(gres))
            dsk = self.S("d:" + pre + "skip")
            self.bn_bwd(pre + "projbn", dsk, c["hp"], None, False, c["stp"], "d:" + pre + "hp")
            dhp = self.S("d:" + pre + "hp")
            wp = self.w(pre + "proj.w")
            dxs = ops.conv3d_dgrad(dhp, wp, x.shape, s, 0)
            self.conv_wgrad(pre + "proj.w", x, dhp, 1, s, 0)
            tdxs = ops.conv3d_dgrad(np.abs(dhp), np.abs(wp), x.shape, s, 0)
            first_raw = dxs if dx_acc is None else dx_acc + dxs
            terms = tdxs if dx_acc is None else tdxs + np.abs(dx_acc)
            first = self.rnd(first_raw)
            extra = self.bound(first, terms) + (0.0 if acc_extra is None else acc_extra)
        elif dx_acc is not None:
            first = self.rnd(dx_acc + gres)
            extra = self.bound(first, np.abs(dx_acc) + np.abs(gres)) + \
                (0.0 if acc_extra is None else acc_extra)
        else:
            first, extra = gres, None  # the skip gradient is stored exactly
        self.conv_dgrad(dxname, dh1, pre + "conv1.w", x.shape, s, 1, base=first,
                        base_extra=extra)
        self.conv_wgrad(pre + "conv1.w", x, dh1, 3, s, 1)

    def am_fwd(self, pre, xname, outname):
        x = self.S(xname)
        c = dict(x=x)
        c["t1"] = self.ru_fwd(pre + "t1.", xname, 1)
        c["t2"] = self.ru_fwd(pre + "t2.", pre + "t1.y", 1)
        T = c["t2"]["y"]
        c["p1"], c["am1"] = self.pool_fwd(x, pre + "p1")
        c["m1"] = self.ru_fwd(pre + "m1.", pre + "p1", 1)
        c["p2"], c["am2"] = self.pool_fwd(c["m1"]["y"], pre + "p2")
        c["m2"] = self.ru_fwd(pre + "m2.", pre + "p2", 1)
        c["m3"] = self.ru_fwd(pre + "m3.", pre + "m2.y", 1)
        r3 = c["m3"]["y"]
        s1 = c["p1"].shape[2:]
        self.chk(pre + "u1", self.S(pre + "u1"), self.rnd(ops.trilinear_fwd(r3, s1)),
                 terms=ops.trilinear_fwd(np.abs(r3), s1))
        c["m4"] = self.ru_fwd(pre + "m4.", pre + "u1", 1)
        c["c1c"] = self.conv_fwd(pre + "c1out.coarse", c["m4"]["y"], pre + "c1.w", None, 1, 0)
        sz = x.shape[2:]
        self.chk(pre + "c1out", self.S(pre + "c1out"), self.rnd(ops.trilinear_fwd(c["c1c"], sz)),
                 terms=ops.trilinear_fwd(np.abs(c["c1c"]), sz))
        c["h1"] = self.S(pre + "c1out")
        c["stb"] = self.bn_fwd(pre + "bn", c["h1"], pre + "a", relu=True)
        c["a"] = self.S(pre + "a")
        c["z"] = self.conv_fwd(pre + "z", c["a"], pre + "c2.w", pre + "c2.bias", 1, 0)
        m = ops.sigmoid(c["z"])
        out = (1.0 + m) * T
        self.chk(outname, self.S(outname), self.rnd(out), terms=np.abs(out))
        c["T"], c["m"] = T, m
        return c

    def am_bwd(self, pre, c, doutname, dxname):
        dout = self.S(doutname)
        T = c["T"]
        # the backward uses M as the forward would store it (recomputed from z
        # and rounded to the storage type); the GPU's float32 sigmoid may round
        # to the neighbouring value: one ulp of M, carried as `extra`
        m = self.rnd(c["m"])
        um = U.ulp(m, self.dt)
        dT = (1.0 + m) * dout
        dz = dout * T * m * (1.0 - m)
        # sum|terms| of the factors 1 + M and 1 - M is 1 + |M| (1 - M cancels
        # when M is close to 1)
        self.chk("d:" + pre + "t2.y", self.S("d:" + pre + "t2.y"), self.rnd(dT),
                 terms=np.abs(dout) * (1.0 + np.abs(m)), extra=um * np.abs(dout))
        self.chk("d:" + pre + "z", self.S("d:" + pre + "z"), self.rnd(dz),
                 terms=np.abs(dout * T * m) * (1.0 + np.abs(m)),
                 extra=um * (np.abs(1.0 - 2.0 * m) + um) * np.abs(dout * T))
        dzg = self.S("d:" + pre + "z")
        self.conv_dgrad("d:" + pre + "a", dzg, pre + "c2.w", c["a"].shape, 1, 0)
        self.conv_wgrad(pre + "c2.w", c["a"], dzg, 1, 1, 0, bname=pre + "c2.bias")
        # BN + ReLU backward, then the upsampling transpose to the coarse map;
        # the GPU forms the BN input gradient inside the transpose (rounded as
        # its store would be), so the rounded value is an intermediate
        dh, _, tdh = self.bn_bwd(pre + "bn", self.S("d:" + pre + "a"), c["h1"], c["a"], True,
                                 c["stb"])
        s1 = c["c1c"].shape[2:]
        ref = self.rnd(ops.trilinear_bwd(dh, s1))
        extra = ops.trilinear_bwd(self.bound(dh, tdh), s1)
        self.chk("d:" + pre + "c1out.coarse", self.S("d:" + pre + "c1out.coarse"), ref,
                 terms=ops.trilinear_bwd(np.abs(dh), s1), extra=extra)
        dc1 = self.S("d:" + pre + "c1out.coarse")
        m4y = c["m4"]["y"]
        self.conv_dgrad("d:" + pre + "m4.y", dc1, pre + "c1.w", m4y.shape, 1, 0)
        self.conv_wgrad(pre + "c1.w", m4y, dc1, 1, 1, 0)
        self.ru_bwd(pre + "m4.", c["m4"], "d:" + pre + "m4.y", "d:" + pre + "u1")
        du1 = self.S("d:" + pre + "u1")
        s2 = c["p2"].shape[2:]
        self.chk("d:" + pre + "m3.y", self.S("d:" + pre + "m3.y"),
                 self.rnd(ops.trilinear_bwd(du1, s2)), terms=ops.trilinear_bwd(np.abs(du1), s2))
        self.ru_bwd(pre + "m3.", c["m3"], "d:" + pre + "m3.y", "d:" + pre + "m2.y")
        self.ru_bwd(pre + "m2.", c["m2"], "d:" + pre + "m2.y", "d:" + pre + "p2")
        ref, t = self.pool_bwd_value(self.S("d:" + pre + "p2"), c["am2"], c["m1"]["y"].shape)
        self.chk("d:" + pre + "m1.y", self.S("d:" + pre + "m1.y"), ref, terms=t)
        self.ru_bwd(pre + "m1.", c["m1"], "d:" + pre + "m1.y", "d:" + pre + "p1")
        # the mask branch's input gradient is stored first, then the trunk's
        # is accumulated onto it
        dxm, t = self.pool_bwd_value(self.S("d:" + pre + "p1"), c["am1"], c["x"].shape)
        self.ru_bwd(pre + "t2.", c["t2"], "d:" + pre + "t2.y", "d:" + pre + "t1.y")
        self.ru_bwd(pre + "t1.", c["t1"], "d:" + pre + "t1.y", dxname, dx_acc=dxm,
                    acc_extra=self.bound(dxm, t))

    def stem_fwd(self, pool):
        x = self.S("x")
        c = dict(x=x)
        c["h"] = self.conv_fwd("stem.h", x, "stem.w", None, 2, 3)
        c["st"] = self.bn_fwd("stem.bn", c["h"], "stem.a", relu=True)
        c["a"] = self.S("stem.a")
        if pool:
            c["p"], c["am"] = self.pool_fwd(c["a"], "stem.p")
        return c

    def stem_bwd(self, c, pool):
        if pool:
            ref, t = self.pool_bwd_value(self.S("d:stem.p"), c["am"], c["a"].shape)
            self.chk("d:stem.a", self.S("d:stem.a"), ref, terms=t)
        self.bn_bwd("stem.bn", self.S("d:stem.a"), c["h"], c["a"], True, c["st"], "d:stem.h")
        self.conv_wgrad("stem.w", c["x"], self.S("d:stem.h"), 7, 2, 3)

    def head(self, topname, labels):
        """GAP -> FC -> CE on the GPU's top features: logits and loss (float32
        gates), the FC gradients and the top gradient."""
        top = self.S(topname)
        n = top.shape[0]
        g = ops.gap_fwd(top)
        W, b = self.P["fc.w"], self.P["fc.b"]
        logits = ops.fc_fwd(g, W, b)
        self.chk("logits", self.S("logits").reshape(n, 2), logits, dt="f32",
                 terms=np.abs(g) @ np.abs(W).T + np.abs(b))
        loss, dl = ops.ce_fwd_bwd(logits, np.asarray(labels))
        gl = float(self.S("loss").ravel()[0])
        assert abs(gl - loss) <= 1e-4 * abs(loss) + 1e-6, ("loss", gl, loss)
        self.checks += 1
        if self.verbose:
            print("   %-30s %.8f vs %.8f" % ("loss", gl, loss), flush=True)
        dg, dwf, dbf = ops.fc_bwd(dl, g, W)
        self.add_grad("fc.w", dwf, np.abs(dl).T @ np.abs(g))
        self.add_grad("fc.b", dbf, np.abs(dl).sum(axis=0))
        dtop = ops.gap_bwd(dg, top.shape[2:])
        tt = ops.gap_bwd(np.abs(dl) @ np.abs(W), top.shape[2:])
        self.chk("d:" + topname, self.S("d:" + topname), self.rnd(dtop), terms=tt)

    # ------------------------------------------------------------ workloads
    def resunit(self, S):
        self.S = S
        c = self.ru_fwd("", "x", 1)
        self.ru_bwd("", c, "d:y", "d:x")

    def attn(self, S):
        self.S = S
        c = self.am_fwd("", "x", "out")
        self.am_bwd("", c, "d:out", "d:x")

    def partition1(self, S):
        self.S = S
        cs = self.stem_fwd(pool=False)
        cr = self.ru_fwd("ru.", "stem.a", 1)
        ca = self.am_fwd("am.", "ru.y", "am.out")
        self.am_bwd("am.", ca, "d:am.out", "d:ru.y")
        self.ru_bwd("ru.", cr, "d:ru.y", "d:stem.a")
        self.stem_bwd(cs, pool=False)

    def resattnet(self, S, labels, stages=3):
        self.S = S
        cs = self.stem_fwd(pool=True)
        h = "stem.p"
        caches = []
        for i in range(stages):
            pre = "s%d." % (i + 1)
            cr = self.ru_fwd(pre + "ru.", h, 1 if i == 0 else 2)
            ca = self.am_fwd(pre + "am.", pre + "ru.y", pre + "am.out")
            caches.append((cr, ca, h))
            h = pre + "am.out"
        self.head(h, labels)
        for i in reversed(range(stages)):
            pre = "s%d." % (i + 1)
            cr, ca, hin = caches[i]
            self.am_bwd(pre + "am.", ca, "d:" + pre + "am.out", "d:" + pre + "ru.y")
            self.ru_bwd(pre + "ru.", cr, "d:" + pre + "ru.y", "d:" + hin)
        self.stem_bwd(cs, pool=True)

    def gradcam(self, S, classes, target, stages=3):
        """Inference-mode Grad-CAM pass (the forward, the logits, the seed
        d logit_k / d top, and the backward down to the target map); the map
        kernels themselves are checked by the caller on the GPU's A and dA."""
        assert self.eval_stats is not None
        self.S = S
        cs = self.stem_fwd(pool=True)
        h = "stem.p"
        caches = []
        for i in range(stages):
            pre = "s%d." % (i + 1)
            cr = self.ru_fwd(pre + "ru.", h, 1 if i == 0 else 2)
            ca = self.am_fwd(pre + "am.", pre + "ru.y", pre + "am.out")
            caches.append((cr, ca, h))
            h = pre + "am.out"
        top = S(h)
        W, b = self.P["fc.w"], self.P["fc.b"]
        g = ops.gap_fwd(top)
        self.chk("logits", S("logits"), ops.fc_fwd(g, W, b), dt="f32",
                 terms=np.abs(g) @ np.abs(W).T + np.abs(b))
        V = top.shape[2] * top.shape[3] * top.shape[4]
        seed = np.stack([W[int(k)] for k in classes])[:, :, None, None, None] / V
        seed = np.broadcast_to(seed, top.shape)
        self.chk("d:" + h, S("d:" + h), self.rnd(seed), terms=np.abs(seed))
        del cs
        for i in reversed(range(target, stages)):
            pre = "s%d." % (i + 1)
            cr, ca, hin = caches[i]
            self.am_bwd(pre + "am.", ca, "d:" + pre + "am.out", "d:" + pre + "ru.y")
            self.ru_bwd(pre + "ru.", cr, "d:" + pre + "ru.y", "d:" + hin)

    # ------------------------------------------------------------ gradients
    def finish(self, G):
        """Gate the GPU's gradient arena against the summed per-layer oracle
        gradients: every tensor element-wise (float32 sums, sum|terms|
        bound) and norm-wise at the stated tolerance, except the per-channel
        BN sums (dgamma, dbeta) and conv biases, which cancel by construction
        and are gated element-wise only."""
        assert set(G) == set(self.G), (sorted(set(G) ^ set(self.G)))
        for k in sorted(self.G):
            ts = self.T[k]
            if all(callable(t) for t in ts):
                def terms(idx, ts=ts):
                    return sum(t(idx) for t in ts)
            else:
                terms = sum(np.asarray(t, np.float64) for t in ts)
            cancel = k.endswith(".g") or k.endswith(".b") or k.endswith(".bias")
            self.chk("grad " + k, G[k], self.G[k], kind="sum", norm=not cancel, terms=terms)
        if self.verbose:
            print("replay: %d checks, %d of %d stored elements differ by more than one ulp" % (
                self.checks, self.above_1ulp, self.elements), flush=True)
