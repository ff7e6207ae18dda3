"""Oracle composition of the 3D-ResAttNet training step (TEST INFRASTRUCTURE ONLY).

Builds the residual unit, the residual attention module, the full network and
the first-stage partition out of the float64 operations in ``oracle.ops``,
with explicit forward and backward passes (plain reverse-mode chain rule).

Paper anchors (arXiv 2104.05035): the network is 3D-ResAttNet built from conv
blocks (3x3x3 conv, 3D batch norm, ReLU), residual layers made of two conv
blocks, and a self-attention layer inside the residual self-attention block
(use-case section); the loss is the batch-mean cross-entropy and the update is
plain SGD at learning rate 1e-4 (experiments section); a partition computes
its weight gradients from the gradient received at its output and accumulates
them before the update (model-parallelisation section).  The paper does not
spell out the attention layer, the stage layout or the rounding points; the
readings implemented here (one per function) are listed in the repository's
design notes:
  * residual unit: conv3 -> BN -> ReLU -> conv3 -> BN, plus skip, then ReLU;
    the skip is a 1^3 conv (stride s, no bias) + BN when the channel count or
    stride changes, identity otherwise; 3^3 convs use pad 1 and no bias;
  * attention module: trunk = 2 residual units; mask = maxpool -> RU ->
    maxpool -> RU -> RU -> trilinear up -> RU -> trilinear up -> 1^3 conv (no
    bias) -> BN -> ReLU -> 1^3 conv (+bias) -> sigmoid; output (1 + M) * T;
    max pooling 3^3 stride 2 pad 1; upsampling goes back to the pre-pool size;
  * stem: 7^3 conv stride 2 pad 3 (no bias) -> BN -> ReLU (-> maxpool 3^3 s2
    p1 in the full network only);
  * full network: stem, then three stages (64, 128, 256 channels), each a
    residual unit (stride 1 for the first, 2 for the others) followed by an
    attention module; global average pool, FC to 2 classes, cross-entropy;
  * bfloat16 mode: every stored activation and activation gradient is rounded
    to bfloat16 where the GPU stores it, and convolutions use the bfloat16
    working copy of their weights (the float32 master rounded to nearest
    even); conv biases, BN parameters, the FC layer, weight gradients, BN
    statistics, the pooled features, logits and loss stay unrounded.
"""
import numpy as np

from . import ops

# --------------------------------------------------------------------------
# Parameter layout (arena order): for each conv, weight then bias if any; for
# each BN, gamma then beta; the FC weight and bias last.  Residual unit order:
# conv1, bn1, conv2, bn2, then (if present) the projection conv and its BN.
# Attention module order: trunk unit 1, trunk unit 2, mask units 1..4, the
# first 1^3 conv, its BN, the second 1^3 conv (weight, bias).
# --------------------------------------------------------------------------


def _ru_params(pre, cin, cout, stride):
    out = [(pre + "conv1.w", (cout, cin, 3, 3, 3)),
           (pre + "bn1.g", (cout,)), (pre + "bn1.b", (cout,)),
           (pre + "conv2.w", (cout, cout, 3, 3, 3)),
           (pre + "bn2.g", (cout,)), (pre + "bn2.b", (cout,))]
    if cin != cout or stride != 1:
        out += [(pre + "proj.w", (cout, cin, 1, 1, 1)),
                (pre + "projbn.g", (cout,)), (pre + "projbn.b", (cout,))]
    return out


def _am_params(pre, c):
    out = []
    for u in ("t1.", "t2.", "m1.", "m2.", "m3.", "m4."):
        out += _ru_params(pre + u, c, c, 1)
    out += [(pre + "c1.w", (c, c, 1, 1, 1)),
            (pre + "bn.g", (c,)), (pre + "bn.b", (c,)),
            (pre + "c2.w", (c, c, 1, 1, 1)), (pre + "c2.bias", (c,))]
    return out


def _stem_params(c):
    return [("stem.w", (c, 1, 7, 7, 7)), ("stem.bn.g", (c,)), ("stem.bn.b", (c,))]


STAGES = (64, 128, 256)


def param_layout(kind, c_in, c, stages=STAGES, stem_c=32):
    """Ordered (name, shape) list of the trainable parameters.

    kind: 'resunit' (c_in -> c, stride 1), 'attn' (c channels),
          'resattnet' (stem to stem_c channels, then one stage per entry of
          `stages`, FC to 2), 'partition1' (stem to stem_c channels,
          RU stem_c -> c, attention module c).
    The forward/backward functions read channel counts from the weight
    shapes, so a reduced channel plan only changes this layout.
    """
    if kind == "resunit":
        return _ru_params("", c_in, c, 1)
    if kind == "attn":
        return _am_params("", c)
    if kind == "resattnet":
        out = _stem_params(stem_c)
        cprev = stem_c
        for i, cs in enumerate(stages):
            out += _ru_params("s%d.ru." % (i + 1), cprev, cs, 1 if i == 0 else 2)
            out += _am_params("s%d.am." % (i + 1), cs)
            cprev = cs
        out += [("fc.w", (2, stages[-1])), ("fc.b", (2,))]
        return out
    if kind == "partition1":
        return (_stem_params(stem_c) + _ru_params("ru.", stem_c, c, 1)
                + _am_params("am.", c))
    raise ValueError(kind)


def bn_names(layout):
    """Names of the BN layers (prefix before '.g'), in arena order."""
    return [n[:-2] for n, _ in layout if n.endswith(".g")]


def n_stages(params):
    """Number of stages of a full-network parameter dict."""
    return len({k.split(".")[0] for k in params if k.startswith("s")
                and k.split(".")[0][1:].isdigit()})


# --------------------------------------------------------------------------
# Execution context
# --------------------------------------------------------------------------
class Ctx:
    """Holds rounding mode, BN settings, the gradient dict and running stats.

    jitter = (rel, seed) multiplies every stored value by (1 + rel * N(0,1))
    before its rounding.  It is off by default; the parity tests use it to
    measure how far the step's results move under rounding-level noise (the
    step has ReLU and max-pool decisions, so it is only piecewise smooth).
    """

    def __init__(self, params, bf16, eps=1e-5, momentum=0.1, running=None, jitter=None,
                 eval_stats=None):
        self.P = params
        # inference mode: BN applies the given running statistics
        # {bn name: (mean, var)} and no parameter gradient is formed
        self.eval_stats = eval_stats
        self.param_grads = eval_stats is None
        base = ops.round_bf16 if bf16 else ops.identity
        if jitter is None:
            self.rnd = base
        else:
            rel, seed = jitter
            noise = np.random.default_rng(seed)
            self.rnd = lambda a: base(np.asarray(a, dtype=np.float64)
                                      * (1.0 + rel * noise.standard_normal(np.shape(a))))
        self.eps = eps
        self.momentum = momentum
        self.G = {k: np.zeros_like(v) for k, v in params.items()}
        self.running = running if running is not None else {}
        self.acts = {}

    def w(self, name):
        """Conv weight as the convolution sees it (bf16 working copy in bf16 mode)."""
        return self.rnd(self.P[name])

    def bn(self, name, x, relu, residual=None):
        if self.eval_stats is not None:
            rm, rv = self.eval_stats[name]
            return self.rnd(ops.bn_eval_fwd(x, self.P[name + ".g"], self.P[name + ".b"], rm, rv,
                                            self.eps, relu, residual)), None
        y, mean, var, invstd = ops.bn_fwd(x, self.P[name + ".g"], self.P[name + ".b"],
                                          self.eps, relu, residual)
        cnt = x.shape[0] * x.shape[2] * x.shape[3] * x.shape[4]
        rm, rv = self.running.get(name, (np.zeros(x.shape[1]), np.ones(x.shape[1])))
        self.running[name] = ops.bn_running_update(rm, rv, mean, var, cnt, self.momentum)
        return self.rnd(y), (mean, invstd)

    def bn_back(self, name, dy, x, y, st, relu):
        if self.eval_stats is not None:
            dx, g = ops.bn_eval_bwd(dy, y, self.P[name + ".g"], self.eval_stats[name][1],
                                    self.eps, relu)
            return self.rnd(dx), self.rnd(g)
        dx, g, dgam, dbet = ops.bn_bwd(dy, x, y, self.P[name + ".g"], st[0], st[1], relu)
        self.G[name + ".g"] += dgam
        self.G[name + ".b"] += dbet
        return self.rnd(dx), self.rnd(g)


# --------------------------------------------------------------------------
# Residual unit
# --------------------------------------------------------------------------
def ru_fwd(ctx, pre, x, stride):
    P, rnd = ctx.P, ctx.rnd
    proj = (pre + "proj.w") in P
    h1 = rnd(ops.conv3d_fwd(x, ctx.w(pre + "conv1.w"), None, stride, 1))
    a1, st1 = ctx.bn(pre + "bn1", h1, relu=True)
    h2 = rnd(ops.conv3d_fwd(a1, ctx.w(pre + "conv2.w"), None, 1, 1))
    if proj:
        hp = rnd(ops.conv3d_fwd(x, ctx.w(pre + "proj.w"), None, stride, 0))
        sp, stp = ctx.bn(pre + "projbn", hp, relu=False)
        skip = sp
    else:
        hp = sp = stp = None
        skip = x
    y, st2 = ctx.bn(pre + "bn2", h2, relu=True, residual=skip)
    ctx.acts[pre + "y"] = y
    cache = dict(x=x, h1=h1, a1=a1, h2=h2, y=y, hp=hp, sp=sp, st1=st1, st2=st2,
                 stp=stp, stride=stride, proj=proj)
    return y, cache


def ru_bwd(ctx, pre, c, dy, dx_acc=None):
    """Backward of ru_fwd.  The gradient of the unit input is formed as
    rnd(rnd(skip-branch gradient [+ dx_acc]) + conv1 input gradient)."""
    P, G, rnd = ctx.P, ctx.G, ctx.rnd
    x, s = c["x"], c["stride"]
    dh2, dskip = ctx.bn_back(pre + "bn2", dy, c["h2"], c["y"], c["st2"], relu=True)
    da1 = rnd(ops.conv3d_dgrad(dh2, ctx.w(pre + "conv2.w"), c["a1"].shape, 1, 1))
    if ctx.param_grads:
        G[pre + "conv2.w"] += ops.conv3d_wgrad(c["a1"], dh2, 3, 1, 1, False)[0]
    dh1, _ = ctx.bn_back(pre + "bn1", da1, c["h1"], c["a1"], c["st1"], relu=True)
    if c["proj"]:
        dhp, _ = ctx.bn_back(pre + "projbn", dskip, c["hp"], c["sp"], c["stp"], relu=False)
        dxs = ops.conv3d_dgrad(dhp, ctx.w(pre + "proj.w"), x.shape, s, 0)
        if ctx.param_grads:
            G[pre + "proj.w"] += ops.conv3d_wgrad(x, dhp, 1, s, 0, False)[0]
    else:
        dxs = dskip
    dx = rnd(dxs if dx_acc is None else dx_acc + dxs)
    dx = rnd(dx + ops.conv3d_dgrad(dh1, ctx.w(pre + "conv1.w"), x.shape, s, 1))
    if ctx.param_grads:
        G[pre + "conv1.w"] += ops.conv3d_wgrad(x, dh1, 3, s, 1, False)[0]
    return dx


# --------------------------------------------------------------------------
# Residual attention module
# --------------------------------------------------------------------------
def am_fwd(ctx, pre, x):
    P, rnd = ctx.P, ctx.rnd
    t1, ct1 = ru_fwd(ctx, pre + "t1.", x, 1)
    T, ct2 = ru_fwd(ctx, pre + "t2.", t1, 1)
    p1, am1 = ops.maxpool3d_fwd(x)
    p1 = rnd(p1)
    r1, cm1 = ru_fwd(ctx, pre + "m1.", p1, 1)
    p2, am2 = ops.maxpool3d_fwd(r1)
    p2 = rnd(p2)
    r2a, cm2 = ru_fwd(ctx, pre + "m2.", p2, 1)
    r2b, cm3 = ru_fwd(ctx, pre + "m3.", r2a, 1)
    u1 = rnd(ops.trilinear_fwd(r2b, r1.shape[2:]))
    r3, cm4 = ru_fwd(ctx, pre + "m4.", u1, 1)
    u2 = rnd(ops.trilinear_fwd(r3, x.shape[2:]))
    c1 = rnd(ops.conv3d_fwd(u2, ctx.w(pre + "c1.w"), None, 1, 0))
    a, stb = ctx.bn(pre + "bn", c1, relu=True)
    z = rnd(ops.conv3d_fwd(a, ctx.w(pre + "c2.w"), P[pre + "c2.bias"], 1, 0))
    out, m = ops.softmask_fwd(z, T, rnd)
    ctx.acts[pre + "T"] = T
    ctx.acts[pre + "z"] = z
    ctx.acts[pre + "out"] = out
    cache = dict(x=x, ct1=ct1, ct2=ct2, T=T, am1=am1, am2=am2, p1=p1, r1=r1,
                 cm1=cm1, cm2=cm2, cm3=cm3, cm4=cm4, r2b=r2b, u1=u1, r3=r3, u2=u2,
                 c1=c1, a=a, stb=stb, z=z, m=m)
    return out, cache


def am_bwd(ctx, pre, c, dout):
    """Backward of am_fwd.  Mask branch first; its input gradient is stored,
    then the trunk's input gradient is accumulated onto it (see ru_bwd)."""
    P, G, rnd = ctx.P, ctx.G, ctx.rnd
    x = c["x"]
    dT, dz = ops.softmask_bwd(dout, c["T"], c["m"], rnd)
    da = rnd(ops.conv3d_dgrad(dz, ctx.w(pre + "c2.w"), c["a"].shape, 1, 0))
    if ctx.param_grads:
        dw, db = ops.conv3d_wgrad(c["a"], dz, 1, 1, 0, True)
        G[pre + "c2.w"] += dw
        G[pre + "c2.bias"] += db
    dc1, _ = ctx.bn_back(pre + "bn", da, c["c1"], c["a"], c["stb"], relu=True)
    du2 = rnd(ops.conv3d_dgrad(dc1, ctx.w(pre + "c1.w"), c["u2"].shape, 1, 0))
    if ctx.param_grads:
        G[pre + "c1.w"] += ops.conv3d_wgrad(c["u2"], dc1, 1, 1, 0, False)[0]
    dr3 = rnd(ops.trilinear_bwd(du2, c["r3"].shape[2:]))
    du1 = ru_bwd(ctx, pre + "m4.", c["cm4"], dr3)
    dr2b = rnd(ops.trilinear_bwd(du1, c["r2b"].shape[2:]))
    dr2a = ru_bwd(ctx, pre + "m3.", c["cm3"], dr2b)
    dp2 = ru_bwd(ctx, pre + "m2.", c["cm2"], dr2a)
    dr1 = rnd(ops.maxpool3d_bwd(dp2, c["am2"], c["r1"].shape))
    dp1 = ru_bwd(ctx, pre + "m1.", c["cm1"], dr1)
    dx = rnd(ops.maxpool3d_bwd(dp1, c["am1"], x.shape))
    dt1 = ru_bwd(ctx, pre + "t2.", c["ct2"], dT)
    return ru_bwd(ctx, pre + "t1.", c["ct1"], dt1, dx_acc=dx)


# --------------------------------------------------------------------------
# Stem
# --------------------------------------------------------------------------
def stem_fwd(ctx, x, pool):
    rnd = ctx.rnd
    h0 = rnd(ops.conv3d_fwd(x, ctx.w("stem.w"), None, 2, 3))
    a0, st0 = ctx.bn("stem.bn", h0, relu=True)
    c = dict(x=x, h0=h0, a0=a0, st0=st0, pool=pool)
    if pool:
        p0, am0 = ops.maxpool3d_fwd(a0)
        p0 = rnd(p0)
        c["am0"] = am0
        return p0, c
    return a0, c


def stem_bwd(ctx, c, dy):
    rnd = ctx.rnd
    da0 = rnd(ops.maxpool3d_bwd(dy, c["am0"], c["a0"].shape)) if c["pool"] else dy
    dh0, _ = ctx.bn_back("stem.bn", da0, c["h0"], c["a0"], c["st0"], relu=True)
    if ctx.param_grads:
        ctx.G["stem.w"] += ops.conv3d_wgrad(c["x"], dh0, 7, 2, 3, False)[0]


# --------------------------------------------------------------------------
# Whole-block drivers
# --------------------------------------------------------------------------
def block_fwd_bwd(kind, params, x, dy, bf16, eps=1e-5, jitter=None):
    """Forward + backward of one residual unit ('resunit') or one attention
    module ('attn').  Returns (y, dx, grads, ctx)."""
    ctx = Ctx(params, bf16, eps, jitter=jitter)
    x = ctx.rnd(np.asarray(x, dtype=np.float64))
    dy = ctx.rnd(np.asarray(dy, dtype=np.float64))
    if kind == "resunit":
        y, c = ru_fwd(ctx, "", x, 1)
        dx = ru_bwd(ctx, "", c, dy)
    elif kind == "attn":
        y, c = am_fwd(ctx, "", x)
        dx = am_bwd(ctx, "", c, dy)
    else:
        raise ValueError(kind)
    return y, dx, ctx.G, ctx


def resattnet_fwd_bwd(params, x, labels, bf16, eps=1e-5, running=None, jitter=None):
    """Full network forward, loss, backward.  Returns (loss, logits, grads, ctx)."""
    ctx = Ctx(params, bf16, eps, running=running, jitter=jitter)
    x = ctx.rnd(np.asarray(x, dtype=np.float64))
    h, cs = stem_fwd(ctx, x, pool=True)
    caches = []
    ns = n_stages(params)
    for i in range(ns):
        pre = "s%d." % (i + 1)
        h, cr = ru_fwd(ctx, pre + "ru.", h, 1 if i == 0 else 2)
        h, ca = am_fwd(ctx, pre + "am.", h)
        caches.append((cr, ca))
    g = ops.gap_fwd(h)
    logits = ops.fc_fwd(g, params["fc.w"], params["fc.b"])
    loss, dl = ops.ce_fwd_bwd(logits, np.asarray(labels))
    dg, dwf, dbf = ops.fc_bwd(dl, g, params["fc.w"])
    ctx.G["fc.w"] += dwf
    ctx.G["fc.b"] += dbf
    dh = ctx.rnd(ops.gap_bwd(dg, h.shape[2:]))
    for i in reversed(range(ns)):
        pre = "s%d." % (i + 1)
        cr, ca = caches[i]
        dh = am_bwd(ctx, pre + "am.", ca, dh)
        dh = ru_bwd(ctx, pre + "ru.", cr, dh)
    stem_bwd(ctx, cs, dh)
    ctx.acts["logits"] = logits
    return loss, logits, ctx.G, ctx


def partition1_fwd_bwd(params, x, dy, bf16, eps=1e-5, running=None, grads=None,
                       jitter=None):
    """First-stage partition (stem -> RU 32->c -> attention module) forward and
    backward for one micro-batch, given the gradient received at its output.
    Gradients are added to `grads` when given.  Returns (y, grads, ctx)."""
    ctx = Ctx(params, bf16, eps, running=running, jitter=jitter)
    if grads is not None:
        ctx.G = grads
    x = ctx.rnd(np.asarray(x, dtype=np.float64))
    dy = ctx.rnd(np.asarray(dy, dtype=np.float64))
    h, cs = stem_fwd(ctx, x, pool=False)
    h, cr = ru_fwd(ctx, "ru.", h, 1)
    y, ca = am_fwd(ctx, "am.", h)
    d = am_bwd(ctx, "am.", ca, dy)
    d = ru_bwd(ctx, "ru.", cr, d)
    stem_bwd(ctx, cs, d)
    return y, ctx.G, ctx


def train_step(kind, params, lr, bf16, x=None, labels=None, dy=None,
               micro_batches=1, eps=1e-5, jitter=None):
    """One SGD step: gradients of the batch (summed over micro-batches), then
    w <- w - lr * g.  Returns (new_params, grads, info)."""
    running = {}
    if kind == "resattnet":
        loss, logits, G, ctx = resattnet_fwd_bwd(params, x, labels, bf16, eps, running,
                                                 jitter)
        info = dict(loss=loss, logits=logits, running=running, acts=ctx.acts)
    elif kind == "partition1":
        G = {k: np.zeros_like(v) for k, v in params.items()}
        ys = []
        nb = x.shape[0] // micro_batches
        for mb in range(micro_batches):
            sl = slice(mb * nb, (mb + 1) * nb)
            jit = None if jitter is None else (jitter[0], jitter[1] + mb)
            y, G, ctx = partition1_fwd_bwd(params, x[sl], dy[sl], bf16, eps, running, G, jit)
            ys.append(y)
        info = dict(y=ys, running=running)
    else:
        raise ValueError(kind)
    new = {k: ops.sgd(v, G[k], lr) for k, v in params.items()}
    return new, G, info


def gradcam(params, x, classes, running, target, bf16, eps=1e-5):
    """3D Grad-CAM of the full network (the explainable block of the use-case
    section; gradient-weighted class activation mapping), in inference mode:
    BN applies the running statistics `running` = {bn name: (mean, var)}.

      y^k    = logit of class k = classes[n] for volume n (before the softmax);
      A      = output of the target stage (0: the stem after pooling, s >= 1:
               stage s's attention module), shape (N, C, D, H, W);
      alpha  = alpha[n, c] = mean over voxels of d y^k / d A[n, c];
      cam    = ReLU(sum_c alpha[n, c] A[n, c]), shape (N, D, H, W);
      up     = cam resampled trilinearly (half-pixel centres) to the input's
               D, H, W.
    bf16 mode rounds stored activations and activation gradients as in
    training; alpha, cam and up stay unrounded.  Returns dict(logits, A, dA,
    alpha, cam, up)."""
    ctx = Ctx(params, bf16, eps, eval_stats=running)
    x = ctx.rnd(np.asarray(x, dtype=np.float64))
    h, cs = stem_fwd(ctx, x, pool=True)
    ns = n_stages(params)
    caches = []
    acts = [h]
    for i in range(ns):
        pre = "s%d." % (i + 1)
        h, cr = ru_fwd(ctx, pre + "ru.", h, 1 if i == 0 else 2)
        h, ca = am_fwd(ctx, pre + "am.", h)
        caches.append((cr, ca))
        acts.append(h)
    g = ops.gap_fwd(h)
    logits = ops.fc_fwd(g, params["fc.w"], params["fc.b"])
    n = x.shape[0]
    # d y^k / d(pooled features) = fc.w[k]; the average pool spreads it evenly
    dg = np.stack([params["fc.w"][int(classes[i])] for i in range(n)])
    dh = ctx.rnd(ops.gap_bwd(dg, h.shape[2:]))
    for i in reversed(range(target, ns)):
        pre = "s%d." % (i + 1)
        cr, ca = caches[i]
        dh = am_bwd(ctx, pre + "am.", ca, dh)
        dh = ru_bwd(ctx, pre + "ru.", cr, dh)
    A = acts[target]
    alpha = dh.mean(axis=(2, 3, 4))
    cam = np.maximum((alpha[:, :, None, None, None] * A).sum(axis=1), 0.0)
    up = ops.trilinear_fwd(cam[:, None], x.shape[2:])[:, 0]
    return dict(logits=logits, A=A, dA=dh, alpha=alpha, cam=cam, up=up)
