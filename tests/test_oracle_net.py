"""Pins for the oracle's composed training step: the hand-written backward of
the residual unit, attention module, full network and partition is checked
against an independent torch-autograd build of the same graph and against
central finite differences (float64); plus the micro-batch accumulation
identity, the parameter counts and the conv FLOP totals."""
import numpy as np
import pytest

from oracle import net, ops
from paper_2104_05035_amd import synth


def _params(kind, c_in, c, seed, **kw):
    rng = np.random.default_rng(seed)
    layout = net.param_layout(kind, c_in, c, **kw)
    return synth.init_params(rng, layout, bias_std=0.1, perturb_bn=0.2), layout


# ------------------------------------------------------- torch re-build
def _torch_graph(running=None):
    """The graph in torch ops; with `running` = {bn name: (mean, var)} the BN
    layers run in inference mode on those statistics."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional

    def bn(P, name, x):
        if running is not None:
            rm, rv = running[name]
            return F.batch_norm(x, torch.tensor(rm), torch.tensor(rv), P[name + ".g"],
                                P[name + ".b"], training=False, eps=1e-5)
        return F.batch_norm(x, None, None, P[name + ".g"], P[name + ".b"], training=True,
                            eps=1e-5)

    def ru(P, pre, x, s):
        a1 = torch.relu(bn(P, pre + "bn1", F.conv3d(x, P[pre + "conv1.w"], None, s, 1)))
        h2 = bn(P, pre + "bn2", F.conv3d(a1, P[pre + "conv2.w"], None, 1, 1))
        if pre + "proj.w" in P:
            skip = bn(P, pre + "projbn", F.conv3d(x, P[pre + "proj.w"], None, s, 0))
        else:
            skip = x
        return torch.relu(h2 + skip)

    def am(P, pre, x):
        T = ru(P, pre + "t2.", ru(P, pre + "t1.", x, 1), 1)
        r1 = ru(P, pre + "m1.", F.max_pool3d(x, 3, 2, 1), 1)
        r2 = ru(P, pre + "m3.", ru(P, pre + "m2.", F.max_pool3d(r1, 3, 2, 1), 1), 1)
        u1 = F.interpolate(r2, size=r1.shape[2:], mode="trilinear", align_corners=False)
        r3 = ru(P, pre + "m4.", u1, 1)
        u2 = F.interpolate(r3, size=x.shape[2:], mode="trilinear", align_corners=False)
        a = torch.relu(bn(P, pre + "bn", F.conv3d(u2, P[pre + "c1.w"])))
        z = F.conv3d(a, P[pre + "c2.w"], P[pre + "c2.bias"])
        return (1.0 + torch.sigmoid(z)) * T

    def stem(P, x, pool):
        a0 = torch.relu(bn(P, "stem.bn", F.conv3d(x, P["stem.w"], None, 2, 3)))
        return F.max_pool3d(a0, 3, 2, 1) if pool else a0

    def resattnet(P, x, labels, nst):
        h = stem(P, x, True)
        for i in range(nst):
            h = ru(P, "s%d.ru." % (i + 1), h, 1 if i == 0 else 2)
            h = am(P, "s%d.am." % (i + 1), h)
        logits = F.linear(h.mean(dim=(2, 3, 4)), P["fc.w"], P["fc.b"])
        return F.cross_entropy(logits, labels), logits

    def partition1(P, x):
        return am(P, "am.", ru(P, "ru.", stem(P, x, False), 1))

    return torch, dict(ru=ru, am=am, resattnet=resattnet, partition1=partition1, stem=stem)


def _tp(torch, params):
    return {k: torch.tensor(v, requires_grad=True) for k, v in params.items()}


def _cmp_grads(G, TP, rtol=1e-9):
    for k, t in TP.items():
        ref = t.grad.numpy()
        err = np.linalg.norm(G[k] - ref) / max(np.linalg.norm(ref), 1e-300)
        assert err < rtol, (k, err)


def test_resunit_against_autograd():
    torch, g = _torch_graph()
    for c_in, c, proj in [(3, 3, False)]:
        P, _ = _params("resunit", c_in, c, 1)
        rng = np.random.default_rng(2)
        x = rng.standard_normal((2, c_in, 5, 6, 4))
        dy = rng.standard_normal((2, c, 5, 6, 4))
        y, dx, G, _ = net.block_fwd_bwd("resunit", P, x, dy, bf16=False)
        TP = _tp(torch, P)
        xt = torch.tensor(x, requires_grad=True)
        yt = g["ru"](TP, "", xt, 1)
        np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-11, atol=1e-11)
        yt.backward(torch.tensor(dy))
        np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-9, atol=1e-10)
        _cmp_grads(G, TP)


def test_attn_against_autograd():
    torch, g = _torch_graph()
    P, _ = _params("attn", 4, 4, 3)
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2, 4, 8, 10, 7))
    dy = rng.standard_normal((2, 4, 8, 10, 7))
    y, dx, G, _ = net.block_fwd_bwd("attn", P, x, dy, bf16=False)
    TP = _tp(torch, P)
    xt = torch.tensor(x, requires_grad=True)
    yt = g["am"](TP, "", xt)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-10, atol=1e-10)
    yt.backward(torch.tensor(dy))
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-8, atol=1e-9)
    _cmp_grads(G, TP, 1e-8)


def test_resattnet_against_autograd():
    torch, g = _torch_graph()
    P, _ = _params("resattnet", 1, 4, 5, stages=(8, 8, 8), stem_c=4)
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 1, 24, 28, 24))
    labels = np.array([0, 1])
    loss, logits, G, _ = net.resattnet_fwd_bwd(P, x, labels, bf16=False)
    TP = _tp(torch, P)
    Lt, lt = g["resattnet"](TP, torch.tensor(x), torch.tensor(labels), 3)
    assert abs(loss - Lt.item()) < 1e-10
    np.testing.assert_allclose(logits, lt.detach().numpy(), rtol=1e-10, atol=1e-10)
    Lt.backward()
    _cmp_grads(G, TP, 1e-7)


def test_partition1_against_autograd_and_accumulation():
    torch, g = _torch_graph()
    P, _ = _params("partition1", 1, 8, 7, stem_c=4)
    rng = np.random.default_rng(8)
    x = rng.standard_normal((2, 1, 12, 14, 12))
    dy = rng.standard_normal((2, 8, 6, 7, 6))
    y, G, _ = net.partition1_fwd_bwd(P, x, dy, bf16=False)
    TP = _tp(torch, P)
    yt = g["partition1"](TP, torch.tensor(x))
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-10, atol=1e-10)
    yt.backward(torch.tensor(dy))
    _cmp_grads(G, TP, 1e-8)
    # four identical micro-batches accumulate to four times one micro-batch
    xs, dys = np.concatenate([x] * 4), np.concatenate([dy] * 4)
    new, G4, info = net.train_step("partition1", P, 1e-4, False, x=xs, dy=dys,
                                   micro_batches=4)
    for k in P:
        np.testing.assert_allclose(G4[k], 4 * G[k], rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(new[k], P[k] - 1e-4 * G4[k], rtol=1e-15, atol=0)


def test_resattnet_finite_differences():
    P, layout = _params("resattnet", 1, 4, 9, stages=(6, 6, 6), stem_c=4)
    rng = np.random.default_rng(10)
    x = rng.standard_normal((2, 1, 20, 24, 20))
    labels = np.array([1, 0])
    loss, _, G, _ = net.resattnet_fwd_bwd(P, x, labels, bf16=False)
    h = 1e-6
    names = ["stem.w", "s1.ru.conv1.w", "s1.ru.projbn.g", "s2.am.m3.conv2.w",
             "s2.am.c2.bias", "s3.am.t1.bn2.b", "s3.am.c1.w", "fc.w"]
    for name in names:
        idx = tuple(rng.integers(0, m) for m in P[name].shape)
        Pp = {k: v.copy() for k, v in P.items()}
        Pm = {k: v.copy() for k, v in P.items()}
        Pp[name][idx] += h
        Pm[name][idx] -= h
        lp = net.resattnet_fwd_bwd(Pp, x, labels, bf16=False)[0]
        lm = net.resattnet_fwd_bwd(Pm, x, labels, bf16=False)[0]
        fd = (lp - lm) / (2 * h)
        assert abs(fd - G[name][idx]) <= 1e-6 * max(1.0, abs(fd)) + 1e-8, (name, fd,
                                                                          G[name][idx])


def test_bf16_mode_stays_close_to_exact():
    P, _ = _params("attn", 4, 4, 12)
    rng = np.random.default_rng(13)
    x = rng.standard_normal((2, 4, 8, 8, 8))
    dy = rng.standard_normal((2, 4, 8, 8, 8))
    y32, dx32, G32, _ = net.block_fwd_bwd("attn", P, x, dy, bf16=False)
    xb, dyb = ops.round_bf16(x), ops.round_bf16(dy)
    y16, dx16, G16, _ = net.block_fwd_bwd("attn", P, xb, dyb, bf16=True)
    assert np.array_equal(y16, ops.round_bf16(y16))
    rel = lambda a, b: np.linalg.norm(a - b) / np.linalg.norm(b)
    # the forward stays within bfloat16 error; the input gradient of this tiny
    # module (BN over 16 values in the deepest mask level, near-tie argmax
    # flips) is far more sensitive, so only a loose sanity bound applies there
    assert rel(y16, y32) < 2e-2 and rel(dx16, dx32) < 0.3


def test_parameter_counts():
    count = lambda L: sum(int(np.prod(s)) for _, s in L)
    L4 = net.param_layout("resattnet", 1, 32)
    L5 = net.param_layout("partition1", 1, 64)
    assert sum(1 for n, s in L4 if len(s) == 5) == 52
    assert sum(1 for n, s in L5 if len(s) == 5) == 18
    assert count(L4) == 31594210 and count(L5) == 1516384


def _conv_list(kind, n, c_in, c, d, h, w):
    """(N, Ci, Co, out_spatial, k, needs_dgrad) of every conv of one pass,
    derived from the graph layout."""
    out = []

    def ru(cin, cout, sp, s):
        o = tuple((x + 2 - 3) // s + 1 for x in sp)
        out.append((n, cin, cout, o, 3, True))
        out.append((n, cout, cout, o, 3, True))
        if cin != cout or s != 1:
            out.append((n, cin, cout, o, 1, True))
        return o

    def am(cc, sp):
        ru(cc, cc, sp, 1); ru(cc, cc, sp, 1)
        p1 = tuple(ops.out_size(x, 3, 2, 1) for x in sp)
        ru(cc, cc, p1, 1)
        p2 = tuple(ops.out_size(x, 3, 2, 1) for x in p1)
        ru(cc, cc, p2, 1); ru(cc, cc, p2, 1); ru(cc, cc, p1, 1)
        out.append((n, cc, cc, sp, 1, True)); out.append((n, cc, cc, sp, 1, True))

    if kind == "attn":
        am(c, (d, h, w))
    elif kind in ("resattnet", "partition1"):
        sp = tuple(ops.out_size(x, 7, 2, 3) for x in (d, h, w))
        out.append((n, 1, 32, sp, 7, False))
        if kind == "resattnet":
            sp = tuple(ops.out_size(x, 3, 2, 1) for x in sp)
            cprev = 32
            for i, cs in enumerate(net.STAGES):
                sp = ru(cprev, cs, sp, 1 if i == 0 else 2)
                am(cs, sp)
                cprev = cs
        else:
            ru(32, c, sp, 1)
            am(c, sp)
    return out


def test_conv_flop_totals():
    def tot(kind, *a):
        L = _conv_list(kind, *a)
        fwd = sum(ops.conv_flops(nn, ci, co, sp, k) for nn, ci, co, sp, k, _ in L)
        allp = sum(ops.conv_flops(nn, ci, co, sp, k) * (3 if dg else 2)
                   for nn, ci, co, sp, k, dg in L)
        return fwd, allp, len(L)
    f3, a3, n3 = tot("attn", 4, 64, 64, 48, 48, 48)
    f4, a4, n4 = tot("resattnet", 8, 1, 32, 96, 112, 96)
    f5, a5, n5 = tot("partition1", 16, 1, 64, 96, 112, 96)
    assert (n3, n4, n5) == (14, 52, 18)
    assert abs(f3 / 1e9 - 453.7) < 0.1 and abs(a3 / 1e12 - 1.361) < 0.001
    assert abs(f4 / 1e9 - 331.2) < 0.1 and abs(a4 / 1e12 - 0.971) < 0.001
    assert abs(f5 / 1e12 - 2.856) < 0.001 and abs(a5 / 1e12 - 8.522) < 0.001


# ------------------------------------------------------- bf16 store points
def _is_bf16(a):
    a = np.asarray(a, dtype=np.float64)
    return np.array_equal(a, ops.round_bf16(a))


# for each operation the network calls: the positions (and keywords) of its
# arguments that are stored tensors -- activations, activation gradients, the
# bf16 weight copy -- in bf16 mode (None arguments are skipped)
_STORED_ARGS = {
    "conv3d_fwd": (0, 1), "conv3d_dgrad": (0, 1), "conv3d_wgrad": (0, 1),
    "maxpool3d_fwd": (0,), "maxpool3d_bwd": (0,), "trilinear_fwd": (0,),
    "trilinear_bwd": (0,), "bn_fwd": (0, 5, "residual"), "bn_bwd": (0, 1, 2),
    "softmask_fwd": (0, 1), "softmask_bwd": (0, 1, 2), "gap_fwd": (0,),
}


def _trace_inputs(monkeypatch):
    """Wraps the operations so that every call records its stored-tensor
    arguments and the unrounded float32 quantities they are given: the conv
    bias, the BN statistics passed to the backward, the pooled features."""
    seen = {"stored": [], "unrounded": []}
    for name, pos in _STORED_ARGS.items():
        f = getattr(ops, name)

        def wrap(*a, _f=f, _name=name, _pos=pos, **kw):
            for p in _pos:
                v = kw.get(p) if isinstance(p, str) else (a[p] if p < len(a) else None)
                if v is not None:
                    seen["stored"].append(("%s arg %s" % (_name, p), v))
            if _name == "conv3d_fwd" and len(a) > 2 and a[2] is not None:
                seen["unrounded"].append(("conv bias", a[2]))
            if _name == "bn_bwd":
                seen["unrounded"] += [("bn mean", a[4]), ("bn invstd", a[5])]
            return _f(*a, **kw)
        monkeypatch.setattr(ops, name, wrap)
    fc = ops.fc_fwd

    def fc_wrap(g, w, b):
        seen["unrounded"].append(("pooled features", g))
        return fc(g, w, b)
    monkeypatch.setattr(ops, "fc_fwd", fc_wrap)
    return seen


def test_bf16_store_points_partition(monkeypatch):
    """In bf16 mode every tensor an operation reads as a stored activation,
    activation gradient or conv weight is exactly bf16-representable (a missing
    rounding at a store point fails here), while the weight gradients, BN
    statistics and conv biases are not rounded (an extra rounding fails)."""
    seen = _trace_inputs(monkeypatch)
    P, _ = _params("partition1", 1, 8, 31)
    P = {k: v.astype(np.float32).astype(np.float64) for k, v in P.items()}
    rng = np.random.default_rng(32)
    x = rng.standard_normal((2, 1, 12, 16, 12))
    dy = rng.standard_normal((2, 8, 6, 8, 6))
    y, G, _ = net.partition1_fwd_bwd(P, x, dy, bf16=True)
    assert len(seen["stored"]) > 100
    for what, v in seen["stored"]:
        assert _is_bf16(v), what + " is not a bf16 store"
    assert _is_bf16(y)
    for what, v in seen["unrounded"]:
        assert not _is_bf16(v), what + " was rounded to bf16"
    for k, g in G.items():
        if g.size >= 4:
            assert not _is_bf16(g), "gradient of %s was rounded to bf16" % k


def test_bf16_store_points_network(monkeypatch):
    """The same for the full network (stem with pooling, two stages, head):
    additionally the logits and the loss stay unrounded."""
    seen = _trace_inputs(monkeypatch)
    P, _ = _params("resattnet", 1, 8, 33, stages=(8, 16), stem_c=8)
    P = {k: v.astype(np.float32).astype(np.float64) for k, v in P.items()}
    rng = np.random.default_rng(34)
    x = rng.standard_normal((2, 1, 48, 40, 48))
    labels = np.array([0, 1])
    loss, logits, G, _ = net.resattnet_fwd_bwd(P, x, labels, bf16=True)
    for what, v in seen["stored"]:
        assert _is_bf16(v), what + " is not a bf16 store"
    for what, v in seen["unrounded"]:
        assert not _is_bf16(v), what + " was rounded to bf16"
    assert not _is_bf16(logits) and not _is_bf16(np.array([loss]))
    for k, g in G.items():
        if g.size >= 4:
            assert not _is_bf16(g), "gradient of %s was rounded to bf16" % k


# ------------------------------------------------------- Grad-CAM
def _running(layout, seed):
    rng = np.random.default_rng(seed)
    return {b: (rng.normal(0, 0.3, dict(layout)[b + ".g"]),
                rng.uniform(0.5, 2.0, dict(layout)[b + ".g"])) for b in net.bn_names(layout)}


def test_gradcam_against_autograd():
    """Inference-mode Grad-CAM of the full network at every target stage
    against a torch build of the same graph (BN on the running statistics,
    autograd for d logit_k / d A): logits, target activations and their
    gradient, alpha, the map and its trilinear upsampling to the input."""
    torch, g = _torch_graph()
    P, layout = _params("resattnet", 1, 4, 41, stages=(8, 8, 8), stem_c=4)
    running = _running(layout, 42)
    torch, g = _torch_graph(running)
    F = torch.nn.functional
    rng = np.random.default_rng(43)
    x = rng.standard_normal((2, 1, 24, 28, 24))
    classes = np.array([1, 0])
    for target in range(4):
        out = net.gradcam(P, x, classes, running, target, bf16=False)
        TP = _tp(torch, P)
        h = g["stem"](TP, torch.tensor(x), True)
        acts = [h]
        for i in range(3):
            h = g["am"](TP, "s%d.am." % (i + 1),
                        g["ru"](TP, "s%d.ru." % (i + 1), h, 1 if i == 0 else 2))
            acts.append(h)
        acts[target].retain_grad()
        logits = F.linear(h.mean(dim=(2, 3, 4)), TP["fc.w"], TP["fc.b"])
        logits[torch.arange(2), torch.tensor(classes)].sum().backward()
        A, dA = acts[target].detach().numpy(), acts[target].grad.numpy()
        np.testing.assert_allclose(out["logits"], logits.detach().numpy(), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(out["A"], A, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(out["dA"], dA, rtol=1e-8, atol=1e-12)
        alpha = dA.mean(axis=(2, 3, 4))
        cam = np.maximum((alpha[:, :, None, None, None] * A).sum(axis=1), 0.0)
        up = F.interpolate(torch.tensor(cam[:, None]), size=x.shape[2:], mode="trilinear",
                           align_corners=False)[:, 0].numpy()
        np.testing.assert_allclose(out["alpha"], alpha, rtol=1e-8, atol=1e-14)
        np.testing.assert_allclose(out["cam"], cam, rtol=1e-8, atol=1e-14)
        np.testing.assert_allclose(out["up"], up, rtol=1e-8, atol=1e-14)
        assert out["cam"].max() > 0.0


def test_gradcam_last_stage_is_cam():
    """At the last stage the head is an average pool and a linear layer, so
    d logit_k / d A[n, c, v] = fc.w[k, c] / V everywhere: alpha is fc.w[k] / V
    exactly (class activation mapping)."""
    P, layout = _params("resattnet", 1, 4, 44, stages=(8, 8, 8), stem_c=4)
    running = _running(layout, 45)
    rng = np.random.default_rng(46)
    x = rng.standard_normal((2, 1, 24, 28, 24))
    out = net.gradcam(P, x, np.array([0, 1]), running, 3, bf16=False)
    V = np.prod(out["A"].shape[2:])
    np.testing.assert_allclose(out["alpha"], P["fc.w"][[0, 1]] / V, rtol=1e-14)
    # the map is invariant to the class-independent bias and scales with fc.w
    P2 = dict(P, **{"fc.w": 2.0 * P["fc.w"], "fc.b": P["fc.b"] + 5.0})
    out2 = net.gradcam(P2, x, np.array([0, 1]), running, 3, bf16=False)
    np.testing.assert_allclose(out2["cam"], 2.0 * out["cam"], rtol=1e-12)
