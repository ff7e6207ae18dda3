// Composite blocks and the training step: a host-side plan (parameter arena
// and workspace layout) plus an executor that enqueues the kernels of the
// forward pass, the backward pass and the SGD update on the caller's stream.
// The partition's training step over several micro-batches also uses a
// stream of its own: micro-batch k + 1's forward runs there while
// micro-batch k's backward runs on the caller's stream, each micro-batch in
// one of two copies of the activation region (see train_partition).
//
// Graph readings (the paper names conv blocks, residual layers and a
// self-attention layer but leaves their wiring open):
//   residual unit   conv3(s) -> BN -> ReLU -> conv3 -> BN, + skip, ReLU; the
//                   skip is a 1^3 conv (stride s) + BN when channels or
//                   stride change;
//   attention       trunk = RU -> RU; mask = maxpool -> RU -> maxpool -> RU ->
//                   RU -> up -> RU -> up -> 1^3 conv -> BN -> ReLU -> 1^3 conv
//                   (+bias) -> sigmoid; out = (1 + M) * T;
//   stem            7^3 conv stride 2 pad 3 -> BN -> ReLU (-> maxpool);
//   full network    stem+pool, stages of 64/128/256 channels (RU with stride
//                   1/2/2, then attention), global average pool, FC, CE.
// Store points: every activation and activation gradient is stored in the
// network dtype.  Where a tensor feeds several consumers its gradient is
// formed in a fixed order: in a residual unit the skip-branch gradient is
// stored first (added to any gradient already there), then the conv1 input
// gradient is accumulated onto it; in an attention module the mask branch's
// input gradient is stored first and the trunk's is accumulated onto it.
#include <string>
#include <vector>

#include "kernels.hpp"

using namespace rat3d;

namespace {

constexpr int64_t kExtX = -1, kExtY = -2, kExtDx = -3, kExtDy = -4, kNone = -100;

struct Shape {
    int n, c, d, h, w;
    int64_t vox() const { return (int64_t)d * h * w; }
    int64_t count() const { return (int64_t)n * c * d * h * w; }
};

struct TRef {  // activation and its gradient: ws byte offsets or external slots
    int64_t off = kNone, goff = kNone;
    Shape s{};
};

struct ConvL {
    ConvGeom g{};
    size_t w_off = 0, b_off = 0;  // parameter-arena offsets (elements)
    bool bias = false;
    int64_t wt_off[2] = {-1, -1};  // ws bytes: prepared forward / input-gradient weights
};

struct BnL {
    int c = 0;
    size_t g_off = 0, b_off = 0;  // arena offsets of gamma, beta
    int64_t stat_off = 0;         // ws bytes: mean [c], invstd [c], apply scale [c], shift [c]
    size_t run_idx = 0;           // index into the running-statistics regions
};

struct RUPlan {
    ConvL c1, c2, cp;
    BnL b1, b2, bp;
    bool proj = false;
    TRef x, h1, a1, h2, hp, sp, y;
    int64_t dskip = kNone;  // ws offset of the skip-branch gradient
    int64_t ybits = kNone;  // ws offset of the output's y > 0 bits (kNone: read y)
};

struct AMPlan {
    RUPlan t1, t2, m1, m2, m3, m4;
    ConvL c1, c2;
    BnL bn;
    TRef x, p1, p2, u1, h1c, h1, a, z, out;
    int64_t zsum = kNone;  // per-block sums of dz (the c2 bias gradient), or kNone
    int64_t am1 = 0, am2 = 0;  // argmax byte offsets
};

struct ParamRec {
    std::string name;
    size_t off;
    int ndim;
    int shape[5];
};

struct TensorRec {
    std::string name;
    size_t off;
    rat3d_dtype dt;
    int shape[5];
};

}  // namespace

struct rat3d_net {
    rat3d_net_desc d{};
    rat3d_dtype dt = RAT3D_BF16;
    size_t esz = 2;
    std::vector<ParamRec> params;
    std::vector<TensorRec> tensors;
    size_t param_count = 0, ws_bytes = 0;
    // layout
    size_t bn_scr2_off = 0;
    size_t mirror_off = 0, conv_scr_off = 0, conv_scr_bytes = 0, bn_scr_off = 0,
           bn_scr_bytes = 0, head_scr_off = 0, run_mean_off = 0, run_var_off = 0,
           logits_off = 0, loss_off = 0;
    size_t run_count = 0;
    size_t gcam_alpha_off = 0;  // Grad-CAM weights alpha [n][256] (RESATTNET)
    // plan
    TRef stem_h, stem_a, stem_p;
    ConvL stem_conv;
    BnL stem_bn;
    int64_t stem_am = 0;
    std::vector<ConvL> convs;  // every conv layer (weight preparation)
    std::vector<RUPlan> rus;   // RESATTNET: 3 stage units; PARTITION1: 1; RESUNIT: 1
    std::vector<AMPlan> ams;   // RESATTNET: 3; PARTITION1 / ATTN: 1
    ConvL fc;                  // only offsets used (FC weight [2][C], bias [2])
    int fc_c = 0;
    // binding
    float* P = nullptr;
    float* G = nullptr;
    char* ws = nullptr;
    bool reset_running = false;
    // external pointers of the current call
    const void* ext_x = nullptr;
    void* ext_y = nullptr;
    void* ext_dx = nullptr;
    const void* ext_dy = nullptr;
    // PARTITION1 with several micro-batches: a second activation context (the
    // graph region [0, graph_bytes) again at graph_bytes, with its own
    // scratch), the forward stream and the events that order the two
    size_t graph_bytes = 0;
    size_t conv_scr_off1 = 0, bn_scr_off1 = 0, bn_scr2_off1 = 0;
    // scratch of the attention modules' mask branches, per context, when
    // they run on a stream of their own (see am_fwd)
    size_t mask_conv_scr[2] = {0, 0}, mask_bn_scr[2] = {0, 0}, mask_bn_scr2[2] = {0, 0};
    size_t wgrad_conv_scr = 0;  // the weight-gradient stream's (RESATTNET, ATTN)
    bool overlap = true;
    hipStream_t fwd_stream = nullptr;
    // mask-branch streams of the forward and of the backward, with the
    // events that fork and join them
    hipStream_t mask_stream[2] = {nullptr, nullptr};
    hipStream_t wgrad_stream = nullptr;
    hipEvent_t ev_prep = nullptr, ev_fwd[2] = {nullptr, nullptr}, ev_bwd[2] = {nullptr, nullptr};
    hipEvent_t ev_fork[2] = {nullptr, nullptr}, ev_join[2] = {nullptr, nullptr};
    hipEvent_t ev_w_in = nullptr, ev_w_done = nullptr;
    ~rat3d_net() {
        for (hipStream_t s : {fwd_stream, mask_stream[0], mask_stream[1], wgrad_stream})
            if (s) (void)hipStreamDestroy(s);
        for (hipEvent_t e : {ev_prep, ev_fwd[0], ev_fwd[1], ev_bwd[0], ev_bwd[1], ev_fork[0],
                             ev_fork[1], ev_join[0], ev_join[1], ev_w_in, ev_w_done})
            if (e) (void)hipEventDestroy(e);
    }
};

namespace {

// ------------------------------------------------------------------ builder
struct Builder {
    rat3d_net* net;
    size_t top = 0;

    size_t alloc(size_t bytes) {
        top = (top + 255) & ~(size_t)255;
        const size_t off = top;
        top += bytes;
        return off;
    }
    void record(const std::string& name, size_t off, rat3d_dtype dt, Shape s) {
        net->tensors.push_back(TensorRec{name, off, dt, {s.n, s.c, s.d, s.h, s.w}});
    }
    size_t param(const std::string& name, std::initializer_list<int> shape) {
        ParamRec r;
        r.name = name;
        r.off = net->param_count;
        r.ndim = (int)shape.size();
        size_t cnt = 1;
        int i = 0;
        for (int v : shape) {
            r.shape[i++] = v;
            cnt *= (size_t)v;
        }
        for (; i < 5; ++i) r.shape[i] = 1;
        net->params.push_back(r);
        net->param_count += cnt;
        return r.off;
    }
    TRef act(const std::string& name, Shape s, bool grad = true) {
        TRef t;
        t.s = s;
        t.off = (int64_t)alloc((size_t)s.count() * net->esz);
        record(name, (size_t)t.off, net->dt, s);
        if (grad) {
            t.goff = (int64_t)alloc((size_t)s.count() * net->esz);
            record("d:" + name, (size_t)t.goff, net->dt, s);
        }
        return t;
    }
    ConvL conv(const std::string& name, int ci, int co, int k, int s, int p, bool bias,
               Shape in) {
        ConvL c;
        c.g = make_geom(in.n, ci, co, in.d, in.h, in.w, k, s, p);
        c.w_off = param(name + ".w", {co, ci, k, k, k});
        c.bias = bias;
        if (bias) c.b_off = param(name + ".bias", {co});
        size_t need = 0;
        for (int pass = 0; pass < 3; ++pass) {
            const size_t b = conv_ws_bytes(c.g, net->dt, pass);
            if (b > need) need = b;
        }
        if (need > net->conv_scr_bytes) net->conv_scr_bytes = need;
        // weights of the brick passes are prepared once per call (they do
        // not change between micro-batches)
        for (int pass = 0; pass < 2; ++pass)
            if (conv_uses_prepared(c.g, net->dt, pass))
                c.wt_off[pass] = (int64_t)alloc(conv_prepared_bytes(c.g));
        net->convs.push_back(c);
        return c;
    }
    BnL bn(const std::string& name, int c, Shape s) {
        BnL b;
        b.c = c;
        b.g_off = param(name + ".g", {c});
        b.b_off = param(name + ".b", {c});
        b.stat_off = (int64_t)alloc((size_t)4 * c * sizeof(float));
        record(name + ".mean", (size_t)b.stat_off, RAT3D_F32, Shape{1, c, 1, 1, 1});
        record(name + ".invstd", (size_t)b.stat_off + c * sizeof(float), RAT3D_F32,
               Shape{1, c, 1, 1, 1});
        b.run_idx = net->run_count;
        net->run_count += (size_t)c;
        const size_t need = bn_ws_bytes(BnGeom{s.n, c, s.vox()});
        if (need > net->bn_scr_bytes) net->bn_scr_bytes = need;
        return b;
    }

    RUPlan ru(const std::string& pre, TRef x, int cout, int stride) {
        RUPlan r;
        const int cin = x.s.c;
        r.proj = cin != cout || stride != 1;
        r.x = x;
        r.c1 = conv(pre + "conv1", cin, cout, 3, stride, 1, false, x.s);
        const Shape o{x.s.n, cout, r.c1.g.Do, r.c1.g.Ho, r.c1.g.Wo};
        r.b1 = bn(pre + "bn1", cout, o);
        r.c2 = conv(pre + "conv2", cout, cout, 3, 1, 1, false, o);
        r.b2 = bn(pre + "bn2", cout, o);
        if (r.proj) {
            r.cp = conv(pre + "proj", cin, cout, 1, stride, 0, false, x.s);
            r.bp = bn(pre + "projbn", cout, o);
        }
        r.h1 = act(pre + "h1", o);
        r.a1 = act(pre + "a1", o);
        r.h2 = act(pre + "h2", o);
        if (r.proj) {
            r.hp = act(pre + "hp", o);
            r.sp = act(pre + "sp", o, false);
        }
        r.y = act(pre + "y", o);
        // the output BN's ReLU mask, one bit per element
        if (bn_bits_ok(BnGeom{o.n, cout, o.vox()}, net->dt))
            r.ybits = (int64_t)alloc((size_t)(o.count() / 8));
        r.dskip = (int64_t)alloc((size_t)o.count() * net->esz);
        record("d:" + pre + "skip", (size_t)r.dskip, net->dt, o);
        return r;
    }

    AMPlan am(const std::string& pre, TRef x) {
        AMPlan a;
        const int c = x.s.c;
        a.x = x;
        a.t1 = ru(pre + "t1.", x, c, 1);
        a.t2 = ru(pre + "t2.", a.t1.y, c, 1);
        const Shape s1{x.s.n, c, out_dim(x.s.d, 3, 2, 1), out_dim(x.s.h, 3, 2, 1),
                       out_dim(x.s.w, 3, 2, 1)};
        a.p1 = act(pre + "p1", s1);
        a.am1 = (int64_t)alloc((size_t)s1.count());
        record(pre + "p1.argmax", (size_t)a.am1, RAT3D_U8, s1);
        a.m1 = ru(pre + "m1.", a.p1, c, 1);
        const Shape s2{x.s.n, c, out_dim(s1.d, 3, 2, 1), out_dim(s1.h, 3, 2, 1),
                       out_dim(s1.w, 3, 2, 1)};
        a.p2 = act(pre + "p2", s2);
        a.am2 = (int64_t)alloc((size_t)s2.count());
        record(pre + "p2.argmax", (size_t)a.am2, RAT3D_U8, s2);
        a.m2 = ru(pre + "m2.", a.p2, c, 1);
        a.m3 = ru(pre + "m3.", a.m2.y, c, 1);
        a.u1 = act(pre + "u1", s1);
        a.m4 = ru(pre + "m4.", a.u1, c, 1);
        // The first 1^3 conv (no bias) runs before the last upsampling: both
        // are linear, one mixes channels and the other voxels, so
        // conv(up(y)) = up(conv(y)) and the conv and its gradients work on the
        // coarse map.  c1out is the upsampled conv output.
        a.c1 = conv(pre + "c1", c, c, 1, 1, 0, false, s1);
        a.bn = bn(pre + "bn", c, x.s);
        a.c2 = conv(pre + "c2", c, c, 1, 1, 0, true, x.s);
        a.h1c = act(pre + "c1out.coarse", s1);
        a.h1 = act(pre + "c1out", x.s);
        a.a = act(pre + "a", x.s);
        a.z = act(pre + "z", x.s);
        a.out = act(pre + "out", x.s);
        // the soft-mask backward also sums dz per channel when blocks of 2048
        // elements tile the planes (bf16)
        if (net->dt == RAT3D_BF16 && x.s.vox() % 2048 == 0)
            a.zsum = (int64_t)alloc((size_t)c * x.s.n * (x.s.vox() / 2048) * sizeof(float));
        return a;
    }
};

// ------------------------------------------------------------------ executor
struct Exec {
    rat3d_net* n;
    hipStream_t st;
    int acc;  // accumulate parameter gradients (micro-batches after the first)
    // activation context: 0, or 1 for the second copy of the graph region
    // (per-micro-batch tensors, BN statistics, masks and scratch)
    int ctx = 0;
    // the call's input and output gradient (null: the net's)
    const void* x_in = nullptr;
    const void* dy_in = nullptr;
    // side >= 0: the attention modules' mask branches run on
    // n->mask_stream[side] (see am_fwd): the partition's forwards use 0 and
    // its backwards 1, which run at the same time; the full network and the
    // block call use 0.  mask: this Exec is such a branch (its own scratch)
    int side = -1;
    bool mask = false;
    // non-null: weight gradients run on this stream (see conv_w)
    hipStream_t wst = nullptr;

    int64_t shift() const { return ctx ? (int64_t)n->graph_bytes : 0; }
    void* p(int64_t off) const {
        switch (off) {
            case kExtX: return const_cast<void*>(x_in ? x_in : n->ext_x);
            case kExtY: return n->ext_y;
            case kExtDx: return n->ext_dx;
            case kExtDy: return const_cast<void*>(dy_in ? dy_in : n->ext_dy);
            default: return n->ws + off + shift();
        }
    }
    void* a(const TRef& t) const { return p(t.off); }
    void* g(const TRef& t) const { return p(t.goff); }
    const void* w(const ConvL& c) const {
        if (n->dt == RAT3D_BF16) return n->ws + n->mirror_off + c.w_off * 2;
        return n->P + c.w_off;
    }
    float* par(size_t off) const { return n->P + off; }
    float* grd(size_t off) const { return n->G + off; }
    void* conv_scr() const {
        return n->ws + (mask ? n->mask_conv_scr[ctx] : ctx ? n->conv_scr_off1 : n->conv_scr_off);
    }
    void* bn_scr() const {
        return n->ws + (mask ? n->mask_bn_scr[ctx] : ctx ? n->bn_scr_off1 : n->bn_scr_off);
    }
    void* bn_scr2() const {
        return n->ws + (mask ? n->mask_bn_scr2[ctx] : ctx ? n->bn_scr2_off1 : n->bn_scr2_off);
    }
    // The Exec of a mask branch forked off this one's stream: everything
    // enqueued on st so far happens before the branch's first kernel.
    rat3d_status fork(Exec& m) const {
        m = *this;
        m.side = -1;
        m.mask = true;
        m.st = n->mask_stream[side];
        if (hipEventRecord(n->ev_fork[side], st) != hipSuccess ||
            hipStreamWaitEvent(m.st, n->ev_fork[side], 0) != hipSuccess) {
            set_error("rat3d_net: mask-branch stream fork failed");
            return RAT3D_EHIP;
        }
        return RAT3D_OK;
    }
    // st waits for the branch m's kernels.
    rat3d_status join(const Exec& m) const {
        if (hipEventRecord(n->ev_join[side], m.st) != hipSuccess ||
            hipStreamWaitEvent(st, n->ev_join[side], 0) != hipSuccess) {
            set_error("rat3d_net: mask-branch stream join failed");
            return RAT3D_EHIP;
        }
        return RAT3D_OK;
    }
    float* mean(const BnL& b) const { return (float*)(n->ws + b.stat_off + shift()); }
    float* invstd(const BnL& b) const { return mean(b) + b.c; }
    float* fcoef(const BnL& b) const { return mean(b) + 2 * b.c; }
    float* rmean(const BnL& b) const { return (float*)(n->ws + n->run_mean_off) + b.run_idx; }
    float* rvar(const BnL& b) const { return (float*)(n->ws + n->run_var_off) + b.run_idx; }

    const void* wt(const ConvL& c, int pass) const {
        return c.wt_off[pass] >= 0 ? n->ws + c.wt_off[pass] : nullptr;
    }
    rat3d_status conv_f(const ConvL& c, const void* x, void* y) const {
        return conv_fwd_prepared(c.g, n->dt, x, w(c), wt(c, 0), c.bias ? par(c.b_off) : nullptr,
                                 y, conv_scr(), n->conv_scr_bytes, st);
    }
    rat3d_status conv_d(const ConvL& c, const void* dy, void* dx, int accumulate) const {
        return conv_dgrad_prepared(c.g, n->dt, dy, w(c), wt(c, 1), dx, accumulate, conv_scr(),
                                   n->conv_scr_bytes, st);
    }
    // With wst set, a weight gradient runs on wst once everything enqueued on
    // st so far (which produced dy) is done: it reads only x, an activation,
    // and dy, which no later kernel of the backward writes, and writes only
    // its own parameter gradients, so it overlaps the rest of the backward;
    // the caller joins wst (join_wgrad) before anything reads the gradients.
    rat3d_status conv_w(const ConvL& c, const void* x, const void* dy) const {
        float* db = c.bias ? grd(c.b_off) : nullptr;
        if (!wst)
            return conv_wgrad(c.g, n->dt, x, dy, grd(c.w_off), db, acc, conv_scr(),
                              n->conv_scr_bytes, st);
        if (hipEventRecord(n->ev_w_in, st) != hipSuccess ||
            hipStreamWaitEvent(wst, n->ev_w_in, 0) != hipSuccess) {
            set_error("rat3d_net: weight-gradient stream hand-off failed");
            return RAT3D_EHIP;
        }
        return conv_wgrad(c.g, n->dt, x, dy, grd(c.w_off), db, acc, n->ws + n->wgrad_conv_scr,
                          n->conv_scr_bytes, wst);
    }
    // st waits for every weight gradient handed to wst.
    rat3d_status join_wgrad() const {
        if (wst && (hipEventRecord(n->ev_w_done, wst) != hipSuccess ||
                    hipStreamWaitEvent(st, n->ev_w_done, 0) != hipSuccess)) {
            set_error("rat3d_net: weight-gradient stream join failed");
            return RAT3D_EHIP;
        }
        return RAT3D_OK;
    }
    // The forward keeps the apply's scale and shift; a BN + ReLU without a
    // residual recomputes its backward mask from x with them (bn_bwd_x).
    // ybits (nullable): where the forward stores the y > 0 bits of a BN +
    // residual + ReLU, so that its backward reads bits instead of y
    rat3d_status bn_f(const BnL& b, const TRef& x, const void* res, int relu, void* y,
                      uint8_t* ybits = nullptr) const {
        return bn_fwd(BnGeom{x.s.n, b.c, x.s.vox()}, n->dt, relu, n->d.bn_eps, n->d.bn_momentum,
                      a(x), res, par(b.g_off), par(b.b_off), y, mean(b), invstd(b), rmean(b),
                      rvar(b), fcoef(b), ybits, bn_scr(), st);
    }
    // dres_acc: add the residual gradient to dres (one rounding) instead of storing it
    rat3d_status bn_b(const BnL& b, const void* dy, const TRef& x, const void* y, int relu,
                      void* dx, void* dres, int dres_acc = 0,
                      const uint8_t* ybits = nullptr) const {
        return bn_bwd(BnGeom{x.s.n, b.c, x.s.vox()}, n->dt, relu, dy, a(x), y, ybits,
                      par(b.g_off), mean(b), invstd(b), nullptr, dx, dres, dres_acc,
                      grd(b.g_off), grd(b.b_off), acc, bn_scr(), st);
    }
    rat3d_status bn_bwd_x(const BnL& b, const void* dy, const TRef& x, void* dx) const {
        return bn_bwd(BnGeom{x.s.n, b.c, x.s.vox()}, n->dt, 1, dy, a(x), nullptr, nullptr,
                      par(b.g_off), mean(b), invstd(b), fcoef(b), dx, nullptr, 0, grd(b.g_off),
                      grd(b.b_off), acc, bn_scr(), st);
    }
    uint8_t* bits(int64_t off) const {
        return off >= 0 ? (uint8_t*)(n->ws + off + shift()) : nullptr;
    }
};

#define RAT3D_TRY(expr)                       \
    do {                                      \
        rat3d_status s_ = (expr);             \
        if (s_ != RAT3D_OK) return s_;        \
    } while (0)

// With e.side set, a projection skip's 1^3 conv runs on the branch stream
// (it reads only x) while conv1 -> BN -> conv2 run on e.st.
rat3d_status ru_fwd(const Exec& e, const RUPlan& r) {
    Exec k = e;
    const bool fork = r.proj && e.side >= 0;
    if (fork) {
        RAT3D_TRY(e.fork(k));
        RAT3D_TRY(k.conv_f(r.cp, k.a(r.x), k.a(r.hp)));
    }
    RAT3D_TRY(e.conv_f(r.c1, e.a(r.x), e.a(r.h1)));
    RAT3D_TRY(e.bn_f(r.b1, r.h1, nullptr, 1, e.a(r.a1)));
    RAT3D_TRY(e.conv_f(r.c2, e.a(r.a1), e.a(r.h2)));
    const void* skip = e.a(r.x);
    if (r.proj) {
        if (fork) RAT3D_TRY(e.join(k));
        else RAT3D_TRY(e.conv_f(r.cp, e.a(r.x), e.a(r.hp)));
        const BnGeom g{r.h2.s.n, r.b2.c, r.h2.s.vox()};
        if (e.n->dt == RAT3D_BF16 && g.V % 8 == 0) {
            // the projection's BN is applied inside the output BN's apply
            const rat3d_net* n = e.n;
            return bn_fwd_res_bn(g, n->d.bn_eps, n->d.bn_momentum, e.a(r.h2), e.par(r.b2.g_off),
                                 e.par(r.b2.b_off), e.a(r.y), e.mean(r.b2), e.invstd(r.b2),
                                 e.rmean(r.b2), e.rvar(r.b2), e.bits(r.ybits), e.bn_scr(),
                                 e.a(r.hp), e.par(r.bp.g_off), e.par(r.bp.b_off), e.mean(r.bp),
                                 e.invstd(r.bp), e.rmean(r.bp), e.rvar(r.bp), e.bn_scr2(), e.st);
        }
        RAT3D_TRY(e.bn_f(r.bp, r.hp, nullptr, 0, e.a(r.sp)));
        skip = e.a(r.sp);
    }
    return e.bn_f(r.b2, r.h2, skip, 1, e.a(r.y), e.bits(r.ybits));
}

// Backward of a residual unit from y's gradient to x's gradient.  acc_dx: the
// input gradient already holds a partial sum to add to.  With e.side set, a
// projection skip's backward (it needs only the skip gradient) runs on the
// branch stream beside conv2's backward and BN1's; conv1's input gradient,
// added onto the projection's, waits for it.
rat3d_status ru_bwd(const Exec& e, const RUPlan& r, bool acc_dx, bool need_dx = true) {
    void* dskip = e.p(r.dskip);
    void* dx = need_dx ? e.g(r.x) : nullptr;
    // identity skip: the skip gradient goes straight into dx (added to the
    // partial sum already there when acc_dx, one rounding)
    const bool skip_direct = !r.proj && need_dx;
    RAT3D_TRY(e.bn_b(r.b2, e.g(r.y), r.h2, e.a(r.y), 1, e.g(r.h2), skip_direct ? dx : dskip,
                     skip_direct && acc_dx ? 1 : 0, e.bits(r.ybits)));
    auto proj_bwd = [&](const Exec& x) -> rat3d_status {
        RAT3D_TRY(x.bn_b(r.bp, dskip, r.hp, nullptr, 0, x.g(r.hp), nullptr));
        if (need_dx) RAT3D_TRY(x.conv_d(r.cp, x.g(r.hp), dx, acc_dx ? 1 : 0));
        return x.conv_w(r.cp, x.a(r.x), x.g(r.hp));
    };
    Exec k = e;
    const bool fork = r.proj && e.side >= 0;
    if (fork) {
        RAT3D_TRY(e.fork(k));
        RAT3D_TRY(proj_bwd(k));
    }
    RAT3D_TRY(e.conv_d(r.c2, e.g(r.h2), e.g(r.a1), 0));
    RAT3D_TRY(e.conv_w(r.c2, e.a(r.a1), e.g(r.h2)));
    RAT3D_TRY(e.bn_bwd_x(r.b1, e.g(r.a1), r.h1, e.g(r.h1)));
    if (fork) RAT3D_TRY(e.join(k));
    else if (r.proj) RAT3D_TRY(proj_bwd(e));
    if (need_dx) RAT3D_TRY(e.conv_d(r.c1, e.g(r.h1), dx, 1));
    return e.conv_w(r.c1, e.a(r.x), e.g(r.h1));
}

// The mask tail's upsampling and BN run fused when the upsampling is an exact
// x2 of a bf16 map the plane kernels take.
static bool fuse_up_bn(const AMPlan& m, rat3d_dtype dt) {
    const Shape& s = m.x.s;
    const Shape& s1 = m.p1.s;
    return s.d == 2 * s1.d && s.h == 2 * s1.h && s.w == 2 * s1.w &&
           up2_bn_ok(s.n, s.c, s1.d, s1.h, s1.w, dt);
}

// The mask branch of the forward: x -> z (the soft mask before its sigmoid).
static rat3d_status am_mask_fwd(const Exec& e, const AMPlan& m) {
    const Shape& s = m.x.s;
    const rat3d_dtype dt = e.n->dt;
    RAT3D_TRY(pool_fwd(s.n, s.c, s.d, s.h, s.w, 3, 2, 1, dt, e.a(m.x), e.a(m.p1),
                       (uint8_t*)e.p(m.am1), e.st));
    RAT3D_TRY(ru_fwd(e, m.m1));
    const Shape& s1 = m.p1.s;
    RAT3D_TRY(pool_fwd(s.n, s.c, s1.d, s1.h, s1.w, 3, 2, 1, dt, e.a(m.m1.y), e.a(m.p2),
                       (uint8_t*)e.p(m.am2), e.st));
    RAT3D_TRY(ru_fwd(e, m.m2));
    RAT3D_TRY(ru_fwd(e, m.m3));
    const Shape& s2 = m.p2.s;
    RAT3D_TRY(up_fwd(s.n, s.c, s2.d, s2.h, s2.w, s1.d, s1.h, s1.w, dt, e.a(m.m3.y), e.a(m.u1),
                     e.st));
    RAT3D_TRY(ru_fwd(e, m.m4));
    RAT3D_TRY(e.conv_f(m.c1, e.a(m.m4.y), e.a(m.h1c)));
    if (fuse_up_bn(m, dt)) {
        // the x2 upsampling also yields the BN statistics of its output
        RAT3D_TRY(up2_bn_relu_fwd(s.n, s.c, s1.d, s1.h, s1.w, e.a(m.h1c), e.a(m.h1),
                                  e.n->d.bn_eps, e.n->d.bn_momentum, e.par(m.bn.g_off),
                                  e.par(m.bn.b_off), e.a(m.a), e.mean(m.bn), e.invstd(m.bn),
                                  e.rmean(m.bn), e.rvar(m.bn), e.fcoef(m.bn), e.bn_scr(), e.st));
    } else {
        RAT3D_TRY(up_fwd(s.n, s.c, s1.d, s1.h, s1.w, s.d, s.h, s.w, dt, e.a(m.h1c), e.a(m.h1),
                         e.st));
        RAT3D_TRY(e.bn_f(m.bn, m.h1, nullptr, 1, e.a(m.a)));
    }
    return e.conv_f(m.c2, e.a(m.a), e.a(m.z));
}

// The trunk (t1, t2) and the mask branch read only the module input, touch
// disjoint tensors, parameters and running statistics, and meet in the
// soft-mask fuse; with e.side set the mask branch runs on a stream of its own.
rat3d_status am_fwd(const Exec& e, const AMPlan& m) {
    Exec k = e;
    if (e.side >= 0) RAT3D_TRY(e.fork(k));
    RAT3D_TRY(ru_fwd(e, m.t1));
    RAT3D_TRY(ru_fwd(e, m.t2));
    RAT3D_TRY(am_mask_fwd(k, m));
    if (e.side >= 0) RAT3D_TRY(e.join(k));
    // m is not stored: the backward recomputes it from z (same bits)
    return softmask_fwd(m.x.s.count(), e.n->dt, e.a(m.z), e.a(m.t2.y), e.a(m.out), nullptr, e.st);
}

// The mask branch of the backward, from z's gradient (and its per-block sums)
// to x's gradient (stored, not added: the trunk's is added onto it).
static rat3d_status am_mask_bwd(const Exec& e, const AMPlan& m, float* zsum, bool need_dx) {
    const Shape& s = m.x.s;
    const Shape& s1 = m.p1.s;
    const Shape& s2 = m.p2.s;
    const rat3d_dtype dt = e.n->dt;
    RAT3D_TRY(e.conv_d(m.c2, e.g(m.z), e.g(m.a), 0));
    if (zsum) {
        // c2's bias gradient from the soft-mask backward's dz sums
        RAT3D_TRY(conv_wgrad(m.c2.g, dt, e.a(m.a), e.g(m.z), e.grd(m.c2.w_off), nullptr, e.acc,
                             e.conv_scr(), e.n->conv_scr_bytes, e.st));
        RAT3D_TRY(bias_grad_from_partials(zsum, s.c, (int)(s.n * (s.vox() / 2048)),
                                          e.grd(m.c2.b_off), e.acc, e.st));
    } else {
        RAT3D_TRY(e.conv_w(m.c2, e.a(m.a), e.g(m.z)));
    }
    if (fuse_up_bn(m, dt)) {
        // the BN apply happens inside the upsampling transpose: h1's gradient
        // is never stored
        RAT3D_TRY(bn_relu_bwd_up2(s.n, s.c, s1.d, s1.h, s1.w, e.g(m.a), e.a(m.h1),
                                  e.par(m.bn.g_off), e.mean(m.bn), e.invstd(m.bn), e.fcoef(m.bn),
                                  e.grd(m.bn.g_off), e.grd(m.bn.b_off), e.acc, e.bn_scr(),
                                  e.g(m.h1c), e.st));
    } else {
        RAT3D_TRY(e.bn_bwd_x(m.bn, e.g(m.a), m.h1, e.g(m.h1)));
        RAT3D_TRY(up_bwd(s.n, s.c, s1.d, s1.h, s1.w, s.d, s.h, s.w, dt, e.g(m.h1), e.g(m.h1c),
                         0, e.st));
    }
    RAT3D_TRY(e.conv_d(m.c1, e.g(m.h1c), e.g(m.m4.y), 0));
    RAT3D_TRY(e.conv_w(m.c1, e.a(m.m4.y), e.g(m.h1c)));
    RAT3D_TRY(ru_bwd(e, m.m4, false));
    RAT3D_TRY(up_bwd(s.n, s.c, s2.d, s2.h, s2.w, s1.d, s1.h, s1.w, dt, e.g(m.u1), e.g(m.m3.y), 0,
                     e.st));
    RAT3D_TRY(ru_bwd(e, m.m3, false));
    RAT3D_TRY(ru_bwd(e, m.m2, false));
    RAT3D_TRY(pool_bwd(s.n, s.c, s1.d, s1.h, s1.w, 3, 2, 1, dt, e.g(m.p2),
                       (const uint8_t*)e.p(m.am2), e.g(m.m1.y), 0, e.st));
    RAT3D_TRY(ru_bwd(e, m.m1, false));
    if (need_dx)
        RAT3D_TRY(pool_bwd(s.n, s.c, s.d, s.h, s.w, 3, 2, 1, dt, e.g(m.p1),
                           (const uint8_t*)e.p(m.am1), e.g(m.x), 0, e.st));
    return RAT3D_OK;
}

// After the soft-mask backward the mask branch and the trunk's second unit
// are independent (with e.side set the mask branch runs on its own stream);
// the first unit adds its input gradient onto the mask branch's.
rat3d_status am_bwd(const Exec& e, const AMPlan& m, bool need_dx = true) {
    const Shape& s = m.x.s;
    float* zsum = m.zsum >= 0 ? (float*)e.p(m.zsum) : nullptr;
    RAT3D_TRY(softmask_bwd(s.count(), e.n->dt, e.g(m.out), e.a(m.t2.y), e.a(m.z), e.g(m.t2.y), 0,
                           e.g(m.z), e.st, 1, zsum, s.n, s.c, s.vox()));
    Exec k = e;
    if (e.side >= 0) RAT3D_TRY(e.fork(k));
    RAT3D_TRY(am_mask_bwd(k, m, zsum, need_dx));
    RAT3D_TRY(ru_bwd(e, m.t2, false));
    if (e.side >= 0) RAT3D_TRY(e.join(k));
    return ru_bwd(e, m.t1, true, need_dx);
}

rat3d_status stem_fwd(const Exec& e, bool pool) {
    rat3d_net* n = e.n;
    RAT3D_TRY(e.conv_f(n->stem_conv, e.p(kExtX), e.a(n->stem_h)));
    RAT3D_TRY(e.bn_f(n->stem_bn, n->stem_h, nullptr, 1, e.a(n->stem_a)));
    if (!pool) return RAT3D_OK;
    const Shape& s = n->stem_a.s;
    return pool_fwd(s.n, s.c, s.d, s.h, s.w, 3, 2, 1, n->dt, e.a(n->stem_a), e.a(n->stem_p),
                    (uint8_t*)e.p(n->stem_am), e.st);
}

rat3d_status stem_bwd(const Exec& e, bool pool) {
    rat3d_net* n = e.n;
    if (pool) {
        const Shape& s = n->stem_a.s;
        RAT3D_TRY(pool_bwd(s.n, s.c, s.d, s.h, s.w, 3, 2, 1, n->dt, e.g(n->stem_p),
                           (const uint8_t*)e.p(n->stem_am), e.g(n->stem_a), 0, e.st));
    }
    RAT3D_TRY(e.bn_bwd_x(n->stem_bn, e.g(n->stem_a), n->stem_h, e.g(n->stem_h)));
    return e.conv_w(n->stem_conv, e.p(kExtX), e.g(n->stem_h));
}

// ------------------------------------------------------------ inference mode
// The explainable block (Grad-CAM) runs the network in inference mode: every
// BN applies its running statistics, an affine map per channel, so its
// gradient needs no batch sums; no parameter gradient is formed.
rat3d_status bn_eval_f(const Exec& e, const BnL& b, const TRef& x, const void* res, int relu,
                       void* y) {
    return bn_eval_fwd(BnGeom{x.s.n, b.c, x.s.vox()}, e.n->dt, relu, e.n->d.bn_eps, e.a(x), res,
                       e.par(b.g_off), e.par(b.b_off), e.rmean(b), e.rvar(b), y, e.st);
}

// x: the BN's input (for its shape); y: its stored output (the ReLU mask)
rat3d_status bn_eval_b(const Exec& e, const BnL& b, const TRef& x, const void* dy, const void* y,
                       int relu, void* dx, void* dres, int dres_acc) {
    return bn_eval_bwd(BnGeom{x.s.n, b.c, x.s.vox()}, e.n->dt, relu, e.n->d.bn_eps, dy, y,
                       e.par(b.g_off), e.rvar(b), dx, dres, dres_acc, e.st);
}

rat3d_status ru_fwd_eval(const Exec& e, const RUPlan& r) {
    RAT3D_TRY(e.conv_f(r.c1, e.a(r.x), e.a(r.h1)));
    RAT3D_TRY(bn_eval_f(e, r.b1, r.h1, nullptr, 1, e.a(r.a1)));
    RAT3D_TRY(e.conv_f(r.c2, e.a(r.a1), e.a(r.h2)));
    const void* skip = e.a(r.x);
    if (r.proj) {
        RAT3D_TRY(e.conv_f(r.cp, e.a(r.x), e.a(r.hp)));
        RAT3D_TRY(bn_eval_f(e, r.bp, r.hp, nullptr, 0, e.a(r.sp)));
        skip = e.a(r.sp);
    }
    return bn_eval_f(e, r.b2, r.h2, skip, 1, e.a(r.y));
}

// Input gradient of a residual unit in inference mode (acc_dx: add onto the
// partial sum already in x's gradient); the same join order as training.
rat3d_status ru_bwd_eval(const Exec& e, const RUPlan& r, bool acc_dx) {
    void* dx = e.g(r.x);
    void* dskip = e.p(r.dskip);
    RAT3D_TRY(bn_eval_b(e, r.b2, r.h2, e.g(r.y), e.a(r.y), 1, e.g(r.h2), r.proj ? dskip : dx,
                        !r.proj && acc_dx ? 1 : 0));
    RAT3D_TRY(e.conv_d(r.c2, e.g(r.h2), e.g(r.a1), 0));
    RAT3D_TRY(bn_eval_b(e, r.b1, r.h1, e.g(r.a1), e.a(r.a1), 1, e.g(r.h1), nullptr, 0));
    if (r.proj) {
        RAT3D_TRY(bn_eval_b(e, r.bp, r.hp, dskip, nullptr, 0, e.g(r.hp), nullptr, 0));
        RAT3D_TRY(e.conv_d(r.cp, e.g(r.hp), dx, acc_dx ? 1 : 0));
    }
    return e.conv_d(r.c1, e.g(r.h1), dx, 1);
}

rat3d_status am_fwd_eval(const Exec& e, const AMPlan& m) {
    const Shape& s = m.x.s;
    const Shape& s1 = m.p1.s;
    const Shape& s2 = m.p2.s;
    const rat3d_dtype dt = e.n->dt;
    RAT3D_TRY(ru_fwd_eval(e, m.t1));
    RAT3D_TRY(ru_fwd_eval(e, m.t2));
    RAT3D_TRY(pool_fwd(s.n, s.c, s.d, s.h, s.w, 3, 2, 1, dt, e.a(m.x), e.a(m.p1),
                       (uint8_t*)e.p(m.am1), e.st));
    RAT3D_TRY(ru_fwd_eval(e, m.m1));
    RAT3D_TRY(pool_fwd(s.n, s.c, s1.d, s1.h, s1.w, 3, 2, 1, dt, e.a(m.m1.y), e.a(m.p2),
                       (uint8_t*)e.p(m.am2), e.st));
    RAT3D_TRY(ru_fwd_eval(e, m.m2));
    RAT3D_TRY(ru_fwd_eval(e, m.m3));
    RAT3D_TRY(up_fwd(s.n, s.c, s2.d, s2.h, s2.w, s1.d, s1.h, s1.w, dt, e.a(m.m3.y), e.a(m.u1),
                     e.st));
    RAT3D_TRY(ru_fwd_eval(e, m.m4));
    RAT3D_TRY(e.conv_f(m.c1, e.a(m.m4.y), e.a(m.h1c)));
    RAT3D_TRY(up_fwd(s.n, s.c, s1.d, s1.h, s1.w, s.d, s.h, s.w, dt, e.a(m.h1c), e.a(m.h1),
                     e.st));
    RAT3D_TRY(bn_eval_f(e, m.bn, m.h1, nullptr, 1, e.a(m.a)));
    RAT3D_TRY(e.conv_f(m.c2, e.a(m.a), e.a(m.z)));
    return softmask_fwd(s.count(), dt, e.a(m.z), e.a(m.t2.y), e.a(m.out), nullptr, e.st);
}

rat3d_status am_bwd_eval(const Exec& e, const AMPlan& m) {
    const Shape& s = m.x.s;
    const Shape& s1 = m.p1.s;
    const Shape& s2 = m.p2.s;
    const rat3d_dtype dt = e.n->dt;
    RAT3D_TRY(softmask_bwd(s.count(), dt, e.g(m.out), e.a(m.t2.y), e.a(m.z), e.g(m.t2.y), 0,
                           e.g(m.z), e.st, 1));
    RAT3D_TRY(e.conv_d(m.c2, e.g(m.z), e.g(m.a), 0));
    RAT3D_TRY(bn_eval_b(e, m.bn, m.h1, e.g(m.a), e.a(m.a), 1, e.g(m.h1), nullptr, 0));
    RAT3D_TRY(up_bwd(s.n, s.c, s1.d, s1.h, s1.w, s.d, s.h, s.w, dt, e.g(m.h1), e.g(m.h1c), 0,
                     e.st));
    RAT3D_TRY(e.conv_d(m.c1, e.g(m.h1c), e.g(m.m4.y), 0));
    RAT3D_TRY(ru_bwd_eval(e, m.m4, false));
    RAT3D_TRY(up_bwd(s.n, s.c, s2.d, s2.h, s2.w, s1.d, s1.h, s1.w, dt, e.g(m.u1), e.g(m.m3.y), 0,
                     e.st));
    RAT3D_TRY(ru_bwd_eval(e, m.m3, false));
    RAT3D_TRY(ru_bwd_eval(e, m.m2, false));
    RAT3D_TRY(pool_bwd(s.n, s.c, s1.d, s1.h, s1.w, 3, 2, 1, dt, e.g(m.p2),
                       (const uint8_t*)e.p(m.am2), e.g(m.m1.y), 0, e.st));
    RAT3D_TRY(ru_bwd_eval(e, m.m1, false));
    RAT3D_TRY(pool_bwd(s.n, s.c, s.d, s.h, s.w, 3, 2, 1, dt, e.g(m.p1),
                       (const uint8_t*)e.p(m.am1), e.g(m.x), 0, e.st));
    RAT3D_TRY(ru_bwd_eval(e, m.t2, false));
    return ru_bwd_eval(e, m.t1, true);
}

rat3d_status stem_fwd_eval(const Exec& e) {
    rat3d_net* n = e.n;
    RAT3D_TRY(e.conv_f(n->stem_conv, n->ext_x, e.a(n->stem_h)));
    RAT3D_TRY(bn_eval_f(e, n->stem_bn, n->stem_h, nullptr, 1, e.a(n->stem_a)));
    const Shape& s = n->stem_a.s;
    return pool_fwd(s.n, s.c, s.d, s.h, s.w, 3, 2, 1, n->dt, e.a(n->stem_a), e.a(n->stem_p),
                    (uint8_t*)e.p(n->stem_am), e.st);
}

// The map Grad-CAM weights: the stem's pooled output (target 0) or a stage's
// attention-module output (targets 1-3).
const TRef& gradcam_target(const rat3d_net* n, int target) {
    return target == 0 ? n->stem_p : n->ams[target - 1].out;
}

rat3d_status prepare_call(rat3d_net* n, hipStream_t st) {
    if (!n->P || !n->G || !n->ws) {
        set_error("rat3d_net: buffers not bound (call rat3d_net_bind first)");
        return RAT3D_EINVAL;
    }
    if (n->reset_running) {
        RAT3D_TRY(fill_f32((int64_t)n->run_count, 0.f, (float*)(n->ws + n->run_mean_off), st));
        RAT3D_TRY(fill_f32((int64_t)n->run_count, 1.f, (float*)(n->ws + n->run_var_off), st));
        n->reset_running = false;
    }
    if (n->dt == RAT3D_BF16)
        RAT3D_TRY(cast_f32_bf16((int64_t)n->param_count, n->P, (bf16*)(n->ws + n->mirror_off), st));
    // every conv's prepared weight layouts, a few launches in all
    std::vector<PrepJob> jobs;
    for (const ConvL& c : n->convs) {
        const void* w = n->dt == RAT3D_BF16 ? (const void*)(n->ws + n->mirror_off + c.w_off * 2)
                                            : (const void*)(n->P + c.w_off);
        for (int pass = 0; pass < 2; ++pass)
            if (c.wt_off[pass] >= 0) jobs.push_back(PrepJob{c.g, pass == 1, w, n->ws + c.wt_off[pass]});
    }
    return jobs.empty() ? RAT3D_OK : brick_prep_weights_batch(jobs.data(), (int)jobs.size(), st);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// One micro-batch of the first-stage partition: forward from x, backward from
// the gradient received at the partition's output (it arrives from the next
// partition); parameter gradients are written (acc = 0) or added (acc = 1).
// The weights must be prepared.
rat3d_status partition_fwd(const Exec& e) {
    rat3d_net* net = e.n;
    RAT3D_TRY(stem_fwd(e, false));
    RAT3D_TRY(ru_fwd(e, net->rus[0]));
    return am_fwd(e, net->ams[0]);
}
rat3d_status partition_bwd(const Exec& e) {
    rat3d_net* net = e.n;
    RAT3D_TRY(am_bwd(e, net->ams[0]));
    RAT3D_TRY(ru_bwd(e, net->rus[0], false));
    return stem_bwd(e, false);
}
rat3d_status partition_micro_batch(rat3d_net* net, const void* x, const void* dy, int acc,
                                   hipStream_t st) {
    Exec e{net, st, acc};
    e.x_in = x;
    e.dy_in = dy;
    RAT3D_TRY(partition_fwd(e));
    return partition_bwd(e);
}

bool hip_ok(hipError_t r, const char* what) {
    if (r == hipSuccess) return true;
    set_error("rat3d_train_step: %s failed (%s)", what, hipGetErrorString(r));
    return false;
}

// The partition's step over M micro-batches.  Micro-batch k runs in context
// (M - 1 - k) % 2 (the last one in context 0, whose tensors
// rat3d_net_tensor_info describes); its forward is enqueued on the net's
// forward stream and its backward on the caller's stream st:
//   forward k      waits for the weight preparation (k = 0) and for the
//                  backward of micro-batch k - 2 (the same context);
//   backward k     waits for forward k and follows backward k - 1 on st.
// So micro-batch k + 1's forward runs while micro-batch k's backward does.
// Each of the two also runs its attention module's mask branch on a stream of
// its own (am_fwd, am_bwd).
// The two share only read-only data (weights, the prepared layouts) and the
// BN running statistics, which only the forwards update, in order; parameter
// gradients are formed by the backwards alone, in order.  Every forward is
// done before the last backward starts, so the caller's stream covers the
// whole step.
rat3d_status train_partition(rat3d_net* net, const char* x, const char* dy, size_t x_bytes,
                             size_t dy_bytes, hipStream_t st) {
    const int M = net->d.micro_batches;
    // under stream capture the micro-batches are enqueued one after another:
    // capturing the two-stream form ended in a crash inside the runtime's end
    // of capture, with every fork joined back within this call
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (!hip_ok(hipStreamIsCapturing(st, &cap), "capture query")) return RAT3D_EHIP;
    if (!net->fwd_stream || !net->overlap || M < 2 || cap != hipStreamCaptureStatusNone) {
        for (int k = 0; k < M; ++k)
            RAT3D_TRY(partition_micro_batch(net, x + k * x_bytes, dy + k * dy_bytes, k > 0 ? 1 : 0,
                                            st));
        return RAT3D_OK;
    }
    hipStream_t fs = net->fwd_stream;
    if (!hip_ok(hipEventRecord(net->ev_prep, st), "event record") ||
        !hip_ok(hipStreamWaitEvent(fs, net->ev_prep, 0), "stream wait"))
        return RAT3D_EHIP;
    for (int k = 0; k < M; ++k) {
        const int c = (M - 1 - k) % 2;
        Exec f{net, fs, 0};
        f.ctx = c;
        f.side = 0;
        f.x_in = x + k * x_bytes;
        if (k >= 2 && !hip_ok(hipStreamWaitEvent(fs, net->ev_bwd[c], 0), "stream wait"))
            return RAT3D_EHIP;
        RAT3D_TRY(partition_fwd(f));
        if (!hip_ok(hipEventRecord(net->ev_fwd[c], fs), "event record") ||
            !hip_ok(hipStreamWaitEvent(st, net->ev_fwd[c], 0), "stream wait"))
            return RAT3D_EHIP;
        Exec b{net, st, k > 0 ? 1 : 0};
        b.ctx = c;
        b.side = 1;
        b.x_in = f.x_in;
        b.dy_in = dy + k * dy_bytes;
        RAT3D_TRY(partition_bwd(b));
        if (!hip_ok(hipEventRecord(net->ev_bwd[c], st), "event record")) return RAT3D_EHIP;
    }
    return RAT3D_OK;
}

}  // namespace

extern "C" {

rat3d_status rat3d_net_create(const rat3d_net_desc* desc, rat3d_net** out) {
    if (!desc || !out) {
        set_error("rat3d_net_create: NULL argument");
        return RAT3D_EINVAL;
    }
    *out = nullptr;
    const rat3d_net_desc& d = *desc;
    if (d.dtype != RAT3D_F32 && d.dtype != RAT3D_BF16) {
        set_error("rat3d_net_create: unsupported dtype");
        return RAT3D_EUNSUPPORTED;
    }
    if (d.n < 1 || d.d < 1 || d.h < 1 || d.w < 1 || d.bn_eps <= 0.f || d.bn_momentum < 0.f ||
        d.bn_momentum > 1.f) {
        set_error("rat3d_net_create: invalid sizes or BN settings");
        return RAT3D_EINVAL;
    }
    const int mb = d.micro_batches < 1 ? 1 : d.micro_batches;
    if (mb != 1 && d.kind != RAT3D_NET_PARTITION1) {
        set_error("rat3d_net_create: micro_batches > 1 only for PARTITION1");
        return RAT3D_EINVAL;
    }
    rat3d_net* n = new rat3d_net();
    n->d = d;
    n->d.micro_batches = mb;
    n->dt = d.dtype;
    n->esz = d.dtype == RAT3D_BF16 ? 2 : 4;
    Builder b{n};
    const Shape in{d.n, d.c_in, d.d, d.h, d.w};
    TRef x;
    x.off = kExtX;
    x.goff = kExtDx;
    x.s = in;
    switch (d.kind) {
        case RAT3D_NET_RESUNIT: {
            if (d.c_in < 1 || d.c < 1) break;
            RUPlan r = b.ru("", x, d.c, 1);
            r.y.off = kExtY;
            r.y.goff = kExtDy;
            n->rus.push_back(r);
            break;
        }
        case RAT3D_NET_ATTN: {
            if (d.c < 1 || d.c_in != d.c) break;
            AMPlan m = b.am("", x);
            m.out.off = kExtY;
            m.out.goff = kExtDy;
            n->ams.push_back(m);
            break;
        }
        case RAT3D_NET_RESATTNET:
        case RAT3D_NET_PARTITION1: {
            if (d.c_in != 1) break;
            const bool full = d.kind == RAT3D_NET_RESATTNET;
            if (!full && d.c < 1) break;
            n->stem_conv = b.conv("stem", 1, 32, 7, 2, 3, false, in);
            const ConvGeom& g = n->stem_conv.g;
            const Shape so{d.n, 32, g.Do, g.Ho, g.Wo};
            n->stem_bn = b.bn("stem.bn", 32, so);
            n->stem_h = b.act("stem.h", so);
            n->stem_a = b.act("stem.a", so);
            TRef h = n->stem_a;
            if (full) {
                const Shape sp{d.n, 32, out_dim(so.d, 3, 2, 1), out_dim(so.h, 3, 2, 1),
                               out_dim(so.w, 3, 2, 1)};
                n->stem_p = b.act("stem.p", sp);
                n->stem_am = (int64_t)b.alloc((size_t)sp.count());
                b.record("stem.p.argmax", (size_t)n->stem_am, RAT3D_U8, sp);
                h = n->stem_p;
                const int stages[3] = {64, 128, 256};
                for (int i = 0; i < 3; ++i) {
                    const std::string pre = "s" + std::to_string(i + 1) + ".";
                    n->rus.push_back(b.ru(pre + "ru.", h, stages[i], i == 0 ? 1 : 2));
                    n->ams.push_back(b.am(pre + "am.", n->rus.back().y));
                    h = n->ams.back().out;
                }
                n->fc_c = 256;
                n->fc.w_off = b.param("fc.w", {2, 256});
                n->fc.b_off = b.param("fc.b", {2});
            } else {
                n->rus.push_back(b.ru("ru.", h, d.c, 1));
                n->ams.push_back(b.am("am.", n->rus.back().y));
                // the output gradient is read straight from the caller's buffer
                n->ams.back().out.goff = kExtDy;
            }
            break;
        }
        default:
            break;
    }
    if (n->params.empty()) {
        delete n;
        set_error("rat3d_net_create: invalid kind or channel counts");
        return RAT3D_EINVAL;
    }
    // the partition's second activation context: the graph region again
    n->graph_bytes = (b.top + 255) & ~(size_t)255;
    const bool two_ctx = d.kind == RAT3D_NET_PARTITION1 && mb > 1;
    if (two_ctx) b.top = 2 * n->graph_bytes;
    // fixed regions
    if (n->dt == RAT3D_BF16) n->mirror_off = b.alloc(n->param_count * 2);
    n->conv_scr_off = b.alloc(n->conv_scr_bytes);
    n->bn_scr_off = b.alloc(n->bn_scr_bytes);
    n->bn_scr2_off = b.alloc(n->bn_scr_bytes);  // a second BN's partials (projection skip)
    if (two_ctx) {
        n->conv_scr_off1 = b.alloc(n->conv_scr_bytes);
        n->bn_scr_off1 = b.alloc(n->bn_scr_bytes);
        n->bn_scr2_off1 = b.alloc(n->bn_scr_bytes);
    }
    // mask-branch scratch: the partition's two contexts, the full network's one
    const int mask_ctx =
        two_ctx ? 2 : d.kind == RAT3D_NET_RESATTNET || d.kind == RAT3D_NET_ATTN ? 1 : 0;
    for (int c = 0; c < mask_ctx; ++c) {
        n->mask_conv_scr[c] = b.alloc(n->conv_scr_bytes);
        n->mask_bn_scr[c] = b.alloc(n->bn_scr_bytes);
        n->mask_bn_scr2[c] = b.alloc(n->bn_scr_bytes);
    }
    if (!two_ctx && mask_ctx) n->wgrad_conv_scr = b.alloc(n->conv_scr_bytes);
    n->head_scr_off = b.alloc(head_ws_bytes(d.n, 256, 2));
    n->run_mean_off = b.alloc(n->run_count * sizeof(float));
    n->run_var_off = b.alloc(n->run_count * sizeof(float));
    if (d.kind == RAT3D_NET_RESATTNET)
        n->gcam_alpha_off = b.alloc((size_t)d.n * 256 * sizeof(float));
    n->logits_off = b.alloc((size_t)d.n * 2 * sizeof(float));
    n->loss_off = b.alloc(sizeof(float));
    b.record("logits", n->logits_off, RAT3D_F32, Shape{d.n, 2, 1, 1, 1});
    b.record("loss", n->loss_off, RAT3D_F32, Shape{1, 1, 1, 1, 1});
    b.record("running_mean", n->run_mean_off, RAT3D_F32, Shape{1, (int)n->run_count, 1, 1, 1});
    b.record("running_var", n->run_var_off, RAT3D_F32, Shape{1, (int)n->run_count, 1, 1, 1});
    n->ws_bytes = (b.top + 255) & ~(size_t)255;
    *out = n;
    return RAT3D_OK;
}

void rat3d_net_destroy(rat3d_net* net) { delete net; }

size_t rat3d_net_param_count(const rat3d_net* net) { return net ? net->param_count : 0; }

size_t rat3d_net_workspace_size(const rat3d_net* net) { return net ? net->ws_bytes : 0; }

int rat3d_net_num_params(const rat3d_net* net) { return net ? (int)net->params.size() : 0; }

rat3d_status rat3d_net_param_info(const rat3d_net* net, int i, const char** name,
                                  size_t* offset, int* ndim, int shape[5]) {
    if (!net || i < 0 || i >= (int)net->params.size()) {
        set_error("rat3d_net_param_info: index out of range");
        return RAT3D_EINVAL;
    }
    const ParamRec& r = net->params[i];
    if (name) *name = r.name.c_str();
    if (offset) *offset = r.off;
    if (ndim) *ndim = r.ndim;
    if (shape)
        for (int k = 0; k < 5; ++k) shape[k] = r.shape[k];
    return RAT3D_OK;
}

int rat3d_net_num_tensors(const rat3d_net* net) { return net ? (int)net->tensors.size() : 0; }

rat3d_status rat3d_net_tensor_info(const rat3d_net* net, int i, const char** name,
                                   size_t* byte_offset, rat3d_dtype* dtype, int shape[5]) {
    if (!net || i < 0 || i >= (int)net->tensors.size()) {
        set_error("rat3d_net_tensor_info: index out of range");
        return RAT3D_EINVAL;
    }
    const TensorRec& r = net->tensors[i];
    if (name) *name = r.name.c_str();
    if (byte_offset) *byte_offset = r.off;
    if (dtype) *dtype = r.dt;
    if (shape)
        for (int k = 0; k < 5; ++k) shape[k] = r.shape[k];
    return RAT3D_OK;
}

rat3d_status rat3d_net_bind(rat3d_net* net, float* params, float* grads, void* ws,
                            size_t ws_bytes) {
    if (!net || !params || !grads || !ws) {
        set_error("rat3d_net_bind: NULL argument");
        return RAT3D_EINVAL;
    }
    if (ws_bytes < net->ws_bytes) {
        set_error("rat3d_net_bind: workspace needs %zu bytes, got %zu", net->ws_bytes, ws_bytes);
        return RAT3D_EWORKSPACE;
    }
    if (!aligned16(params) || !aligned16(grads) || ((uintptr_t)ws & 255u) != 0) {
        set_error("rat3d_net_bind: arenas must be 16-byte and the workspace 256-byte aligned");
        return RAT3D_EALIGN;
    }
    if (net->mask_conv_scr[0] && !net->mask_stream[0]) {
        // the partition's forward stream, the mask-branch streams (default
        // priority) and their events
        hipError_t r = hipSuccess;
        if (net->conv_scr_off1) r = hipStreamCreateWithFlags(&net->fwd_stream, hipStreamNonBlocking);
        for (hipStream_t* s : {&net->mask_stream[0], &net->mask_stream[1]})
            if (r == hipSuccess) r = hipStreamCreateWithFlags(s, hipStreamNonBlocking);
        if (r == hipSuccess && net->wgrad_conv_scr)
            r = hipStreamCreateWithFlags(&net->wgrad_stream, hipStreamNonBlocking);
        for (hipEvent_t* e : {&net->ev_prep, &net->ev_fwd[0], &net->ev_fwd[1], &net->ev_bwd[0],
                              &net->ev_bwd[1], &net->ev_fork[0], &net->ev_fork[1],
                              &net->ev_join[0], &net->ev_join[1], &net->ev_w_in, &net->ev_w_done})
            if (r == hipSuccess) r = hipEventCreateWithFlags(e, hipEventDisableTiming);
        if (r != hipSuccess) {
            set_error("rat3d_net_bind: stream or event creation failed (%s)",
                      hipGetErrorString(r));
            return RAT3D_EHIP;
        }
    }
    net->P = params;
    net->G = grads;
    net->ws = (char*)ws;
    net->reset_running = true;
    return RAT3D_OK;
}

rat3d_status rat3d_net_set_overlap(rat3d_net* net, int enable) {
    if (!net) {
        set_error("rat3d_net_set_overlap: NULL network");
        return RAT3D_EINVAL;
    }
    net->overlap = enable != 0;
    return RAT3D_OK;
}

rat3d_status rat3d_block_fwd_bwd(rat3d_net* net, const void* x, const void* dy, void* y,
                                 void* dx, void* stream) {
    if (!net || (net->d.kind != RAT3D_NET_RESUNIT && net->d.kind != RAT3D_NET_ATTN)) {
        set_error("rat3d_block_fwd_bwd: needs a RESUNIT or ATTN network");
        return RAT3D_EINVAL;
    }
    if (!x || !dy || !y || !dx) {
        set_error("rat3d_block_fwd_bwd: NULL tensor");
        return RAT3D_EINVAL;
    }
    if (!aligned16(x) || !aligned16(dy) || !aligned16(y) || !aligned16(dx)) {
        set_error("rat3d_block_fwd_bwd: tensors must be 16-byte aligned");
        return RAT3D_EALIGN;
    }
    hipStream_t st = (hipStream_t)stream;
    RAT3D_TRY(prepare_call(net, st));
    net->ext_x = x;
    net->ext_dy = dy;
    net->ext_y = y;
    net->ext_dx = dx;
    Exec e{net, st, 0};
    if (net->d.kind == RAT3D_NET_RESUNIT) {
        RAT3D_TRY(ru_fwd(e, net->rus[0]));
        return ru_bwd(e, net->rus[0], false);
    }
    // the mask branch and the weight gradients on streams of their own
    if (net->overlap && net->mask_stream[0]) {
        e.side = 0;
        e.wst = net->wgrad_stream;
    }
    RAT3D_TRY(am_fwd(e, net->ams[0]));
    RAT3D_TRY(am_bwd(e, net->ams[0]));
    return e.join_wgrad();
}

rat3d_status rat3d_train_step(rat3d_net* net, const void* x, const int32_t* labels,
                              const void* dy_upstream, float* loss_dev, void* stream) {
    if (!net || (net->d.kind != RAT3D_NET_RESATTNET && net->d.kind != RAT3D_NET_PARTITION1)) {
        set_error("rat3d_train_step: needs a RESATTNET or PARTITION1 network");
        return RAT3D_EINVAL;
    }
    const bool full = net->d.kind == RAT3D_NET_RESATTNET;
    if (!x || (full && !labels) || (!full && !dy_upstream)) {
        set_error("rat3d_train_step: NULL input");
        return RAT3D_EINVAL;
    }
    if (!aligned16(x) || (dy_upstream && !aligned16(dy_upstream))) {
        set_error("rat3d_train_step: tensors must be 16-byte aligned");
        return RAT3D_EALIGN;
    }
    hipStream_t st = (hipStream_t)stream;
    RAT3D_TRY(prepare_call(net, st));
    const rat3d_net_desc& d = net->d;
    const size_t x_bytes = (size_t)d.n * d.d * d.h * d.w * net->esz;
    if (full) {
        net->ext_x = x;
        Exec e{net, st, 0};
        // the attention modules' mask branches and the weight gradients on
        // streams of their own
        if (net->overlap && net->mask_stream[0]) {
            e.side = 0;
            e.wst = net->wgrad_stream;
        }
        RAT3D_TRY(stem_fwd(e, true));
        for (int i = 0; i < 3; ++i) {
            RAT3D_TRY(ru_fwd(e, net->rus[i]));
            RAT3D_TRY(am_fwd(e, net->ams[i]));
        }
        const TRef& top = net->ams[2].out;
        RAT3D_TRY(head_fwd_bwd(d.n, net->fc_c, top.s.vox(), 2, net->dt, e.a(top),
                               e.par(net->fc.w_off), e.par(net->fc.b_off), labels,
                               (float*)(net->ws + net->logits_off),
                               (float*)(net->ws + net->loss_off), e.g(top), e.grd(net->fc.w_off),
                               e.grd(net->fc.b_off), 0, net->ws + net->head_scr_off, st));
        for (int i = 2; i >= 0; --i) {
            RAT3D_TRY(am_bwd(e, net->ams[i]));
            RAT3D_TRY(ru_bwd(e, net->rus[i], false));
        }
        RAT3D_TRY(stem_bwd(e, true));
        RAT3D_TRY(e.join_wgrad());
        if (loss_dev) {
            if (hipMemcpyAsync(loss_dev, net->ws + net->loss_off, sizeof(float),
                               hipMemcpyDeviceToDevice, st) != hipSuccess) {
                set_error("rat3d_train_step: loss copy failed");
                return RAT3D_EHIP;
            }
        }
    } else {
        const size_t dy_bytes = (size_t)net->ams[0].out.s.count() * net->esz;
        RAT3D_TRY(train_partition(net, (const char*)x, (const char*)dy_upstream, x_bytes,
                                  dy_bytes, st));
    }
    return sgd_update((int64_t)net->param_count, d.lr, net->P, net->G, st);
}

rat3d_status rat3d_partition_micro_batch(rat3d_net* net, const void* x, const void* dy_upstream,
                                         int accumulate, void* stream) {
    if (!net || net->d.kind != RAT3D_NET_PARTITION1) {
        set_error("rat3d_partition_micro_batch: needs a PARTITION1 network");
        return RAT3D_EINVAL;
    }
    if (!x || !dy_upstream) {
        set_error("rat3d_partition_micro_batch: NULL input");
        return RAT3D_EINVAL;
    }
    if (!aligned16(x) || !aligned16(dy_upstream)) {
        set_error("rat3d_partition_micro_batch: tensors must be 16-byte aligned");
        return RAT3D_EALIGN;
    }
    hipStream_t st = (hipStream_t)stream;
    RAT3D_TRY(prepare_call(net, st));
    return partition_micro_batch(net, x, dy_upstream, accumulate ? 1 : 0, st);
}

rat3d_status rat3d_net_update(rat3d_net* net, void* stream) {
    if (!net || !net->P || !net->G) {
        set_error("rat3d_net_update: network missing or not bound");
        return RAT3D_EINVAL;
    }
    return sgd_update((int64_t)net->param_count, net->d.lr, net->P, net->G, (hipStream_t)stream);
}

size_t rat3d_net_running_count(const rat3d_net* net) { return net ? net->run_count : 0; }

rat3d_status rat3d_net_running_save(const rat3d_net* net, float* dst, void* stream) {
    if (!net || !net->ws || !dst) {
        set_error("rat3d_net_running_save: network not bound or NULL destination");
        return RAT3D_EINVAL;
    }
    if (net->reset_running) {
        set_error("rat3d_net_running_save: no step has run since the buffers were bound");
        return RAT3D_EINVAL;
    }
    hipStream_t st = (hipStream_t)stream;
    const size_t bytes = net->run_count * sizeof(float);
    if (hipMemcpyAsync(dst, net->ws + net->run_mean_off, bytes, hipMemcpyDeviceToDevice, st) !=
            hipSuccess ||
        hipMemcpyAsync(dst + net->run_count, net->ws + net->run_var_off, bytes,
                       hipMemcpyDeviceToDevice, st) != hipSuccess) {
        set_error("rat3d_net_running_save: copy failed");
        return RAT3D_EHIP;
    }
    return RAT3D_OK;
}

rat3d_status rat3d_net_running_load(rat3d_net* net, const float* src, void* stream) {
    if (!net || !net->ws || !src) {
        set_error("rat3d_net_running_load: network not bound or NULL source");
        return RAT3D_EINVAL;
    }
    hipStream_t st = (hipStream_t)stream;
    const size_t bytes = net->run_count * sizeof(float);
    if (hipMemcpyAsync(net->ws + net->run_mean_off, src, bytes, hipMemcpyDeviceToDevice, st) !=
            hipSuccess ||
        hipMemcpyAsync(net->ws + net->run_var_off, src + net->run_count, bytes,
                       hipMemcpyDeviceToDevice, st) != hipSuccess) {
        set_error("rat3d_net_running_load: copy failed");
        return RAT3D_EHIP;
    }
    net->reset_running = false;  // the loaded statistics replace the bind-time reset
    return RAT3D_OK;
}

rat3d_status rat3d_gradcam_shape(const rat3d_net* net, int target, int shape[4]) {
    if (!net || net->d.kind != RAT3D_NET_RESATTNET || target < 0 || target > 3 || !shape) {
        set_error("rat3d_gradcam_shape: needs a RESATTNET network and 0 <= target <= 3");
        return RAT3D_EINVAL;
    }
    const Shape& t = gradcam_target(net, target).s;
    shape[0] = t.c;
    shape[1] = t.d;
    shape[2] = t.h;
    shape[3] = t.w;
    return RAT3D_OK;
}

rat3d_status rat3d_gradcam(rat3d_net* net, const void* x, const int32_t* classes, int target,
                           float* logits, float* cam, float* cam_up, void* stream) {
    if (!net || net->d.kind != RAT3D_NET_RESATTNET) {
        set_error("rat3d_gradcam: needs a RESATTNET network");
        return RAT3D_EINVAL;
    }
    if (!x || !classes || !cam || target < 0 || target > 3) {
        set_error("rat3d_gradcam: x, classes and cam must be non-NULL and 0 <= target <= 3");
        return RAT3D_EINVAL;
    }
    if (!aligned16(x)) {
        set_error("rat3d_gradcam: x must be 16-byte aligned");
        return RAT3D_EALIGN;
    }
    hipStream_t st = (hipStream_t)stream;
    RAT3D_TRY(prepare_call(net, st));
    const rat3d_net_desc& d = net->d;
    net->ext_x = x;
    Exec e{net, st, 0};
    RAT3D_TRY(stem_fwd_eval(e));
    for (int i = 0; i < 3; ++i) {
        RAT3D_TRY(ru_fwd_eval(e, net->rus[i]));
        RAT3D_TRY(am_fwd_eval(e, net->ams[i]));
    }
    const TRef& top = net->ams[2].out;
    if (logits)
        RAT3D_TRY(gradcam_logits(d.n, net->fc_c, top.s.vox(), 2, net->dt, e.a(top),
                                 e.par(net->fc.w_off), e.par(net->fc.b_off), logits, st));
    // d logit_k / d top: the FC row of class k spread evenly by the average pool
    RAT3D_TRY(gradcam_seed(d.n, net->fc_c, top.s.vox(), 2, net->dt, e.par(net->fc.w_off), classes,
                           e.g(top), st));
    for (int i = 2; i >= target; --i) {
        RAT3D_TRY(am_bwd_eval(e, net->ams[i]));
        RAT3D_TRY(ru_bwd_eval(e, net->rus[i], false));
    }
    const TRef& A = gradcam_target(net, target);
    return gradcam_maps(d.n, A.s.c, A.s.d, A.s.h, A.s.w, net->dt, e.a(A), e.g(A),
                        (float*)(net->ws + net->gcam_alpha_off), cam, d.d, d.h, d.w, cam_up, st);
}

}  // extern "C"
