"""Oracle BigGAN networks and the G+D train step (test infrastructure only).

Architecture reading (the paper uses BigGAN as its benchmark, Evaluation
"Experiment Setup", and pins it only by its parameter count, 158.42M in
Table tab:GAN; `param_count(biggan128())` reproduces 158,416,358):

generator   z split into (n_blocks + 1) equal chunks; chunk 0 -> SN linear
            (with bias) -> 4x4xC0 (NHWC order); block i is conditioned on
            [shared_embedding(y) || chunk i+1]; attention after the block
            whose output resolution equals attn_res; output layer
            BN (affine) -> ReLU -> SN conv3x3 -> 3 channels -> tanh (fp32).
discriminator  blocks with ReLU pre-activation except the first; skip is a
            learnable SN 1x1 conv when channels change or the block pools;
            attention after the first block at attn_res; head
            ReLU -> spatial sum -> SN linear (+bias) + <SN embed(y), h>
            (fp32).
train step  n_D discriminator steps on concat(real, fake) (inputs that
            share a weight are batched, Implementation "Hardware-Aware
            Layout Transformation"), then one generator step; the D:G
            ratio is adjustable (Numerical Optimizations, "Asynchronous
            Update Scheme").  Hinge loss; each network has its own
            optimiser (Numerical Optimizations, "Asymmetric Optimization
            Policy": AdaBelief for G with Adam for D is the paper's pick).
"""
from dataclasses import dataclass, field

import numpy as np

from . import layers as L
from .blocks import (BlockCfg, attn_bwd, attn_fwd, attn_param_shapes,
                     dblock_bwd, dblock_fwd, dblock_param_shapes, gblock_bwd,
                     gblock_fwd, gblock_param_shapes, spectral)
from .numerics import rounder


@dataclass
class Arch:
    img: int
    ch: int
    g_mult: tuple        # C0 multiplier, then each G block's output multiplier
    d_mult: tuple        # each D block's output multiplier
    d_down: tuple        # each D block pools 2x2
    attn_res: int        # 0: no attention
    n_classes: int
    dz: int
    shared_dim: int

    @property
    def n_g(self):
        return len(self.g_mult) - 1

    @property
    def zchunk(self):
        return self.dz // (self.n_g + 1)

    @property
    def dc(self):
        return self.shared_dim + self.zchunk


def biggan128():
    return Arch(128, 96, (16, 16, 8, 4, 2, 1), (1, 2, 4, 8, 16, 16),
                (1, 1, 1, 1, 1, 0), 64, 1000, 120, 128)


def biggan512():
    return Arch(512, 64, (16, 16, 8, 8, 4, 2, 1, 1), (1, 1, 2, 4, 8, 8, 16, 16),
                (1, 1, 1, 1, 1, 1, 1, 0), 64, 1000, 128, 128)


@dataclass
class OptSpec:
    """One network's optimiser: kind "adam" or "adabelief"."""
    kind: str = "adam"
    lr: float = 1e-4
    beta1: float = 0.0
    beta2: float = 0.999
    eps: float = 1e-6


def adam_g():
    return OptSpec("adam", 1e-4, 0.0, 0.999, 1e-6)


def adam_d():
    return OptSpec("adam", 4e-4, 0.0, 0.999, 1e-6)


def adabelief_g():
    """AdaBelief for the generator.  beta1 > 0 is required: with beta1 = 0
    the running mean equals the gradient and the belief term vanishes."""
    return OptSpec("adabelief", 1e-4, 0.5, 0.999, 1e-12)


@dataclass
class HParams:
    bn_eps: float = 1e-5
    sn_eps: float = 1e-12
    n_power_iter: int = 1
    opt_g: OptSpec = field(default_factory=adam_g)
    opt_d: OptSpec = field(default_factory=adam_d)
    bf16: bool = True
    frozen: dict = None          # test hook, see BlockCfg.frozen

    def block(self, prefix=""):
        fz = None
        if self.frozen is not None:
            fz = {k[len(prefix):]: v for k, v in self.frozen.items()
                  if k.startswith(prefix)}
        return BlockCfg(bf16=self.bf16, bn_eps=self.bn_eps, sn_eps=self.sn_eps,
                        n_power_iter=self.n_power_iter, frozen=fz)


# --------------------------------------------------------------------------
# parameter layout
# --------------------------------------------------------------------------
def g_layout(a):
    """Ordered {name: shape} of the generator's parameters, and the SN set."""
    c0 = a.g_mult[0] * a.ch
    s = {"shared": (a.n_classes, a.shared_dim),
         "linear.w": (16 * c0, a.zchunk), "linear.b": (16 * c0,)}
    sn = ["linear.w"]
    res = 4
    for i in range(a.n_g):
        cin, cout = a.g_mult[i] * a.ch, a.g_mult[i + 1] * a.ch
        for k, v in gblock_param_shapes(cin, cout, a.dc).items():
            s["g%d.%s" % (i, k)] = v
        sn += ["g%d.%s" % (i, k) for k in ("bn1.gain", "bn1.bias", "conv1.w",
                                           "bn2.gain", "bn2.bias", "conv2.w",
                                           "sc.w")]
        res *= 2
        if res == a.attn_res:
            for k, v in attn_param_shapes(cout).items():
                s["attn.%s" % k] = v
            sn += ["attn.%s" % k for k in ("theta", "phi", "g", "o")]
    c = a.g_mult[-1] * a.ch
    s.update({"out_bn.gain": (c,), "out_bn.bias": (c,),
              "out_conv.w": (3, 3, 3, c), "out_conv.b": (3,)})
    sn.append("out_conv.w")
    return s, sn


def d_blocks(a):
    """Per D block: (cin, cout, preact, down, learnable_sc, attention_after)."""
    out, res, cin, placed = [], a.img, 3, False
    for j, (m, down) in enumerate(zip(a.d_mult, a.d_down)):
        cout = m * a.ch
        res = res // 2 if down else res
        att = (res == a.attn_res) and not placed
        placed = placed or att
        out.append((cin, cout, j > 0, bool(down), cin != cout or bool(down), att))
        cin = cout
    return out


def d_layout(a):
    s, sn = {}, []
    for j, (cin, cout, pre, down, lsc, att) in enumerate(d_blocks(a)):
        for k, v in dblock_param_shapes(cin, cout, lsc).items():
            s["d%d.%s" % (j, k)] = v
        sn += ["d%d.%s" % (j, k) for k in ("conv1.w", "conv2.w")]
        if lsc:
            sn.append("d%d.sc.w" % j)
        if att:
            for k, v in attn_param_shapes(cout).items():
                s["attn.%s" % k] = v
            sn += ["attn.%s" % k for k in ("theta", "phi", "g", "o")]
    c = a.d_mult[-1] * a.ch
    s.update({"head.w": (1, c), "head.b": (1,), "embed": (a.n_classes, c)})
    sn += ["head.w", "embed"]
    return s, sn


def param_count(a):
    g, _ = g_layout(a)
    d, _ = d_layout(a)
    cnt = lambda s: sum(int(np.prod(v)) for v in s.values())
    return cnt(g), cnt(d)


def _sub(d, prefix):
    n = len(prefix)
    return {k[n:]: v for k, v in d.items() if k.startswith(prefix)}


def _put(dst, prefix, src):
    for k, v in src.items():
        dst[prefix + k] = v


# --------------------------------------------------------------------------
# generator
# --------------------------------------------------------------------------
def g_out_fwd(x5, p, u, cfg, bn_eps):
    """Generator output layer, fp32 (model: Architecture; the last layer in
    full precision: Design, "System Optimizations"): BN with batch
    statistics and an affine gain / bias -> ReLU -> SN conv3x3 to 3 channels
    (+ bias) -> tanh.  Reads out_bn.gain, out_bn.bias, out_conv.w and
    out_conv.b of p.  Returns the image, the new u of out_conv.w and the
    cache for g_out_bwd."""
    bn, cbn = L.cbn_fwd(x5, p["out_bn.gain"][None, :], p["out_bn.bias"][None, :],
                        bn_eps)
    act = L.relu(bn)
    wo, sto = spectral(p, u, "out_conv.w", cfg)
    img = np.tanh(L.conv2d(act, wo, p["out_conv.b"]))
    return img, sto[0], dict(bn=bn, cbn=cbn, act=act, wo=wo, sto=sto, img=img)


def g_out_bwd(dimg, c):
    """dimg (N, H, W, 3) -> (gradient of the layer's input, gradients of its
    four parameters)."""
    grads = {}
    dt = dimg * (1.0 - c["img"] ** 2)
    dwo = L.conv2d_wgrad(dt, c["act"], 3)
    grads["out_conv.b"] = L.bias_grad(dt)
    un, v, s = c["sto"]
    grads["out_conv.w"] = L.sn_bwd(dwo, c["wo"], un, v, s)
    dact = L.conv2d_dgrad(dt, c["wo"])
    dbn = dact * (c["bn"] > 0)
    dh, dgain, dbias = L.cbn_bwd(dbn, c["cbn"])
    grads["out_bn.gain"] = dgain[0]
    grads["out_bn.bias"] = dbias[0]
    return dh, grads


def g_fwd(a, hp, p, u, z, y):
    """z (N, dz), y (N,) int -> image (N, img, img, 3) in [-1, 1]."""
    R = rounder(hp.bf16)
    cfg = hp.block()
    n = z.shape[0]
    u_new = dict(u)
    zc = a.zchunk
    zs = [z[:, i * zc:(i + 1) * zc] for i in range(a.n_g + 1)]
    emb = p["shared"][y]
    wl, stl = spectral(p, u, "linear.w", cfg)
    u_new["linear.w"] = stl[0]
    c0 = a.g_mult[0] * a.ch
    h = R(zs[0] @ wl.T + p["linear.b"]).reshape(n, 4, 4, c0)
    caches = []
    res = 4
    for i in range(a.n_g):
        cond = np.concatenate([emb, zs[i + 1]], axis=1)
        pre = "g%d." % i
        h, ub, cb = gblock_fwd(h, cond, _sub(p, pre), _sub(u, pre),
                               hp.block(pre))
        _put(u_new, pre, {k: ub[k] for k in ub})
        caches.append(("g", cb))
        res *= 2
        if res == a.attn_res:
            h, ua, ca = attn_fwd(h, _sub(p, "attn."), _sub(u, "attn."),
                                 hp.block("attn."))
            _put(u_new, "attn.", ua)
            caches.append(("a", ca))
    # output layer, fp32
    img, u_new["out_conv.w"], hc = g_out_fwd(h, p, u, cfg, hp.bn_eps)
    cache = dict(zs=zs, y=y, emb=emb, wl=wl, stl=stl, caches=caches, **hc)
    return img, u_new, cache


def g_bwd(a, hp, p, dimg, cache):
    """dimg (N, img, img, 3) -> gradients of every generator parameter."""
    R = rounder(hp.bf16)
    cfg = hp.block()
    c = cache
    dh, grads = g_out_bwd(dimg, c)
    dh = R(dh)
    n = dimg.shape[0]
    demb = np.zeros((n, a.shared_dim))
    blk = a.n_g - 1
    for kind, cb in reversed(c["caches"]):
        if kind == "a":
            dh, ga = attn_bwd(dh, cb, cfg)
            _put(grads, "attn.", ga)
        else:
            dh, dcond, gb = gblock_bwd(dh, cb, cfg)
            _put(grads, "g%d." % blk, gb)
            demb += dcond[:, :a.shared_dim]
            blk -= 1
    dshared = np.zeros(p["shared"].shape)
    np.add.at(dshared, c["y"], demb)
    grads["shared"] = dshared
    dh0 = dh.reshape(n, -1)
    grads["linear.b"] = dh0.sum(axis=0)
    dwl = dh0.T @ c["zs"][0]
    un, v, s = c["stl"]
    grads["linear.w"] = L.sn_bwd(dwl, c["wl"], un, v, s)
    return grads


# --------------------------------------------------------------------------
# discriminator
# --------------------------------------------------------------------------
def d_fwd(a, hp, p, u, x, y):
    """x (N, img, img, 3) float images, y (N,) -> logits (N,)."""
    cfg = hp.block()
    u_new = dict(u)
    caches = []
    h = x
    for j, (cin, cout, pre, down, lsc, att) in enumerate(d_blocks(a)):
        bp = "d%d." % j
        h, ub, cb = dblock_fwd(h, _sub(p, bp), _sub(u, bp), hp.block(bp), pre,
                               down, lsc)
        _put(u_new, bp, ub)
        caches.append(("d", j, cb))
        if att:
            h, ua, ca = attn_fwd(h, _sub(p, "attn."), _sub(u, "attn."),
                                 hp.block("attn."))
            _put(u_new, "attn.", ua)
            caches.append(("a", j, ca))
    # head, fp32
    act = L.relu(h)
    hs = act.sum(axis=(1, 2))
    wh, sth = spectral(p, u, "head.w", cfg)
    we, ste = spectral(p, u, "embed", cfg)
    u_new["head.w"], u_new["embed"] = sth[0], ste[0]
    ey = we[y]
    out = hs @ wh[0] + p["head.b"][0] + (ey * hs).sum(axis=1)
    cache = dict(caches=caches, h=h, hs=hs, wh=wh, sth=sth, we=we, ste=ste,
                 ey=ey, y=y)
    return out, u_new, cache


def d_bwd(a, hp, p, dout, cache, need_dx):
    """dout (N,) -> (dx or None, grads)."""
    R = rounder(hp.bf16)
    cfg = hp.block()
    c = cache
    grads = {}
    hs = c["hs"]
    grads["head.b"] = np.array([dout.sum()])
    dwh = (dout @ hs)[None, :]
    dwe = np.zeros(c["we"].shape)
    np.add.at(dwe, c["y"], dout[:, None] * hs)
    un, v, s = c["sth"]
    grads["head.w"] = L.sn_bwd(dwh, c["wh"], un, v, s)
    un, v, s = c["ste"]
    grads["embed"] = L.sn_bwd(dwe, c["we"], un, v, s)
    dhs = dout[:, None] * (c["wh"][0][None, :] + c["ey"])
    dh = R(dhs[:, None, None, :] * (c["h"] > 0))
    blocks = d_blocks(a)
    for kind, j, cb in reversed(c["caches"]):
        if kind == "a":
            dh, ga = attn_bwd(dh, cb, cfg)
            _put(grads, "attn.", ga)
        else:
            cin, cout, pre, down, lsc, att = blocks[j]
            dh, gb = dblock_bwd(dh, cb, cfg, pre, down, lsc, dx_f32=(j == 0))
            _put(grads, "d%d." % j, gb)
    return (dh if need_dx else None), grads


# --------------------------------------------------------------------------
# train step
# --------------------------------------------------------------------------
@dataclass
class OptState:
    m: dict
    v: dict
    t: int = 0


def opt_init(p):
    return OptState({k: np.zeros_like(v) for k, v in p.items()},
                     {k: np.zeros_like(v) for k, v in p.items()}, 0)


def opt_update(p, grads, st, spec):
    """One optimiser step of every parameter (step t = st.t + 1)."""
    st.t += 1
    step = {"adam": L.adam, "adabelief": L.adabelief}[spec.kind]
    newp = {}
    for k in p:
        newp[k], st.m[k], st.v[k] = step(p[k], grads[k], st.m[k], st.v[k], st.t,
                                         spec.lr, spec.beta1, spec.beta2, spec.eps)
    return newp


def d_step_images(a, hp, D, optD, x_real, y_real, x_fake, y_fake):
    """One discriminator step on given images: D forward on
    concat(real, fake) with labels concat(y_real, y_fake), hinge, backward,
    D's optimiser.  Returns (D, L_D, D's gradients)."""
    dp, du = D
    b = x_real.shape[0]
    x = np.concatenate([x_real, x_fake], axis=0)
    yy = np.concatenate([y_real, y_fake], axis=0)
    out, du, cache = d_fwd(a, hp, dp, du, x, yy)
    loss, dr, df = L.hinge_d(out[:b], out[b:])
    _, grads = d_bwd(a, hp, dp, np.concatenate([dr, df]), cache, need_dx=False)
    dp = opt_update(dp, grads, optD, hp.opt_d)
    return (dp, du), loss, grads


def d_step(a, hp, G, D, optD, x_real, y_real, z, y_fake):
    """One discriminator step: G forward (no gradient; G's u advances),
    then the D step on concat(real, G(z, y_fake))."""
    gp, gu = G
    fake, gu, _ = g_fwd(a, hp, gp, gu, z, y_fake)
    D, loss, grads = d_step_images(a, hp, D, optD, x_real, y_real, fake, y_fake)
    return (gp, gu), D, loss, grads


def g_step(a, hp, G, D, optG, z, y):
    gp, gu = G
    dp, du = D
    fake, gu, gcache = g_fwd(a, hp, gp, gu, z, y)
    out, du, dcache = d_fwd(a, hp, dp, du, fake, y)
    loss, dout = L.hinge_g(out)
    dimg, _ = d_bwd(a, hp, dp, dout, dcache, need_dx=True)
    grads = g_bwd(a, hp, gp, dimg, gcache)
    gp = opt_update(gp, grads, optG, hp.opt_g)
    return (gp, gu), (dp, du), loss, grads


def train_step(a, hp, G, D, optG, optD, d_inputs, g_inputs):
    """n_D = len(d_inputs) D steps, then one G step.

    d_inputs: list of (x_real, y_real, z, y_fake); g_inputs: (z, y).
    Returns (G, D, losses [L_D ... , L_G], last D grads, G grads)."""
    losses = []
    gd = None
    for (xr, yr, z, yf) in d_inputs:
        G, D, ld, gd = d_step(a, hp, G, D, optD, xr, yr, z, yf)
        losses.append(ld)
    G, D, lg, gg = g_step(a, hp, G, D, optG, *g_inputs)
    losses.append(lg)
    return G, D, losses, gd, gg


def async_step(a, hp, G, D, optG, optD, d_inputs, g_inputs, img_buff, lab_buff):
    """One iteration of the asynchronous update scheme (Numerical
    Optimizations, "Asynchronous Update Scheme"), written sequentially: the
    two halves below read disjoint state, so running them one after the
    other or side by side gives the same numbers.

    * The generator half takes a snapshot of D as it is at the start of the
      iteration and makes one generator step of batch len(z) against it
      (the snapshot's SN vectors advance and are dropped with the snapshot).
      Its samples, their labels and the snapshot's predictions on them are
      what goes into img_buff / lab_buff / pred_buff for the next iteration.
    * The discriminator half makes len(d_inputs) D steps; step k sees the
      real batch d_inputs[k] = (x_real, y_real) and the k-th len(x_real)
      images and labels of img_buff / lab_buff, the samples of the previous
      iteration's generator.

    Returns (G, D, losses [L_D ..., L_G], img_buff, lab_buff, pred_buff,
    last D grads, G grads)."""
    z, y = g_inputs
    snapshot = (dict(D[0]), dict(D[1]))
    gp, gu = G
    fake, gu, gcache = g_fwd(a, hp, gp, gu, z, y)
    pred, _, dcache = d_fwd(a, hp, snapshot[0], snapshot[1], fake, y)
    lg, dout = L.hinge_g(pred)
    dimg, _ = d_bwd(a, hp, snapshot[0], dout, dcache, need_dx=True)
    gg = g_bwd(a, hp, gp, dimg, gcache)
    gp = opt_update(gp, gg, optG, hp.opt_g)
    losses, gd = [], None
    for k, (xr, yr) in enumerate(d_inputs):
        b = xr.shape[0]
        D, ld, gd = d_step_images(a, hp, D, optD, xr, yr, img_buff[k * b:(k + 1) * b],
                                  lab_buff[k * b:(k + 1) * b])
        losses.append(ld)
    losses.append(lg)
    return (gp, gu), D, losses, fake, np.array(y), pred, gd, gg
