"""Oracle BigGAN residual blocks and self-attention block (test infra only).

The paper names BigGAN as its benchmark backbone (Design, "Network
Backbones"; Evaluation, "Experiment Setup") and pins its size at 158.42M
parameters (Table tab:GAN) but does not restate its layers.  The block
structure below is the reading that reproduces that parameter count
(checked in the tests):

* generator block:  cBN -> ReLU -> 2x nearest upsample -> SN conv3x3 ->
  cBN -> ReLU -> SN conv3x3, plus an SN conv1x1 skip on the upsampled input;
* discriminator block: [ReLU] -> SN conv3x3 -> ReLU -> SN conv3x3 ->
  [2x2 avg-pool], plus an SN conv1x1 skip (pooled input) or the identity;
* attention: SN 1x1 projections theta (C/8), phi (C/8), g (C/2) with phi
  and g 2x2 max-pooled, softmax over keys without scaling, SN 1x1 output
  projection (C/2 -> C), y = x + gamma * o.

Class-conditional BN: gain = 1 + cond W_g^T, bias = cond W_b^T with SN,
bias-free linears; batch statistics; eps from the config.

Precision (Implementation, "Mixed-Precision Training"): with
`cfg.bf16` set, every tensor stored in bfloat16 is rounded here at that
point: block outputs, the intermediate conv output, every conv operand after
its prologue (BN/ReLU/pooling), the SN-normalised weight operands and the
activation gradients.  Accumulation, statistics, SN, softmax and weight
gradients stay in float64.  With `cfg.bf16` unset nothing is rounded (the
fp32 path, compared at 1e-4).

The spectral normalisation of a block convolution is applied to its
accumulated product: conv(a, W / sigma) is evaluated as conv(a, W) / sigma,
the stored weight operand being the master filter itself, so that its bf16
rounding does not depend on sigma (sigma stays in float64 here, fp32 on the
GPU).  Two convolutions sit next to a 2x resampling: the generator's conv1
reads the nearest upsample, the pooling discriminator block's conv2 feeds
the 2x2 average.  Their weight operand is the folded filter
(layers.up2_conv_fold, layers.pool2_conv_fold: the 3x3 taps that meet one
input pixel added), so under bf16 it is the folded filter that is rounded,
once.  In exact arithmetic all of this equals the plain compositions with
the normalised 3x3 filter (pinned in the layer and block tests), and the
weight gradients are those of the plain filter.
"""
from dataclasses import dataclass

import numpy as np

from . import layers as L
from .numerics import rounder


@dataclass
class BlockCfg:
    bf16: bool = True
    bn_eps: float = 1e-5
    sn_eps: float = 1e-12
    n_power_iter: int = 1
    update_u: bool = True
    # test hook: {key: (u, v)} held fixed, sigma = u^T W v (for finite
    # differences, which must see the same u, v as the analytic gradient)
    frozen: dict = None


def spectral(p, u, key, cfg):
    """SN of parameter `key`: returns (W/sigma, (u_new, v, sigma))."""
    w = p[key]
    wmat = w.reshape(w.shape[0], -1)
    if cfg.frozen is not None:
        un, v = cfg.frozen[key]
        sigma = float(un @ (wmat @ v))
    else:
        un, v, sigma = L.sn_power_iter(wmat, u[key], cfg.n_power_iter,
                                       cfg.sn_eps)
    return w / sigma, (un, v, sigma)


def _sn_all(p, u, keys, cfg, u_out):
    ws, st = {}, {}
    for k in keys:
        ws[k], st[k] = spectral(p, u, k, cfg)
        if cfg.update_u:
            u_out[k] = st[k][0]
    return ws, st


def _sn_grads(dws, ws, st, grads):
    for k, d in dws.items():
        un, v, sigma = st[k]
        grads[k] = L.sn_bwd(d, ws[k], un, v, sigma)


# --------------------------------------------------------------------------
# generator block
# --------------------------------------------------------------------------
GBLOCK_SN = ("bn1.gain", "bn1.bias", "conv1.w", "bn2.gain", "bn2.bias",
             "conv2.w", "sc.w")


def gblock_param_shapes(cin, cout, dc):
    return {
        "bn1.gain": (cin, dc), "bn1.bias": (cin, dc),
        "conv1.w": (cout, 3, 3, cin), "conv1.b": (cout,),
        "bn2.gain": (cout, dc), "bn2.bias": (cout, dc),
        "conv2.w": (cout, 3, 3, cout), "conv2.b": (cout,),
        "sc.w": (cout, 1, 1, cin), "sc.b": (cout,),
    }


def gblock_fwd(x, cond, p, u, cfg):
    """x (N,H,W,Cin), cond (N,dc) -> y (N,2H,2W,Cout).  Returns (y, u_new, cache)."""
    R = rounder(cfg.bf16)
    u_new = dict(u)
    ws, st = _sn_all(p, u, GBLOCK_SN, cfg, u_new)
    g1 = 1.0 + cond @ ws["bn1.gain"].T
    b1 = cond @ ws["bn1.bias"].T
    bn1, c1 = L.cbn_fwd(x, g1, b1, cfg.bn_eps)
    a1 = R(L.relu(bn1))
    s1, s2, ssc = (st[k][2] for k in ("conv1.w", "conv2.w", "sc.w"))
    f1 = R(L.up2_conv_fold(p["conv1.w"]))      # conv3x3 over up2, folded
    h1 = R(L.up2_conv(a1, f1) / s1 + p["conv1.b"])
    g2 = 1.0 + cond @ ws["bn2.gain"].T
    b2 = cond @ ws["bn2.bias"].T
    bn2, c2 = L.cbn_fwd(h1, g2, b2, cfg.bn_eps)
    a2 = R(L.relu(bn2))
    w2 = R(p["conv2.w"])
    wsc = R(p["sc.w"])
    # conv1x1(up2(x)) == up2(conv1x1(x)) exactly; the skip is summed unrounded
    skip = L.up2(L.conv2d(x, wsc) / ssc + p["sc.b"])
    y = R(L.conv2d(a2, w2) / s2 + p["conv2.b"] + skip)
    cache = dict(x=x, cond=cond, ws=ws, st=st, bn1=bn1, c1=c1, a1=a1, f1=f1,
                 h1=h1, bn2=bn2, c2=c2, a2=a2, w2=w2, wsc=wsc, s1=s1, s2=s2,
                 ssc=ssc)
    return y, u_new, cache


def gblock_bwd(dy, cache, cfg):
    """dy (N,2H,2W,Cout) -> (dx, dcond, grads dict)."""
    R = rounder(cfg.bf16)
    c = cache
    dws, grads = {}, {}
    dws["conv2.w"] = L.conv2d_wgrad(dy, c["a2"], 3)
    grads["conv2.b"] = L.bias_grad(dy)
    dys = L.up2_bwd(dy)                       # skip gradient at low resolution
    dws["sc.w"] = L.conv2d_wgrad(dys, c["x"], 1)
    grads["sc.b"] = L.bias_grad(dys)
    dx_skip = L.conv2d_dgrad(R(dys), c["wsc"]) / c["ssc"]
    da2 = L.conv2d_dgrad(dy, c["w2"]) / c["s2"]
    dbn2 = da2 * (c["bn2"] > 0)
    dh1, dg2, db2 = L.cbn_bwd(dbn2, c["c2"])
    dh1 = R(dh1)
    dws["conv1.w"] = L.conv2d_wgrad(dh1, L.up2(c["a1"]), 3)
    grads["conv1.b"] = L.bias_grad(dh1)
    da1 = L.up2_conv_dgrad(dh1, c["f1"]) / c["s1"]
    dbn1 = da1 * (c["bn1"] > 0)
    dx1, dg1, db1 = L.cbn_bwd(dbn1, c["c1"])
    dx = R(dx1 + dx_skip)
    cond, ws = c["cond"], c["ws"]
    dws["bn1.gain"] = dg1.T @ cond
    dws["bn1.bias"] = db1.T @ cond
    dws["bn2.gain"] = dg2.T @ cond
    dws["bn2.bias"] = db2.T @ cond
    dcond = (dg1 @ ws["bn1.gain"] + db1 @ ws["bn1.bias"]
             + dg2 @ ws["bn2.gain"] + db2 @ ws["bn2.bias"])
    _sn_grads(dws, ws, c["st"], grads)
    return dx, dcond, grads


# --------------------------------------------------------------------------
# discriminator block
# --------------------------------------------------------------------------
def dblock_param_shapes(cin, cout, learnable_sc):
    s = {"conv1.w": (cout, 3, 3, cin), "conv1.b": (cout,),
         "conv2.w": (cout, 3, 3, cout), "conv2.b": (cout,)}
    if learnable_sc:
        s.update({"sc.w": (cout, 1, 1, cin), "sc.b": (cout,)})
    return s


def dblock_fwd(x, p, u, cfg, preact, down, learnable_sc):
    """x (N,H,W,Cin) -> y (N,H/2,W/2,Cout) if down else (N,H,W,Cout)."""
    R = rounder(cfg.bf16)
    u_new = dict(u)
    keys = ("conv1.w", "conv2.w") + (("sc.w",) if learnable_sc else ())
    ws, st = _sn_all(p, u, keys, cfg, u_new)
    x = R(x)                                  # operand precision of the input
    a0 = L.relu(x) if preact else x
    s1, s2 = st["conv1.w"][2], st["conv2.w"][2]
    w1 = R(p["conv1.w"])
    h = R(L.conv2d(a0, w1) / s1 + p["conv1.b"])
    a1 = L.relu(h)
    if down:
        # avgpool2(conv3x3): one stride-2 4x4 filter, folded
        w2 = R(L.pool2_conv_fold(p["conv2.w"]))
        main = L.pool2_conv(a1, w2) / s2 + p["conv2.b"]
    else:
        w2 = R(p["conv2.w"])
        main = L.conv2d(a1, w2) / s2 + p["conv2.b"]
    cache = dict(x=x, a0=a0, h=h, a1=a1, w1=w1, w2=w2, s1=s1, s2=s2, ws=ws,
                 st=st)
    if learnable_sc:
        # avgpool and conv1x1 commute exactly; pool first, operand in bf16
        xs = R(L.avgpool2(x)) if down else x
        wsc = R(p["sc.w"])
        ssc = st["sc.w"][2]
        sc = L.conv2d(xs, wsc) / ssc + p["sc.b"]
        cache.update(xs=xs, wsc=wsc, ssc=ssc)
    else:
        sc = x
    y = R(main + sc)
    return y, u_new, cache


def dblock_bwd(dy, cache, cfg, preact, down, learnable_sc, dx_f32=False):
    """dy -> (dx, grads).  dx is left unrounded when dx_f32 (the image
    gradient that feeds the fp32 generator output layer)."""
    R = rounder(cfg.bf16)
    c = cache
    dws, grads = {}, {}
    dc2 = L.avgpool2_bwd(dy) if down else dy
    dws["conv2.w"] = L.conv2d_wgrad(dc2, c["a1"], 3)
    grads["conv2.b"] = L.bias_grad(dc2)
    da1 = (L.pool2_conv_dgrad(dy, c["w2"]) if down else L.conv2d_dgrad(dy, c["w2"])) / c["s2"]
    dh = R(da1 * (c["h"] > 0))
    dws["conv1.w"] = L.conv2d_wgrad(dh, c["a0"], 3)
    grads["conv1.b"] = L.bias_grad(dh)
    dxm = L.conv2d_dgrad(dh, c["w1"]) / c["s1"]
    if preact:
        dxm = dxm * (c["x"] > 0)
    if learnable_sc:
        dws["sc.w"] = L.conv2d_wgrad(dy, c["xs"], 1)
        grads["sc.b"] = L.bias_grad(dy)
        dxs = L.conv2d_dgrad(dy, c["wsc"]) / c["ssc"]
        dxsc = L.avgpool2_bwd(dxs) if down else dxs
    else:
        dxsc = dy
    dx = dxm + dxsc
    if not dx_f32:
        dx = R(dx)
    _sn_grads(dws, c["ws"], c["st"], grads)
    return dx, grads


# --------------------------------------------------------------------------
# self-attention block
# --------------------------------------------------------------------------
ATTN_SN = ("theta", "phi", "g", "o")


def attn_param_shapes(c):
    return {"theta": (c // 8, 1, 1, c), "phi": (c // 8, 1, 1, c),
            "g": (c // 2, 1, 1, c), "o": (c, 1, 1, c // 2), "gamma": (1,)}


def attn_fwd(x, p, u, cfg):
    """x (N,H,W,C) -> y = x + gamma * o.  Keys/values are 2x2 max-pooled."""
    R = rounder(cfg.bf16)
    u_new = dict(u)
    ws, st = _sn_all(p, u, ATTN_SN, cfg, u_new)
    n, h, w, ch = x.shape
    wt, wp, wg, wo = (R(ws[k]) for k in ATTN_SN)
    theta = R(L.conv2d(x, wt))
    phif = R(L.conv2d(x, wp))
    gf = R(L.conv2d(x, wg))
    phi, argp = L.maxpool2(phif)
    g, argg = L.maxpool2(gf)
    q = theta.reshape(n, h * w, -1)
    k = phi.reshape(n, h * w // 4, -1)
    v = g.reshape(n, h * w // 4, -1)
    o_att, pm = L.attention_core_fwd(q, k, v)
    o_att = R(o_att).reshape(n, h, w, -1)
    o = L.conv2d(o_att, wo)
    gamma = float(p["gamma"][0])
    y = R(x + gamma * o)
    cache = dict(x=x, ws=ws, st=st, wt=wt, wp=wp, wg=wg, wo=wo, q=q, k=k, v=v,
                 pm=pm, argp=argp, argg=argg, o_att=o_att, o=o, gamma=gamma)
    return y, u_new, cache


def attn_bwd(dy, cache, cfg):
    R = rounder(cfg.bf16)
    c = cache
    n, h, w, ch = dy.shape
    gamma = c["gamma"]
    grads, dws = {}, {}
    grads["gamma"] = np.array([float((dy * c["o"]).sum())])
    dws["o"] = gamma * L.conv2d_wgrad(dy, c["o_att"], 1)
    do_att = R(gamma * L.conv2d_dgrad(dy, c["wo"]))
    dq, dk, dv = L.attention_core_bwd(do_att.reshape(n, h * w, -1),
                                      c["q"], c["k"], c["v"], c["pm"])
    dtheta = R(dq.reshape(n, h, w, -1))
    dphif = R(L.maxpool2_bwd(dk.reshape(n, h // 2, w // 2, -1), c["argp"]))
    dgf = R(L.maxpool2_bwd(dv.reshape(n, h // 2, w // 2, -1), c["argg"]))
    x = c["x"]
    dws["theta"] = L.conv2d_wgrad(dtheta, x, 1)
    dws["phi"] = L.conv2d_wgrad(dphif, x, 1)
    dws["g"] = L.conv2d_wgrad(dgf, x, 1)
    dx = R(dy + L.conv2d_dgrad(dtheta, c["wt"]) + L.conv2d_dgrad(dphif, c["wp"])
           + L.conv2d_dgrad(dgf, c["wg"]))
    _sn_grads(dws, c["ws"], c["st"], grads)
    return dx, grads
