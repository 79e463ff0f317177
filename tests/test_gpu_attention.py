"""GPU parity: the self-attention block vs the oracle (bf16 path)."""
import numpy as np
import pytest

from oracle import blocks as OB
from oracle.numerics import bf16
from paragan_2411_03999_amd import lib
from paragan_2411_03999_amd.synth import Stream, init_params, init_u

from .bounds import tie_ambiguous, ulp_bf16
from .parity import TOL_BF16, Report, check, check_with_bound, need_gpu, context, harvest

pytestmark = pytest.mark.gpu


def f32(d):
    return {k: np.asarray(v, np.float32).astype(np.float64) for k, v in d.items()}


def run_attn(B, H, W, C, seed, gamma=0.7, weights="gaussian"):
    s = Stream(seed)
    shapes = OB.attn_param_shapes(C)
    p = f32(init_params(shapes, s, weights=weights, attn_gamma=gamma))
    u = f32(init_u(shapes, OB.ATTN_SN, s))
    x = bf16(s.normal((B, H, W, C)))
    dy = bf16(s.normal((B, H, W, C)))
    print("attn case", dict(B=B, H=H, W=W, C=C, seed=seed), flush=True)
    return compare_attn(x, p, u, dy)


def compare_attn(x, p, u, dy):
    """The attention block on the GPU against the oracle, on given bf16
    inputs x, output gradient dy, parameters p and SN vectors u."""
    torch = need_gpu()
    p, u = f32(p), f32(u)
    B, H, W, C = x.shape
    shapes = OB.attn_param_shapes(C)
    cfg = OB.BlockCfg(bf16=True)
    y_r, u_r, cache = OB.attn_fwd(x, p, u, cfg)
    dx_r, g_r = OB.attn_bwd(dy, cache, cfg)
    d = lib.AttnDesc(B, H, W, C, 1, 1e-12)
    ents, npar, nu = lib.paragan_attn_layout(d)
    assert [(e["name"], e["shape"]) for e in ents] == list(shapes.items())
    sb, wb = lib.paragan_attn_sizes(d)
    ctx = context()
    P = lib.flat_from_named(ents, npar, p)
    U = lib.u_from_named(ents, nu, u)
    X = lib.to_device_nhwc(x, lib.BF16)
    Y = lib.empty_nhwc(B, H, W, C, lib.BF16)
    saved, ws = lib.workspace(sb), lib.workspace(wb)
    lib.paragan_attn_fwd(ctx, d, P, U, X, Y, saved, ws)
    DX = lib.empty_nhwc(B, H, W, C, lib.BF16)
    G = torch.zeros(npar, dtype=torch.float32, device="cuda")
    lib.paragan_attn_bwd(ctx, d, P, X, saved, lib.to_device_nhwc(dy, lib.BF16), DX, G, ws)
    torch.cuda.synchronize()
    harvest(ctx)
    rep = Report()
    check("y", lib.from_device_nhwc(Y, C), y_r, True, rep)
    # the attention contribution alone (y - x), a sharper view of the core.
    # Both sides round y = x + gamma o to bf16; where |x| is large next to
    # gamma o, a change of o within the bar moves y across a rounding
    # midpoint by one ulp of y, which this view would see at full size: allow
    # that ulp exactly where the oracle's unrounded y lies within
    # gamma * 2e-2 * max|o| of a midpoint.
    yx = cache["x"] + cache["gamma"] * cache["o"]
    band = abs(cache["gamma"]) * TOL_BF16 * np.abs(cache["o"]).max()
    flip = np.where(tie_ambiguous(yx, band), ulp_bf16(yx), 0.0)
    check_with_bound("y-x", lib.from_device_nhwc(Y, C) - x, y_r - x, flip, True, rep)
    gu = lib.named_u_from_flat(ents, U)
    for k in OB.ATTN_SN:
        check("u." + k, gu[k], u_r[k], False, rep)
    gg = lib.named_from_flat(ents, G)
    for k in shapes:
        check("grad." + k, gg[k], g_r[k], True, rep)
    check("dx", lib.from_device_nhwc(DX, C), dx_r, True, rep)
    check("dx-dy", lib.from_device_nhwc(DX, C) - dy, dx_r - dy, True, rep)
    rep.done()
    return rep


def test_attn_small_padded_keys():
    # H = W = 6: 36 queries and 9 keys, both padded to 32 inside the kernels
    run_attn(B=2, H=6, W=6, C=96, seed=201)


def test_attn_g_width():
    run_attn(B=2, H=8, W=8, C=192, seed=202)        # dv = 96


def test_attn_d_width_64x64():
    """The BigGAN-128 discriminator's attention shape: 64x64, C = 96."""
    run_attn(B=2, H=64, W=64, C=96, seed=203)


def test_attn_g_width_64x64():
    """The BigGAN-128 generator's attention shape: 64x64, C = 192."""
    run_attn(B=1, H=64, W=64, C=192, seed=204)
