"""GPU parity: generator / discriminator residual blocks vs the oracle.

Calls go through the C ABI (ctypes binding).  Inputs are seeded synthetic
tensors; the oracle sees exactly the values the GPU sees (bf16 inputs are
rounded before both).
"""
import numpy as np
import pytest

from oracle import blocks as OB
from oracle import layers as OL
from oracle.numerics import bf16
from paragan_2411_03999_amd import lib
from paragan_2411_03999_amd.synth import Stream, init_params, init_u

from .parity import TOL_BF16, Report, check, check_cancelling_sum, check_with_bound, need_gpu, norm_maxabs

pytestmark = pytest.mark.gpu


def run_dblock(B, H, W, cin, cout, preact, down, lsc, dtype, seed, weights="orthogonal", want_dx=True):
    torch = need_gpu()
    s = Stream(seed)
    shapes = OB.dblock_param_shapes(cin, cout, lsc)
    keys = [k for k in ("conv1.w", "conv2.w", "sc.w") if k in shapes]
    p = init_params(shapes, s, weights=weights)
    u = init_u(shapes, keys, s)
    is_bf = dtype == lib.BF16
    R = bf16 if is_bf else (lambda a: a)
    x = R(s.normal((B, H, W, cin)))
    Ho, Wo = (H // 2, W // 2) if down else (H, W)
    dy = R(s.normal((B, Ho, Wo, cout)))
    print("dblock case", dict(B=B, H=H, W=W, cin=cin, cout=cout, preact=preact, down=down, lsc=lsc,
                              dtype=dtype, seed=seed), flush=True)
    # oracle
    cfg = OB.BlockCfg(bf16=is_bf)
    y_r, u_r, cache = OB.dblock_fwd(x, p, u, cfg, preact, down, lsc)
    dx_r, g_r = OB.dblock_bwd(dy, cache, cfg, preact, down, lsc)
    # GPU
    d = lib.DBlockDesc(B, H, W, cin, cout, int(preact), int(down), int(lsc), dtype, 1, 1e-12)
    ents, npar, nu = lib.paragan_dblock_layout(d)
    assert [e["name"] for e in ents] == list(shapes)
    saved_b, ws_b = lib.paragan_dblock_sizes(d)
    ctx = lib.Context()
    P = lib.flat_from_named(ents, npar, p)
    U = lib.u_from_named(ents, nu, u)
    X = lib.to_device_nhwc(x, dtype)
    Y = lib.empty_nhwc(B, Ho, Wo, cout, dtype)
    saved = lib.workspace(saved_b)
    ws = lib.workspace(ws_b)
    lib.paragan_dblock_fwd(ctx, d, P, U, X, Y, saved, ws)
    DY = lib.to_device_nhwc(dy, dtype)
    DX = lib.empty_nhwc(B, H, W, cin, dtype) if want_dx else None
    G = torch.zeros(npar, dtype=torch.float32, device="cuda")
    lib.paragan_dblock_bwd(ctx, d, P, X, saved, DY, DX, G, ws)
    torch.cuda.synchronize()
    rep = Report()
    check("y", lib.from_device_nhwc(Y, cout), y_r, is_bf, rep)
    gu = lib.named_u_from_flat(ents, U)
    for k in keys:
        check("u." + k, gu[k], u_r[k], False, rep)
    gg = lib.named_from_flat(ents, G)
    # dh = (conv2^T dc2) * [h > 0]: where |h| is within fp32 summation error
    # of zero the two sides may disagree on the mask; bound what that moves
    b_dh = dblock_mask_bound(cache, dy, down)
    for k in shapes:
        if k == "conv1.w":
            bw = OL.conv2d_wgrad(b_dh, np.abs(cache["a0"]), 3)
            check_with_bound("grad." + k, gg[k], g_r[k], np.abs(bw) / cache["st"]["conv1.w"][2],
                             is_bf, rep)
        else:
            check("grad." + k, gg[k], g_r[k], is_bf, rep)
    if want_dx:
        bdx = OL.conv2d_dgrad(b_dh, np.abs(cache["w1"]))
        check_with_bound("dx", lib.from_device_nhwc(DX, cin), dx_r, bdx, is_bf, rep)
    rep.done()
    return rep


def dblock_mask_bound(cache, dy, down):
    """|change of dh| allowed by ReLU-mask ambiguity of h, elementwise."""
    dc2 = OL.avgpool2_bwd(dy) if down else dy
    da = OL.conv2d_dgrad(dc2, cache["w2"])
    absum = OL.conv2d(np.abs(cache["a0"]), np.abs(cache["w1"]))     # sum |a w|
    ambiguous = np.abs(cache["h"]) <= 2.0 ** -16 * absum
    return np.where(ambiguous, np.abs(da), 0.0)


@pytest.mark.parametrize("preact,down,lsc", [(True, True, True), (False, True, True),
                                             (True, False, True), (True, False, False)])
def test_dblock_bf16_ragged(preact, down, lsc):
    cin, cout = (40, 40) if not lsc else (24, 40)
    run_dblock(B=3, H=10, W=10, cin=cin, cout=cout, preact=preact, down=down, lsc=lsc,
               dtype=lib.BF16, seed=101)


def test_dblock_f32_small():
    run_dblock(B=2, H=6, W=6, cin=20, cout=36, preact=True, down=True, lsc=True, dtype=lib.F32,
               seed=102, weights="gaussian")


def test_dblock_bf16_wide_channels():
    # N = 192 / 384 exercise the 96-wide and 128-wide MFMA tile shapes
    run_dblock(B=2, H=8, W=8, cin=192, cout=384, preact=True, down=True, lsc=True, dtype=lib.BF16,
               seed=103)


def test_dblock_config2_full():
    """BigGAN D block, batch 64, 256 -> 512 channels, 32x32 -> 16x16, bf16."""
    run_dblock(B=64, H=32, W=32, cin=256, cout=512, preact=True, down=True, lsc=True, dtype=lib.BF16,
               seed=1002)


# ----------------------------------------------------------------- G block
def run_gblock(B, H, W, cin, cout, dc, dtype, seed, weights="orthogonal", n_classes=None):
    torch = need_gpu()
    s = Stream(seed)
    shapes = OB.gblock_param_shapes(cin, cout, dc)
    p = init_params(shapes, s, weights=weights)
    u = init_u(shapes, OB.GBLOCK_SN, s)
    is_bf = dtype == lib.BF16
    R = bf16 if is_bf else (lambda a: a)
    x = R(s.normal((B, H, W, cin)))
    if n_classes:
        emb = s.normal((n_classes, dc))
        cond = emb[s.labels(B, n_classes)]
    else:
        cond = s.normal((B, dc))
    cond = cond.astype(np.float32).astype(np.float64)
    dy = R(s.normal((B, 2 * H, 2 * W, cout)))
    print("gblock case", dict(B=B, H=H, W=W, cin=cin, cout=cout, dc=dc, dtype=dtype, seed=seed), flush=True)
    cfg = OB.BlockCfg(bf16=is_bf)
    y_r, u_r, cache = OB.gblock_fwd(x, cond, p, u, cfg)
    dx_r, dc_r, g_r = OB.gblock_bwd(dy, cache, cfg)
    sens = conv1_rounding_sensitivity(x, cond, p, u, dy, cfg, g_r, dx_r, dc_r, seed) if is_bf else {}
    d = lib.GBlockDesc(B, H, W, cin, cout, dc, dtype, 1, 1e-5, 1e-12)
    ents, npar, nu = lib.paragan_gblock_layout(d)
    assert [e["name"] for e in ents] == list(shapes)
    saved_b, ws_b = lib.paragan_gblock_sizes(d)
    ctx = lib.Context()
    P = lib.flat_from_named(ents, npar, p)
    U = lib.u_from_named(ents, nu, u)
    X = lib.to_device_nhwc(x, dtype)
    COND = torch.from_numpy(cond.astype(np.float32)).cuda()
    Y = lib.empty_nhwc(B, 2 * H, 2 * W, cout, dtype)
    saved = lib.workspace(saved_b)
    ws = lib.workspace(ws_b)
    lib.paragan_gblock_fwd(ctx, d, P, U, X, COND, Y, saved, ws)
    DY = lib.to_device_nhwc(dy, dtype)
    DX = lib.empty_nhwc(B, H, W, cin, dtype)
    DC = torch.zeros((B, dc), dtype=torch.float32, device="cuda")
    G = torch.zeros(npar, dtype=torch.float32, device="cuda")
    lib.paragan_gblock_bwd(ctx, d, P, X, COND, saved, DY, DX, DC, G, ws)
    torch.cuda.synchronize()
    rep = Report()
    check("y", lib.from_device_nhwc(Y, cout), y_r, is_bf, rep)
    gu = lib.named_u_from_flat(ents, U)
    for k in OB.GBLOCK_SN:
        check("u." + k, gu[k], u_r[k], False, rep)
    gg = lib.named_from_flat(ents, G)

    def chk(name, got, ref):
        if name in sens:
            # bf16: conv1 runs as sub-pixel 2x2 filters whose taps sum 3x3
            # taps and round once; cBN2's ReLU masks near zero may flip
            assert np.all(np.isfinite(got)), name
            rep.add(name, norm_maxabs(got, ref), max(TOL_BF16, 3 * sens[name]))
            rep.err[name + ".sens"] = sens[name]
        else:
            check(name, got, ref, is_bf, rep)

    for k in shapes:
        if k == "conv1.b":
            # conv1's bias feeds a batch-statistics BN: its gradient is
            # identically zero and both sides return summation noise
            l1 = np.abs(cache_dh1(cache, dy, cfg)).sum(axis=(0, 1, 2))
            check_cancelling_sum("grad." + k, gg[k], g_r[k], l1, is_bf, rep)
        else:
            chk("grad." + k, gg[k], g_r[k])
    chk("dx", lib.from_device_nhwc(DX, cin), dx_r)
    chk("dcond", DC.cpu().numpy(), dc_r)
    rep.done()
    return rep


def conv1_rounding_sensitivity(x, cond, p, u, dy, cfg, g_r, dx_r, dc_r, seed):
    """The oracle's own movement (max-abs metric) when conv1's filter moves
    by the rounding of the GPU's sub-pixel form: each 2x2 sub-pixel tap sums
    up to four 3x3 taps and is rounded to bf16 once (relative error up to
    2^-8); moving each 3x3 tap by a relative uniform +-2^-7 covers that."""
    rng = np.random.default_rng(seed)
    p2 = dict(p)
    p2["conv1.w"] = p["conv1.w"] * (1 + 2.0 ** -7 * rng.uniform(-1, 1, p["conv1.w"].shape))
    _, _, cache2 = OB.gblock_fwd(x, cond, p2, u, cfg)
    dx2, dc2, g2 = OB.gblock_bwd(dy, cache2, cfg)
    out = {"grad." + k: norm_maxabs(g2[k], g_r[k]) for k in g_r}
    out["dx"] = norm_maxabs(dx2, dx_r)
    out["dcond"] = norm_maxabs(dc2, dc_r)
    return out


def cache_dh1(cache, dy, cfg):
    """The oracle's gradient at conv1's output (the terms of conv1.b's sum)."""
    from oracle import layers as L
    from oracle.numerics import rounder
    da2 = L.conv2d_dgrad(dy, cache["w2"])
    dh1, _, _ = L.cbn_bwd(da2 * (cache["bn2"] > 0), cache["c2"])
    return rounder(cfg.bf16)(dh1)


def test_gblock_config1_f32():
    """BigGAN G block, fp32, batch 4, 64 -> 64, 8x8 -> 16x16, cBN from a 128-d
    class embedding over 10 classes, orthogonal weights, 1 power iteration."""
    run_gblock(B=4, H=8, W=8, cin=64, cout=64, dc=128, dtype=lib.F32, seed=1001, n_classes=10)


def test_gblock_config1_f32_gaussian_148():
    # Gaussian weights (sigma != 1 so a missing SN shows) and the 148-d cond
    run_gblock(B=4, H=8, W=8, cin=64, cout=64, dc=148, dtype=lib.F32, seed=1011, weights="gaussian")


def test_gblock_bf16_ragged():
    run_gblock(B=3, H=5, W=7, cin=40, cout=24, dc=20, dtype=lib.BF16, seed=104)


def test_gblock_bf16_wide():
    run_gblock(B=2, H=4, W=4, cin=384, cout=192, dc=148, dtype=lib.BF16, seed=105)


def test_gblock_biggan128_last_block():
    """BigGAN-128's last G block, 192 -> 96 channels, 64x64 -> 128x128, bf16,
    batch 2: the 96-channel kernels of the full model (its conv1 as four
    sub-pixel convs over the 64x64 source, conv2 a 3x3 conv over four-row
    tiles of the 128-wide image) at their real image shapes."""
    run_gblock(B=2, H=64, W=64, cin=192, cout=96, dc=148, dtype=lib.BF16, seed=106)


def test_dblock_biggan128_first_resolution():
    """A 96 -> 96 channel D block at 128x128 -> 64x64, bf16, batch 2: the
    stride-2 conv2 and its data gradient as four sub-pixel 2x2 convs with 96
    output channels over the 64x64 grid, the shapes of BigGAN-128's first D
    block after its image layer."""
    run_dblock(B=2, H=128, W=128, cin=96, cout=96, preact=True, down=True, lsc=True, dtype=lib.BF16,
               seed=107)


def test_dblock_biggan128_second_resolution():
    """BigGAN-128's second D block, 96 -> 192 channels, 64x64 -> 32x32, bf16,
    batch 2: its stride-2 conv2 with 192 output channels over four-row tiles
    of the 32-wide output."""
    run_dblock(B=2, H=64, W=64, cin=96, cout=192, preact=True, down=True, lsc=True, dtype=lib.BF16,
               seed=108)


def test_dblock_deep_resolution_768():
    """A 768-channel D block at 8x8 (no pooling, identity skip), bf16, batch
    192: 12288-pixel convs with 768 outputs, the shape class of BigGAN-128's
    deep layers whose tiles fill the CUs in whole rounds only at 192 x 256."""
    run_dblock(B=192, H=8, W=8, cin=768, cout=768, preact=True, down=False, lsc=False, dtype=lib.BF16,
               seed=109)
