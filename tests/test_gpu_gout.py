"""GPU parity: the generator output layer (BN -> ReLU -> SN conv3x3 to 3
channels -> tanh, fp32 arithmetic on bf16 input) vs the oracle, forward and
backward, from a few pixels up to BigGAN-128's 128x128x96 and BigGAN-512's
width."""
import numpy as np
import pytest

from oracle import biggan as O
from oracle.blocks import BlockCfg
from oracle.numerics import bf16
from paragan_2411_03999_amd import lib
from paragan_2411_03999_amd.synth import Stream, init_params, init_u

from .parity import Report, check, need_gpu, norm_maxabs, context, harvest

pytestmark = pytest.mark.gpu


def shapes_of(C):
    return {"out_bn.gain": (C,), "out_bn.bias": (C,), "out_conv.w": (3, 3, 3, C), "out_conv.b": (3,)}


def run_gout(B, H, W, C, seed):
    torch = need_gpu()
    s = Stream(seed)
    shapes = shapes_of(C)
    p = {k: np.asarray(v, np.float32).astype(np.float64)
         for k, v in init_params(shapes, s, weights="gaussian").items()}
    u = {k: np.asarray(v, np.float32).astype(np.float64) for k, v in init_u(shapes, ["out_conv.w"], s).items()}
    # a block output: per-channel offsets and scales, so BN has work to do
    x = bf16(s.normal((B, H, W, C)) * s.uniform((C,), 0.5, 2.0) + s.normal((C,)))
    dimg = s.normal((B, H, W, 3))
    print("gout case", dict(B=B, H=H, W=W, C=C, seed=seed), flush=True)
    cfg = BlockCfg(bf16=False, bn_eps=1e-5, sn_eps=1e-12, n_power_iter=1)
    img_r, u_r, cache = O.g_out_fwd(x, p, u, cfg, 1e-5)
    dx_r, g_r = O.g_out_bwd(dimg, cache)

    d = lib.GoutDesc(B, H, W, C, 1, 1e-5, 1e-12)
    assert lib.paragan_gout_check(d) == 0
    ents, npar, nu = lib.paragan_gout_layout(d)
    assert [(e["name"], tuple(e["shape"])) for e in ents] == list(shapes.items())
    sb, wb = lib.paragan_gout_sizes(d)
    ctx = context()
    P = lib.flat_from_named(ents, npar, p)
    U = lib.u_from_named(ents, nu, u)
    X = lib.to_device_nhwc(x, lib.BF16)
    IMG = torch.zeros((B, H, W, 3), dtype=torch.float32, device="cuda")
    saved, ws = lib.workspace(sb), lib.workspace(wb)
    lib.paragan_gout_fwd(ctx, d, P, U, X, IMG, saved, ws)
    DX = lib.empty_nhwc(B, H, W, C, lib.BF16)
    G = torch.zeros(npar, dtype=torch.float32, device="cuda")
    DIMG = torch.from_numpy(dimg.astype(np.float32)).cuda()
    lib.paragan_gout_bwd(ctx, d, P, X, IMG, saved, DIMG, DX, G, ws)
    torch.cuda.synchronize()
    harvest(ctx)

    rep = Report()
    check("img", IMG.cpu().numpy().astype(np.float64), img_r, False, rep)
    check("u.out_conv.w", lib.named_u_from_flat(ents, U)["out_conv.w"], u_r, False, rep)
    gg = lib.named_from_flat(ents, G)
    for k in shapes:
        check("grad." + k, gg[k], g_r[k], False, rep)
    # dx is stored in bf16.  Where the BN output sits within fp32 rounding of
    # 0 the ReLU's decision is not fixed by either side's precision: those
    # elements (expected: none or a handful) are left out and counted.
    dx = lib.from_device_nhwc(DX, C)
    bn = cache["bn"]
    sure = np.abs(bn) > 1e-5 * np.abs(bn).max()
    print("dx elements left out at the ReLU kink:", int((~sure).sum()), flush=True)
    rep.add("dx", norm_maxabs(np.where(sure, dx, 0.0), np.where(sure, dx_r, 0.0)), 2e-2)
    assert np.all(np.isfinite(dx))
    assert np.all(lib.from_device_nhwc(DX, lib.cpad(C))[..., C:] == 0), "padded channels of dx must be 0"
    rep.done()


def test_gout_tiny():
    run_gout(2, 8, 8, 8, seed=501)


def test_gout_ragged_rows_and_tiles():
    # 40 columns: one full and one partial 32-position tile per Z row; 20 rows:
    # a partial 16-row band
    run_gout(3, 20, 40, 40, seed=502)


def test_gout_column_windows():
    # 300 columns: three column windows (126, 126, 48), 100 channels (128 padded)
    run_gout(1, 6, 300, 100, seed=503)


def test_gout_biggan512_width():
    # BigGAN-512's output layer width (C = 64) at 512 columns; 17 rows leave
    # a one-row weight-gradient band
    run_gout(1, 17, 512, 64, seed=504)


def test_gout_biggan128_full():
    # BigGAN-128's output layer at its full shape (C = 96, 128 x 128), B = 2
    run_gout(2, 128, 128, 96, seed=505)

