"""GPU parity of every block of BigGAN-128 in its place in a training step.

The oracle runs BigGAN-128's generator step and discriminator step (batch 2,
Evaluation "Experiment Setup"; bf16 storage) and records, for each residual
block and attention block, the input the block sees there, its conditioning,
its parameters and SN state, and the output gradient the backward pass hands
it.  The GPU then runs that block from exactly those values (teacher forcing:
oracle values go to the GPU, never the other way) and is held element by
element to the 2e-2 bar plus the bound on ReLU decisions within summation
error of zero (tests/bounds.py).

Why per block: across a whole deep network every block's input already
carries the rounding of the blocks before it, and the oracle itself, rerun
with noise of 2^-20 of a value before each bf16 rounding (the size of a
summation-order difference), moves its BigGAN-128 generator gradients by
4-12 % in relative L2; the composition of the blocks is checked at the
network level in tests/test_gpu_train_step.py.
"""
import numpy as np
import pytest

from oracle import biggan as O
from oracle import blocks as OB
from oracle import layers as OL
from oracle.numerics import rounder
from paragan_2411_03999_amd import lib
from paragan_2411_03999_amd.synth import Stream, init_params, init_u

from .parity import need_gpu
from .test_gpu_attention import compare_attn
from .test_gpu_blocks import compare_dblock, compare_gblock

pytestmark = pytest.mark.gpu


def f32(d):
    return {k: np.asarray(v, np.float32).astype(np.float64) for k, v in d.items()}


def sub(d, prefix):
    return {k[len(prefix):]: v for k, v in d.items() if k.startswith(prefix)}


def nets(a, seed):
    s = Stream(seed)
    glay, gsn = O.g_layout(a)
    dlay, dsn = O.d_layout(a)
    gp, gu = f32(init_params(glay, s, weights="gaussian")), f32(init_u(glay, gsn, s))
    dp, du = f32(init_params(dlay, s, weights="gaussian")), f32(init_u(dlay, dsn, s))
    return s, gp, gu, dp, du


def d_records(a, hp, dp, du, x, y, dout_fn):
    """D forward on x, then its backward from dout_fn(logits), recording
    (kind, block index, cache, output gradient) of every block."""
    R = rounder(hp.bf16)
    cfg = hp.block()
    out, _, c = O.d_fwd(a, hp, dp, du, x, y)
    dout = dout_fn(out)
    dhs = dout[:, None] * (c["wh"][0][None, :] + c["ey"])
    dh = R(dhs[:, None, None, :] * (c["h"] > 0))
    blocks = O.d_blocks(a)
    recs = []
    for kind, j, cb in reversed(c["caches"]):
        recs.append((kind, j, cb, dh))
        if kind == "a":
            dh, _ = OB.attn_bwd(dh, cb, cfg)
        else:
            cin, cout, pre, down, lsc, att = blocks[j]
            dh, _ = OB.dblock_bwd(dh, cb, cfg, pre, down, lsc, dx_f32=(j == 0))
    return recs


def check_d_records(a, recs, dp, du):
    blocks = O.d_blocks(a)
    for kind, j, cb, dy in recs:
        if kind == "a":
            print("D attention after block", j, flush=True)
            compare_attn(cb["x"], sub(dp, "attn."), sub(du, "attn."), dy)
        else:
            cin, cout, pre, down, lsc, att = blocks[j]
            print("D block", j, flush=True)
            compare_dblock(cb["x"], sub(dp, "d%d." % j), sub(du, "d%d." % j), dy, cout, pre, down, lsc, lib.BF16)


def test_biggan128_d_step_blocks_in_place():
    """Every D block and the D attention block of a BigGAN-128 D step on
    2 real + 2 fake images."""
    need_gpu()
    a, hp = O.biggan128(), O.HParams()
    s, gp, gu, dp, du = nets(a, 501)
    B = 2
    xr = s.uniform((B, a.img, a.img, 3)).astype(np.float32).astype(np.float64)
    xf = (0.5 * s.uniform((B, a.img, a.img, 3)) + 0.25).astype(np.float32).astype(np.float64)
    yr, yf = s.labels(B, a.n_classes), s.labels(B, a.n_classes)

    def dout(out):
        _, dr, df = OL.hinge_d(out[:B], out[B:])
        return np.concatenate([dr, df])

    recs = d_records(a, hp, dp, du, np.concatenate([xr, xf]), np.concatenate([yr, yf]), dout)
    check_d_records(a, recs, dp, du)


def test_biggan128_g_step_blocks_in_place():
    """Every G block, the G attention block, and every D block and the D
    attention block on the input-gradient path, of a BigGAN-128 G step on
    2 samples."""
    need_gpu()
    a, hp = O.biggan128(), O.HParams()
    s, gp, gu, dp, du = nets(a, 502)
    B = 2
    R = rounder(hp.bf16)
    cfg = hp.block()
    z = s.normal((B, a.dz)).astype(np.float32).astype(np.float64)
    y = s.labels(B, a.n_classes)
    img, _, gc = O.g_fwd(a, hp, gp, gu, z, y)

    def dout(out):
        _, d = OL.hinge_g(out)
        return d

    drecs = d_records(a, hp, dp, du, img, y, dout)
    # the image gradient out of D's first block, then G's backward replayed
    cin, cout, pre, down, lsc, att = O.d_blocks(a)[0]
    cb0, dy0 = next((cb, dy) for kind, j, cb, dy in drecs if kind == "d" and j == 0)
    dimg, _ = OB.dblock_bwd(dy0, cb0, cfg, pre, down, lsc, dx_f32=True)
    dh, _ = O.g_out_bwd(dimg, gc)
    dh = R(dh)
    grecs, i = [], a.n_g - 1
    for kind, cb in reversed(gc["caches"]):
        grecs.append((kind, i, cb, dh))
        if kind == "a":
            dh, _ = OB.attn_bwd(dh, cb, cfg)
        else:
            dh, _, _ = OB.gblock_bwd(dh, cb, cfg)
            i -= 1
    for kind, i, cb, dy in grecs:
        if kind == "a":
            print("G attention", flush=True)
            compare_attn(cb["x"], sub(gp, "attn."), sub(gu, "attn."), dy)
        else:
            print("G block", i, flush=True)
            compare_gblock(cb["x"], cb["cond"], sub(gp, "g%d." % i), sub(gu, "g%d." % i), dy, lib.BF16)
    check_d_records(a, drecs, dp, du)
