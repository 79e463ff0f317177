"""GPU parity: the asynchronous update scheme (Numerical Optimizations,
"Asynchronous Update Scheme") through paragan_async_step.

* The iteration equals its pieces bit for bit: the generator half equals
  paragan_g_sample + paragan_g_step of batch n_D B against a copy of D taken
  before the call, and the discriminator half equals n_D paragan_d_step
  calls on the slices of the sample buffer the call was given -- though the
  two halves ran concurrently on two streams -- and two runs from one state
  are bit-identical.
* It matches the oracle's sequential emulation (oracle/biggan.py,
  async_step): element-wise at the 2e-2 bar on the minimal network, and at
  the network composition bar (tests/test_gpu_train_step.py explains it) on
  the small network and on BigGAN-128.
The buffer of previous samples both sides start from is synthetic (images
0.5 U + 0.25, as a generator's differ in statistics from the real ones).
"""
import ctypes as C

import numpy as np
import pytest

from oracle import biggan as O
from paragan_2411_03999_amd import lib

from .parity import TOL_BF16, Report, biggan_desc, check, context, harvest, need_gpu, norm_maxabs, rel_l2
from .test_gpu_train_step import (TOL_NET, check_grads, check_update, dev, f32, hparams, loss_err, make_nets,
                                  minimal_arch, small_arch)

pytestmark = pytest.mark.gpu


def async_inputs(torch, s, a, B, n_D):
    xs = [s.uniform((B, a.img, a.img, 3)).astype(np.float32) for _ in range(n_D)]
    yrs = [s.labels(B, a.n_classes) for _ in range(n_D)]
    z = f32({"z": s.normal((n_D * B, a.dz))})["z"]
    y = s.labels(n_D * B, a.n_classes)
    img = (0.5 * s.uniform((n_D * B, a.img, a.img, 3)) + 0.25).astype(np.float32)
    lab = s.labels(n_D * B, a.n_classes)
    host = dict(xs=xs, yrs=yrs, z=z, y=y, img=img, lab=lab)
    keep = dict(xs=[dev(torch, v) for v in xs], yrs=[dev(torch, v) for v in yrs],
                z=dev(torch, z.astype(np.float32)), y=dev(torch, y))
    return host, keep


class Buffers:
    """img_buff / lab_buff / pred_buff on the device, and the call's inputs."""

    def __init__(self, torch, keep, host, n_D):
        self.img = dev(torch, host["img"])
        self.lab = dev(torch, host["lab"])
        self.pred = torch.full((host["lab"].shape[0],), float("nan"), dtype=torch.float32, device="cuda")
        arr = lambda lst: (C.c_void_p * n_D)(*[t.data_ptr() for t in lst])
        self.inp = lib.AsyncInputs(arr(keep["xs"]), arr(keep["yrs"]), keep["z"].data_ptr(), keep["y"].data_ptr(),
                                   self.img.data_ptr(), self.lab.data_ptr(), self.pred.data_ptr())


def run_async(torch, ctx, d, G, D, buf, n_D, ws):
    losses = (C.c_float * (n_D + 1))()
    rc = lib.paragan_async_step(ctx, d, G.state, D.state, buf.inp, n_D, ws, losses)
    assert rc == lib.OK, lib.load().paragan_last_error(ctx.h)
    torch.cuda.synchronize()
    return list(losses)


def test_async_step_equals_its_pieces_and_is_deterministic():
    torch = need_gpu()
    a, B, n_D = small_arch(), 4, 2
    hp = hparams()
    d, s, _, _, G0, D0 = make_nets(torch, a, B, 421, hp)
    host, keep = async_inputs(torch, s, a, B, n_D)
    ctx = context()
    ws = lib.workspace(lib.paragan_async_ws_size(d, n_D))
    runs = []
    for _ in range(2):
        G, D = G0.clone(torch), D0.clone(torch)
        buf = Buffers(torch, keep, host, n_D)
        losses = run_async(torch, ctx, d, G, D, buf, n_D, ws)
        runs.append((losses, G, D, buf))
    (l1, G1, D1, b1), (l2, G2, D2, b2) = runs
    assert l1 == l2, (l1, l2)
    for X, Y in ((G1, G2), (D1, D2)):
        for t1, t2 in zip(X.tensors(), Y.tensors()):
            assert torch.equal(t1, t2)
    for t1, t2 in ((b1.img, b2.img), (b1.lab, b2.lab), (b1.pred, b2.pred)):
        assert torch.equal(t1, t2)
    # the generator half: g_sample + g_step of batch n_D B against a copy of D
    dg = biggan_desc(a, n_D * B, hp)
    wsg = lib.workspace(lib.paragan_train_step_ws_size(dg))
    Gs, Gp, Dsnap = G0.clone(torch), G0.clone(torch), D0.clone(torch)
    img = torch.empty((n_D * B, a.img, a.img, 3), dtype=torch.float32, device="cuda")
    ctx.check(lib.paragan_g_sample(ctx, dg, Gs.state, keep["z"], keep["y"], img, wsg))
    loss = (C.c_float * 1)()
    ctx.check(lib.paragan_g_step(ctx, dg, Gp.state, Dsnap.state, keep["z"], keep["y"], wsg, loss))
    torch.cuda.synchronize()
    assert l1[n_D] == loss[0], (l1, loss[0])
    assert torch.equal(b1.img, img) and torch.equal(b1.lab, keep["y"])
    for t1, t2 in zip(G1.tensors(), Gp.tensors()):
        assert torch.equal(t1, t2)
    assert G1.state.opt_t == Gp.state.opt_t
    # L_G is minus the mean of the snapshot's predictions in pred_buff
    pred = b1.pred.cpu().numpy().astype(np.float64)
    assert abs(-pred.mean() - l1[n_D]) <= 1e-6 * max(1.0, abs(l1[n_D]))
    # the discriminator half: n_D d_steps on the slices of the given buffer
    Dp = D0.clone(torch)
    wsd = lib.workspace(lib.paragan_train_step_ws_size(d))
    prev_img, prev_lab = dev(torch, host["img"]), dev(torch, host["lab"])
    for k in range(n_D):
        sl = slice(k * B, (k + 1) * B)
        ctx.check(lib.paragan_d_step(ctx, d, Dp.state, keep["xs"][k], keep["yrs"][k], prev_img[sl].contiguous(),
                                     prev_lab[sl].contiguous(), wsd, loss))
        torch.cuda.synchronize()
        assert l1[k] == loss[0], (k, l1, loss[0])
    harvest(ctx)
    for t1, t2 in zip(D1.tensors(), Dp.tensors()):
        assert torch.equal(t1, t2)
    assert D1.state.opt_t == Dp.state.opt_t == n_D


@pytest.mark.parametrize("arch,B,n_D", [("minimal", 8, 2), ("small", 4, 2), ("biggan128", 1, 2)])
def test_async_step_vs_oracle(arch, B, n_D):
    """L_D of each step, L_G, the last D step's and the G step's gradients,
    both updates, the new sample and prediction buffers (labels exactly)."""
    torch = need_gpu()
    a = {"minimal": minimal_arch, "small": small_arch, "biggan128": O.biggan128}[arch]()
    hp = hparams()
    d, s, (gp, gu, glay, gsn, optG), (dp, du, dlay, dsn, optD), G, D = make_nets(torch, a, B, 422, hp,
                                                                                 smooth_opt=True)
    host, keep = async_inputs(torch, s, a, B, n_D)
    print("async case", arch, B, n_D, flush=True)
    ctx = context()
    ws = lib.workspace(lib.paragan_async_ws_size(d, n_D))
    buf = Buffers(torch, keep, host, n_D)
    losses = run_async(torch, ctx, d, G, D, buf, n_D, ws)
    harvest(ctx)
    d_in = [(host["xs"][k].astype(np.float64), host["yrs"][k]) for k in range(n_D)]
    Gr, Dr, loss_r, img_r, lab_r, pred_r, gd_r, gg_r = O.async_step(
        a, hp, (gp, gu), (dp, du), optG, optD, d_in, (host["z"], host["y"]), host["img"].astype(np.float64),
        host["lab"])
    rep = Report()
    strict = arch == "minimal"
    # The first D step and the G half start from the common state and take
    # the block bar.  A later D step starts from D after an Adam update with
    # beta1 = 0, which early on is close to lr * sign(g) per element: where a
    # gradient element is near zero its sign, and so the update, comes out
    # either way on a deep network (the oracle's own spread is 4-12 %), so
    # what depends on it takes the composition bar there.
    for k in range(n_D + 1):
        later = 0 < k < n_D and not strict
        rep.add("loss%d" % k, loss_err(losses[k], loss_r[k]), TOL_NET if later else TOL_BF16)
    check_grads(rep, "gD.", a, lib.named_from_flat(D.ents, D.G), gd_r, dlay, False, strict)
    check_grads(rep, "gG.", a, lib.named_from_flat(G.ents, G.G), gg_r, glay, True, strict)
    check_update(rep, "stepD.", a, lib.named_from_flat(D.ents, D.P), dp, Dr[0], list(dlay), False, strict)
    check_update(rep, "stepG.", a, lib.named_from_flat(G.ents, G.P), gp, Gr[0], list(glay), True, strict)
    gu_new = lib.named_u_from_flat(G.ents, G.U)
    for k in gsn:
        check("uG." + k, gu_new[k], Gr[1][k], False, rep)
    du_new = lib.named_u_from_flat(D.ents, D.U)
    for k in dsn:
        if strict or n_D == 1:
            check("uD." + k, du_new[k], Dr[1][k], False, rep)
        else:
            rep.add("uD." + k + ".l2", rel_l2(du_new[k], Dr[1][k]), TOL_NET)
    img = buf.img.cpu().numpy()
    if strict:
        rep.add("img_buff", norm_maxabs(img, img_r), TOL_BF16)
        rep.add("pred_buff", norm_maxabs(buf.pred.cpu().numpy(), pred_r), TOL_BF16)
    else:
        rep.err["img_buff.maxabs"] = norm_maxabs(img, img_r)
        rep.add("img_buff.l2", rel_l2(img, img_r), TOL_NET)
        rep.add("pred_buff", loss_err(-buf.pred.cpu().numpy().mean(), -pred_r.mean()), TOL_BF16)
    assert np.array_equal(buf.lab.cpu().numpy(), lab_r)
    assert G.state.opt_t == 8 and D.state.opt_t == 7 + n_D
    rep.done()


def test_async_step_rejects_bad_arguments_before_launching():
    torch = need_gpu()
    a, B = minimal_arch(), 4
    hp = hparams()
    d, s, _, _, G, D = make_nets(torch, a, B, 423, hp)
    host, keep = async_inputs(torch, s, a, B, 1)
    ctx = context()
    ws = lib.workspace(lib.paragan_async_ws_size(d, 1))
    buf = Buffers(torch, keep, host, 1)
    keepP = G.P.clone()
    losses = (C.c_float * 2)()
    for n_D in (0, 64):
        assert lib.paragan_async_step(ctx, d, G.state, D.state, buf.inp, n_D, ws, losses) == lib.EINVAL
    bad = lib.AsyncInputs(buf.inp.x_real, buf.inp.y_real, buf.inp.z, buf.inp.y, buf.inp.img_buff, None,
                          buf.inp.pred_buff)
    assert lib.paragan_async_step(ctx, d, G.state, D.state, bad, 1, ws, losses) == lib.EINVAL
    torch.cuda.synchronize()
    assert torch.equal(keepP, G.P) and G.state.opt_t == 0
