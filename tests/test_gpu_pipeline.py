"""The host data pipeline feeding the train step (Implementation,
"Congestion-Aware Data Pipelining"): batches that arrive through the
pipeline's threads and pinned slots give the same training result, bit for
bit, as the same synthetic batches written straight to the device, whatever
the number of fetch threads."""
import ctypes as C

import numpy as np
import pytest

from paragan_2411_03999_amd import lib

from .parity import context, need_gpu
from .test_gpu_train_step import hparams, make_nets, small_arch

pytestmark = pytest.mark.gpu


def _source(a, B, seed):
    s = lib.SynthSource()
    s.seed, s.B, s.img, s.n_classes = seed, B, a.img, a.n_classes
    return s


def _inputs(torch, a, B, n_D, s):
    dev = lambda shape, dt: torch.empty(shape, dtype=dt, device="cuda")
    xs = [dev((B, a.img, a.img, 3), torch.float32) for _ in range(n_D)]
    yrs = [dev((B,), torch.int32) for _ in range(n_D)]
    zs = [torch.from_numpy(s.normal((B, a.dz)).astype(np.float32)).cuda() for _ in range(n_D)]
    yfs = [torch.from_numpy(s.labels(B, a.n_classes)).cuda() for _ in range(n_D)]
    zg = torch.from_numpy(s.normal((B, a.dz)).astype(np.float32)).cuda()
    yg = torch.from_numpy(s.labels(B, a.n_classes)).cuda()
    arr = lambda lst: (C.c_void_p * n_D)(*[t.data_ptr() for t in lst])
    inp = lib.StepInputs(arr(xs), arr(yrs), arr(zs), arr(yfs), zg.data_ptr(), yg.data_ptr())
    return inp, (xs, yrs, zs, yfs, zg, yg)


def _run(torch, a, B, n_D, steps, threads, fed):
    d, s, _, _, G, D = make_nets(torch, a, B, 431, hparams())
    inp, (xs, yrs, *_rest) = _inputs(torch, a, B, n_D, s)
    ctx = context()
    ws = lib.workspace(lib.paragan_train_step_ws_size(d))
    src = _source(a, B, 77)
    nbytes = lib.load().paragan_synth_batch_bytes(C.byref(src))
    n = B * a.img * a.img * 3
    losses = (C.c_float * (n_D + 1))()
    out = []
    if fed:
        slots = [torch.empty(nbytes, dtype=torch.uint8, pin_memory=True) for _ in range(6)]
        cfg = lib.PipelineCfg()
        cfg.min_threads, cfg.max_threads, cfg.min_depth, cfg.max_depth, cfg.window, cfg.threshold_ms = \
            threads, threads, 4, 4, 4, 1e6
        pipe = lib.Pipeline(cfg, [t.data_ptr() for t in slots], nbytes, synth=src)
    host = np.zeros(nbytes, np.uint8)
    seq = 0
    for _ in range(steps):
        held = []
        for k in range(n_D):
            if fed:
                rc, got, slot = pipe.next(60000)
                assert rc == lib.OK and got == seq, (rc, got, seq, pipe.error())
                buf = slots[slot]
                xs[k].copy_(buf[:4 * n].view(torch.float32).view(xs[k].shape), non_blocking=True)
                yrs[k].copy_(buf[4 * n:4 * n + 4 * B].view(torch.int32), non_blocking=True)
                held.append(slot)
            else:
                assert lib.load().paragan_synth_fetch(C.byref(src), seq, host.ctypes.data, nbytes) == 0
                xs[k].copy_(torch.from_numpy(host[:4 * n].view(np.float32).reshape(xs[k].shape)))
                yrs[k].copy_(torch.from_numpy(host[4 * n:4 * n + 4 * B].view(np.int32)))
            seq += 1
        rc = lib.paragan_train_step(ctx, d, G.state, D.state, inp, n_D, ws, losses)
        assert rc == lib.OK, lib.load().paragan_last_error(ctx.h)
        torch.cuda.synchronize()
        for slot in held:
            assert pipe.release(slot) == lib.OK
        out.append(list(losses))
    if fed:
        pipe.close()
    return out, G, D


@pytest.mark.parametrize("threads", [1, 3])
def test_pipeline_fed_steps_equal_direct_feed(threads):
    torch = need_gpu()
    a, B, n_D = small_arch(), 4, 2
    ref, G0, D0 = _run(torch, a, B, n_D, 3, 1, fed=False)
    got, G1, D1 = _run(torch, a, B, n_D, 3, threads, fed=True)
    assert got == ref, (got, ref)
    for X, Y in ((G0, G1), (D0, D1)):
        for t0, t1 in zip(X.tensors(), Y.tensors()):
            assert torch.equal(t0, t1)
