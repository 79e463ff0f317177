"""Every kernel-template instance that the benchmark's BigGAN-128 step
(batch 256, two D steps per G step) launches -- convolutions, weight
gradients, attention -- must have been launched by a parity test of this
session.  Tile choice depends on the GEMM shape, so a parity test at another
shape does not by itself cover the instance the benchmark times.

Runs after the other GPU tests (pytest collects this file after them) and
only when the whole GPU parity suite ran in the same session."""
import ctypes as C
import os

import pytest

from paragan_2411_03999_amd import lib

from .parity import SEEN, context, need_gpu

pytestmark = pytest.mark.gpu

PARITY_FILES = ("test_gpu_blocks.py", "test_gpu_attention.py", "test_gpu_gout.py", "test_gpu_sn.py",
                "test_gpu_train_step.py")


def _full_suite_ran(session):
    here = os.path.dirname(os.path.abspath(__file__))
    ran = {os.path.basename(str(it.fspath)) for it in session.items}
    if not all(f in ran for f in PARITY_FILES):
        return False
    for f in PARITY_FILES:
        src = open(os.path.join(here, f)).read()
        n_defs = src.count("\ndef test_")
        if sum(1 for it in session.items if os.path.basename(str(it.fspath)) == f and
               it.originalname.startswith("test_")) < n_defs:
            return False
    return True


def test_benchmark_instances_are_under_parity(request):
    torch = need_gpu()
    if not _full_suite_ran(request.session):
        pytest.skip("needs the whole GPU parity suite in the same session")
    import bench
    B, n_D = 256, 2
    d = bench.make_desc(lib, "biggan128", B)
    gen = torch.Generator(device="cuda").manual_seed(7)
    nets = [bench.device_net(torch, lib, *lib.paragan_net_layout(d, w), gen) for w in (0, 1)]
    img = d.img
    keep = []
    for _ in range(n_D):
        keep += [torch.rand((B, img, img, 3), device="cuda", generator=gen) * 2 - 1,
                 torch.randint(0, d.n_classes, (B,), device="cuda", dtype=torch.int32, generator=gen),
                 torch.randn((B, d.dz), device="cuda", generator=gen),
                 torch.randint(0, d.n_classes, (B,), device="cuda", dtype=torch.int32, generator=gen)]
    zg = torch.randn((B, d.dz), device="cuda", generator=gen)
    yg = torch.randint(0, d.n_classes, (B,), device="cuda", dtype=torch.int32, generator=gen)
    arr = lambda i: (C.c_void_p * n_D)(*[keep[4 * k + i].data_ptr() for k in range(n_D)])
    inp = lib.StepInputs(arr(0), arr(1), arr(2), arr(3), zg.data_ptr(), yg.data_ptr())
    ws = lib.workspace(lib.paragan_train_step_ws_size(d))
    ctx = context()
    losses = (C.c_float * (n_D + 1))()
    rc = lib.paragan_train_step(ctx, d, nets[0]["state"], nets[1]["state"], inp, n_D, ws, losses)
    assert rc == lib.OK, lib.load().paragan_last_error(ctx.h)
    bench_names = {st["name"] for st in lib.paragan_profile_read(ctx)}
    print("benchmark instances:", sorted(bench_names), flush=True)
    missing = sorted(bench_names - SEEN)
    assert not missing, "benchmark kernel instances no parity test launched: %s" % missing
