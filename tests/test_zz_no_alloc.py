"""The allocation-free SN power iteration (paragan_sn_power_iter_noalloc,
for callers that cannot allocate) against paragan_sn_power_iter with a
workspace: the same kernels on the same inputs, so u, v and sigma must agree
bit for bit -- on two calls in a row, the second smaller, so that the
library's shared scratch array still holds the first call's contents --
and against the oracle at the fp32 bar.  A weight whose scratch would
exceed the array is refused before any work."""
import numpy as np
import pytest

from oracle import layers as L
from paragan_2411_03999_amd import lib
from paragan_2411_03999_amd.synth import Stream

from .parity import Report, check, need_gpu

pytestmark = pytest.mark.gpu


def _case(torch, rows, cols, seed):
    s = Stream(seed)
    w = (s.normal((rows, cols)) / np.sqrt(cols)).astype(np.float32)
    u0 = s.normal((rows,)).astype(np.float32)
    W = torch.from_numpy(w).cuda()
    return w, u0, W


def _outs(torch, rows, cols, u0):
    U = torch.from_numpy(u0).cuda()
    V = torch.full((cols,), float("nan"), dtype=torch.float32, device="cuda")
    S = torch.full((1,), float("nan"), dtype=torch.float32, device="cuda")
    return U, V, S


@pytest.mark.parametrize("n_iter", [1, 3])
def test_noalloc_equals_workspace_path_on_two_calls(n_iter):
    torch = need_gpu()
    ctx = lib.Context()
    # the largest BigGAN-128 SN weight (d4.conv1.w, 1536 x 3*3*768), then a
    # far smaller one (the generator's output conv, 3 x 3*3*96)
    for rows, cols, seed in ((1536, 6912, 901), (3, 864, 902)):
        print("noalloc case", dict(rows=rows, cols=cols, n_iter=n_iter), flush=True)
        w, u0, W = _case(torch, rows, cols, seed + n_iter)
        U1, V1, S1 = _outs(torch, rows, cols, u0)
        rc = lib.paragan_sn_power_iter_noalloc(ctx, W, rows, cols, U1, V1, S1, n_iter, 1e-12)
        assert rc == lib.OK, lib.load().paragan_last_error(ctx.h)
        U2, V2, S2 = _outs(torch, rows, cols, u0)
        ws = lib.workspace(lib.paragan_sn_ws_size(rows, cols))
        lib.paragan_sn_power_iter(ctx, W, rows, cols, U2, V2, S2, n_iter, 1e-12, ws)
        torch.cuda.synchronize()
        assert torch.equal(U1, U2) and torch.equal(V1, V2) and torch.equal(S1, S2)
        u_r, v_r, sig_r = L.sn_power_iter(w.astype(np.float64), u0.astype(np.float64), n_iter, 1e-12)
        rep = Report()
        check("u", U1.cpu().numpy(), u_r, False, rep)
        check("v", V1.cpu().numpy(), v_r, False, rep)
        check("sigma", S1.cpu().numpy(), np.array([sig_r]), False, rep)
        rep.done()


def test_noalloc_refuses_a_weight_beyond_its_scratch():
    """A 128 x 131072 weight needs 16 row chunks x 131072 columns of partial
    sums (8 MiB): refused with EINVAL, nothing launched, the outputs
    untouched.  (The weight pointer is a small real buffer: the call is
    refused on its sizes before anything reads it.)"""
    torch = need_gpu()
    rows, cols = 128, 1 << 17
    assert lib.paragan_sn_ws_size(rows, cols) > 4 << 20
    ctx = lib.Context()
    W = torch.zeros(16, dtype=torch.float32, device="cuda")
    U = torch.full((16,), 3.0, dtype=torch.float32, device="cuda")
    V = torch.full((16,), 3.0, dtype=torch.float32, device="cuda")
    S = torch.full((1,), 3.0, dtype=torch.float32, device="cuda")
    rc = lib.paragan_sn_power_iter_noalloc(ctx, W, rows, cols, U, V, S, 1, 1e-12)
    assert rc == lib.EINVAL
    assert b"scratch" in lib.load().paragan_last_error(ctx.h)
    torch.cuda.synchronize()
    assert bool((U == 3.0).all()) and bool((V == 3.0).all()) and float(S[0]) == 3.0
