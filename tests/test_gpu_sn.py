"""GPU parity: paragan_sn_power_iter (the spectral-norm power iteration of
one weight viewed as (rows, cols)) vs the oracle, at BigGAN-128's real
weight shapes and the degenerate ones, for one and several iterations."""
import numpy as np
import pytest

from oracle import layers as L
from paragan_2411_03999_amd import lib
from paragan_2411_03999_amd.synth import Stream

from .parity import Report, check, need_gpu

pytestmark = pytest.mark.gpu

SHAPES = [
    (1, 1), (1, 7), (5, 1), (3, 864),      # degenerate and the G output conv (3 x 3*3*96)
    (96, 148), (1536, 148),                # conditional-BN linears
    (512, 2304), (192, 1728),              # config-2 conv1, a 64x64 G conv
    (1536, 13824),                         # the largest 3x3 conv (1536 -> 1536)
    (1000, 1536), (24, 192),               # class embedding, attention theta
    (24576, 20), (3000, 5), (1000, 70),    # the z linear (16*1536 x 20), narrow tiles with idle lanes
]


@pytest.mark.parametrize("rows,cols", SHAPES)
@pytest.mark.parametrize("n_iter", [1, 3])
def test_sn_power_iter(rows, cols, n_iter):
    torch = need_gpu()
    s = Stream(500 + rows + 7 * cols + n_iter)
    w = (s.normal((rows, cols)) / np.sqrt(cols)).astype(np.float32)
    u0 = s.normal((rows,)).astype(np.float32)
    print("sn case", dict(rows=rows, cols=cols, n_iter=n_iter), flush=True)
    u_r, v_r, sig_r = L.sn_power_iter(w.astype(np.float64), u0.astype(np.float64), n_iter, 1e-12)
    W = torch.from_numpy(w).cuda()
    U = torch.from_numpy(u0).cuda()
    V = torch.zeros(cols, dtype=torch.float32, device="cuda")
    S = torch.zeros(1, dtype=torch.float32, device="cuda")
    ws = lib.workspace(lib.paragan_sn_ws_size(rows, cols))
    ctx = lib.Context()
    lib.paragan_sn_power_iter(ctx, W, rows, cols, U, V, S, n_iter, 1e-12, ws)
    torch.cuda.synchronize()
    rep = Report()
    check("u", U.cpu().numpy(), u_r, False, rep)
    check("v", V.cpu().numpy(), v_r, False, rep)
    check("sigma", S.cpu().numpy(), np.array([sig_r]), False, rep)
    rep.done()


def test_sn_power_iter_zero_weight():
    """W = 0: both normalisations hit the eps floor, u and v become 0 and
    sigma = 0 (the oracle's definition), with nothing non-finite."""
    torch = need_gpu()
    rows, cols = 64, 288
    u0 = Stream(77).normal((rows,)).astype(np.float32)
    u_r, v_r, sig_r = L.sn_power_iter(np.zeros((rows, cols)), u0.astype(np.float64), 1, 1e-12)
    W = torch.zeros((rows, cols), dtype=torch.float32, device="cuda")
    U = torch.from_numpy(u0).cuda()
    V = torch.full((cols,), 7.0, dtype=torch.float32, device="cuda")
    S = torch.full((1,), 7.0, dtype=torch.float32, device="cuda")
    ws = lib.workspace(lib.paragan_sn_ws_size(rows, cols))
    ctx = lib.Context()
    lib.paragan_sn_power_iter(ctx, W, rows, cols, U, V, S, 1, 1e-12, ws)
    torch.cuda.synchronize()
    assert np.array_equal(U.cpu().numpy(), u_r.astype(np.float32))
    assert np.array_equal(V.cpu().numpy(), v_r.astype(np.float32))
    assert S.item() == sig_r == 0.0
