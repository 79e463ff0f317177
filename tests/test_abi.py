"""C-ABI checks that need no GPU: the library loads, exports every function
include/paragan.h declares, validates arguments on the host, and describes
parameter layouts that match the oracle's (names, shapes, order)."""
import ctypes as C
import os
import re

import pytest

from oracle import biggan as O
from oracle import blocks as OB
from paragan_2411_03999_amd import lib

from .parity import biggan_desc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lib.LIB_PATH):
        from paragan_2411_03999_amd.build import build
        build()
    return lib.load()


def header_functions():
    src = open(os.path.join(ROOT, "include", "paragan.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(paragan_\w+)\s*\(", src)))


def test_exports_every_declared_function(L):
    names = header_functions()
    assert len(names) >= 25
    for n in names:
        assert hasattr(L, n), n
        assert n in lib.exported_symbols(), n


def test_sn_validation(L):
    assert L.paragan_sn_check(1536, 13824, 1, 1e-12) == lib.OK
    assert L.paragan_sn_check(0, 4, 1, 1e-12) == lib.EINVAL
    assert L.paragan_sn_check(4, 4, 0, 1e-12) == lib.EINVAL
    assert L.paragan_sn_check(4, 4, 1, 0.0) == lib.EINVAL
    assert L.paragan_sn_check(1 << 31, 4, 1, 1e-12) == lib.EINVAL


def test_cpad():
    assert [lib.cpad(c) for c in (1, 3, 32, 33, 96, 148)] == [32, 32, 32, 64, 96, 160]


def test_gblock_validation(L):
    good = lib.GBlockDesc(4, 8, 8, 64, 64, 128, lib.F32, 1, 1e-5, 1e-12)
    assert lib.paragan_gblock_check(good) == lib.OK
    for field, bad in [("B", 0), ("cin", 0), ("dtype", 7), ("n_power_iter", 0), ("bn_eps", 0.0)]:
        d = lib.GBlockDesc(4, 8, 8, 64, 64, 128, lib.F32, 1, 1e-5, 1e-12)
        setattr(d, field, bad)
        assert lib.paragan_gblock_check(d) == lib.EINVAL, field
        assert L.paragan_last_error(None).decode()
    assert L.paragan_gblock_check(None) == lib.EINVAL


def test_dblock_validation(L):
    ok = lib.DBlockDesc(2, 8, 8, 16, 32, 1, 1, 1, lib.BF16, 1, 1e-12)
    assert lib.paragan_dblock_check(ok) == lib.OK
    odd = lib.DBlockDesc(2, 7, 8, 16, 32, 1, 1, 1, lib.BF16, 1, 1e-12)
    assert lib.paragan_dblock_check(odd) == lib.EINVAL           # pooling needs even H
    ident = lib.DBlockDesc(2, 8, 8, 16, 32, 1, 0, 0, lib.BF16, 1, 1e-12)
    assert lib.paragan_dblock_check(ident) == lib.EINVAL         # identity skip, cin != cout


def test_pixel_count_limits(L):
    """Offsets inside the kernels are 32-bit: each module's check accepts
    the largest pixel count below 2^31 and rejects the next one (before
    anything is launched), and the network check bounds the concatenated
    real + fake batch the same way."""
    big = 1 << 15                       # H = W = 2^15: 2^30 pixels per image
    g = lib.GBlockDesc(1, big // 4, big, 64, 64, 128, lib.BF16, 1, 1e-5, 1e-12)
    assert lib.paragan_gblock_check(g) == lib.OK                  # output pixels 4 B H W = 2^30
    g.H = big // 2
    assert lib.paragan_gblock_check(g) == lib.EINVAL              # 2^31
    d = lib.DBlockDesc(1, big, big, 16, 32, 1, 1, 1, lib.BF16, 1, 1e-12)
    assert lib.paragan_dblock_check(d) == lib.OK                  # 2^30 pixels
    d.B = 2
    assert lib.paragan_dblock_check(d) == lib.EINVAL              # 2^31 pixels
    a = lib.AttnDesc(1, big, big, 64, 1, 1e-12)
    assert lib.paragan_attn_check(a) == lib.OK
    a.B = 2
    assert lib.paragan_attn_check(a) == lib.EINVAL
    o = lib.GoutDesc(1, big, 704, 96, 1, 1e-5, 1e-12)
    assert lib.paragan_gout_check(o) == lib.OK                    # 2.3e7 pixels
    o.B = (1 << 31) // (big * 704) + 1
    assert lib.paragan_gout_check(o) == lib.EINVAL
    n = _desc(O.biggan128())
    n.B = (1 << 31) // (2 * 128 * 128)                            # 2 B img^2 = 2^31: rejected
    assert lib.paragan_biggan_check(n) == lib.EINVAL
    n.B -= 1
    assert lib.paragan_biggan_check(n) == lib.OK


def test_entry_points_reject_null_context(L):
    d = lib.DBlockDesc(2, 8, 8, 16, 32, 1, 1, 1, lib.BF16, 1, 1e-12)
    assert L.paragan_dblock_fwd(None, C.byref(d), None, None, None, None, None, None) == lib.EINVAL
    assert L.paragan_sn_power_iter(None, None, 1, 1, None, None, None, 1, 1e-12, None) == lib.EINVAL


def test_layouts_match_oracle(L):
    ents, npar, nu = lib.paragan_gblock_layout(lib.GBlockDesc(4, 8, 8, 64, 48, 148, lib.BF16, 1, 1e-5, 1e-12))
    ref = OB.gblock_param_shapes(64, 48, 148)
    assert [(e["name"], e["shape"]) for e in ents] == list(ref.items())
    assert npar == sum(int(__import__("numpy").prod(s)) for s in ref.values())
    sn = [e["name"] for e in ents if e["u_offset"] >= 0]
    assert sn == list(OB.GBLOCK_SN)
    for lsc in (0, 1):
        ents, _, _ = lib.paragan_dblock_layout(lib.DBlockDesc(2, 8, 8, 32, 32, 1, lsc, lsc, lib.BF16, 1, 1e-12))
        assert [(e["name"], e["shape"]) for e in ents] == list(OB.dblock_param_shapes(32, 32, lsc).items())


def test_sizes_queries_need_no_gpu(L):
    s, w = lib.paragan_dblock_sizes(lib.DBlockDesc(64, 32, 32, 256, 512, 1, 1, 1, lib.BF16, 1, 1e-12))
    assert s > 0 and w > 0 and s % 256 == 0
    assert lib.paragan_sn_ws_size(512, 2304) > 0


def _desc(a, B=2):
    return biggan_desc(a, B, O.HParams(opt_g=O.adabelief_g()))


@pytest.mark.parametrize("arch", [O.biggan128, O.biggan512])
def test_network_layouts_match_oracle(L, arch):
    a = arch()
    d = _desc(a)
    assert lib.paragan_biggan_check(d) == lib.OK
    for which, fn in ((0, O.g_layout), (1, O.d_layout)):
        ents, npar, nu = lib.paragan_net_layout(d, which)
        lay, sn = fn(a)
        assert [(e["name"], e["shape"]) for e in ents] == list(lay.items())
        assert [e["name"] for e in ents if e["u_offset"] >= 0] == sn
    if arch is O.biggan128:
        g = lib.paragan_net_layout(d, 0)[1]
        dd = lib.paragan_net_layout(d, 1)[1]
        assert g + dd == 158_416_358            # Table tab:GAN: 158.42M


def test_biggan_validation(L):
    a = O.biggan128()
    d = _desc(a)
    d.img = 64
    assert lib.paragan_biggan_check(d) == lib.EINVAL          # img != 4 * 2^n_g
    d = _desc(a)
    d.dz = 121
    assert lib.paragan_biggan_check(d) == lib.EINVAL          # z does not split evenly
    d = _desc(a)
    assert lib.paragan_train_step_ws_size(d) > 0
    for field, bad in (("kind", 2), ("lr", -1.0), ("beta1", 1.0), ("beta2", -0.1), ("eps", 0.0)):
        for net in ("opt_g", "opt_d"):
            d = _desc(a)
            setattr(getattr(d, net), field, bad)
            assert lib.paragan_biggan_check(d) == lib.EINVAL, (net, field)


def test_gout_validation_and_layout(L):
    ok = lib.GoutDesc(2, 128, 128, 96, 1, 1e-5, 1e-12)
    assert lib.paragan_gout_check(ok) == lib.OK
    assert lib.paragan_gout_check(lib.GoutDesc(1, 8, 8, 129, 1, 1e-5, 1e-12)) == lib.EINVAL    # cpad(C) = 160
    assert lib.paragan_gout_check(lib.GoutDesc(1, 8, 10, 8, 1, 1e-5, 1e-12)) == lib.EINVAL     # W % 4 != 0
    assert lib.paragan_gout_check(lib.GoutDesc(1, 8, 2048, 96, 1, 1e-5, 1e-12)) == lib.EINVAL  # tile too wide
    assert lib.paragan_gout_check(lib.GoutDesc(1, 8, 704, 128, 1, 1e-5, 1e-12)) == lib.OK
    assert lib.paragan_gout_check(lib.GoutDesc(0, 8, 8, 8, 1, 1e-5, 1e-12)) == lib.EINVAL
    ents, npar, nu = lib.paragan_gout_layout(ok)
    lay, sn = O.g_layout(O.biggan128())
    out = [(k, v) for k, v in lay.items() if k.startswith("out_")]
    assert [(e["name"], e["shape"]) for e in ents] == out
    assert [e["name"] for e in ents if e["u_offset"] >= 0] == ["out_conv.w"] and nu == 3
    s, w = lib.paragan_gout_sizes(ok)
    assert s > 0 and w > 0


def test_biggan_rejects_wide_output_layer(L):
    a = O.biggan128()
    d = _desc(a)
    d.g_mult[a.n_g] = 2        # output layer input 192 channels
    assert lib.paragan_biggan_check(d) == lib.EINVAL
