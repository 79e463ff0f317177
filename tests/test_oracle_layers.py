"""Pins for the oracle's layer primitives (CPU only).

Each primitive is checked against something other than itself: a library
routine (torch float64 CPU ops, LAPACK's SVD), brute-force loops on tiny
inputs, closed forms, invariants, or central finite differences.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import layers as L
from oracle.numerics import bf16

RNG = np.random.default_rng(12345)


def t(x):
    return torch.from_numpy(np.ascontiguousarray(x))


def nchw(x):
    return t(x.transpose(0, 3, 1, 2))


def nhwc(y):
    return y.detach().numpy().transpose(0, 2, 3, 1)


# ---------------------------------------------------------------- bfloat16
def test_bf16_matches_torch_cast():
    x = np.concatenate([RNG.standard_normal(20000) * 10.0 ** RNG.integers(-30, 30, 20000),
                        RNG.standard_normal(1000)]).astype(np.float32).astype(np.float64)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16(x), ref)


def test_bf16_closed_forms():
    ulp = 2.0 ** -7                       # spacing of bfloat16 in [1, 2)
    assert bf16(1.0 + ulp / 2) == 1.0     # tie -> even (1.0)
    assert bf16(1.0 + 1.5 * ulp) == 1.0 + 2 * ulp   # tie -> even (1+2ulp)
    assert bf16(1.0 + 0.75 * ulp) == 1.0 + ulp
    assert bf16(-3.0) == -3.0
    assert np.isinf(bf16(3.5e38)) and bf16(3.389e38) == (2 - 2 ** -7) * 2.0 ** 127
    assert np.isnan(bf16(np.nan))
    assert bf16(2.0 ** -133) == 2.0 ** -133 and bf16(2.0 ** -135) == 0.0
    # not via fp32: 1 + ulp/2 + 2**-40 is above the tie and must round up
    assert bf16(1.0 + ulp / 2 + 2.0 ** -40) == 1.0 + ulp


# ------------------------------------------------------------- convolution
@pytest.mark.parametrize("k", [1, 3])
def test_conv_matches_torch(k):
    x = RNG.standard_normal((2, 5, 6, 4))
    w = RNG.standard_normal((3, k, k, 4))
    b = RNG.standard_normal(3)
    ref = F.conv2d(nchw(x), t(w.transpose(0, 3, 1, 2)), t(b), padding=(k - 1) // 2)
    np.testing.assert_allclose(L.conv2d(x, w, b), nhwc(ref), rtol=1e-12, atol=1e-12)


def test_conv_brute_force():
    x = RNG.standard_normal((1, 3, 4, 2))
    w = RNG.standard_normal((2, 3, 3, 2))
    y = L.conv2d(x, w)
    ref = np.zeros((1, 3, 4, 2))
    for h in range(3):
        for ww in range(4):
            for o in range(2):
                s = 0.0
                for r in range(3):
                    for q in range(3):
                        hh, wq = h + r - 1, ww + q - 1
                        if 0 <= hh < 3 and 0 <= wq < 4:
                            for i in range(2):
                                s += x[0, hh, wq, i] * w[o, r, q, i]
                ref[0, h, ww, o] = s
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("k", [1, 3])
def test_conv_backward_matches_torch_autograd(k):
    x = RNG.standard_normal((2, 4, 5, 3))
    w = RNG.standard_normal((4, k, k, 3))
    dy = RNG.standard_normal((2, 4, 5, 4))
    xt = nchw(x).requires_grad_()
    wt = t(w.transpose(0, 3, 1, 2)).requires_grad_()
    F.conv2d(xt, wt, padding=(k - 1) // 2).backward(nchw(dy))
    np.testing.assert_allclose(L.conv2d_dgrad(dy, w), nhwc(xt.grad), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(L.conv2d_wgrad(dy, x, k),
                               wt.grad.numpy().transpose(0, 2, 3, 1), rtol=1e-12, atol=1e-12)


def test_conv_adjointness():
    x = RNG.standard_normal((2, 6, 6, 3))
    w = RNG.standard_normal((5, 3, 3, 3))
    dy = RNG.standard_normal((2, 6, 6, 5))
    lhs = (L.conv2d(x, w) * dy).sum()
    assert abs(lhs - (x * L.conv2d_dgrad(dy, w)).sum()) < 1e-9 * abs(lhs)
    assert abs(lhs - (w * L.conv2d_wgrad(dy, x, 3)).sum()) < 1e-9 * abs(lhs)


# -------------------------------------------------------------- resampling
def test_resampling_matches_torch():
    x = RNG.standard_normal((2, 6, 4, 3))
    np.testing.assert_array_equal(L.up2(x), nhwc(F.interpolate(nchw(x), scale_factor=2, mode="nearest")))
    np.testing.assert_allclose(L.avgpool2(x), nhwc(F.avg_pool2d(nchw(x), 2)), rtol=1e-14)
    y, _ = L.maxpool2(x)
    np.testing.assert_array_equal(y, nhwc(F.max_pool2d(nchw(x), 2)))


def test_resampling_adjoints():
    x = RNG.standard_normal((2, 4, 6, 3))
    d = RNG.standard_normal((2, 8, 12, 3))
    assert np.isclose((L.up2(x) * d).sum(), (x * L.up2_bwd(d)).sum())
    d2 = RNG.standard_normal((2, 2, 3, 3))
    assert np.isclose((L.avgpool2(x) * d2).sum(), (x * L.avgpool2_bwd(d2)).sum())
    y, arg = L.maxpool2(x)
    g = L.maxpool2_bwd(d2, arg)
    assert np.isclose((y * d2).sum(), (x * g).sum())        # piecewise linear
    assert np.count_nonzero(g) == d2.size


# ------------------------------------------- convolutions fused with resampling
def test_up2_conv_fold_equals_conv_over_upsample():
    """conv3x3(up2(x)) with the taps that meet one source pixel added first:
    equal to torch's conv over torch's nearest upsample, forward and data
    gradient, on an odd ragged shape."""
    x = RNG.standard_normal((2, 3, 5, 4))
    w = RNG.standard_normal((6, 3, 3, 4))
    b = RNG.standard_normal(6)
    dy = RNG.standard_normal((2, 6, 10, 6))
    Fw = L.up2_conv_fold(w)
    xt = nchw(x).requires_grad_()
    up = F.interpolate(xt, scale_factor=2, mode="nearest")
    ref = F.conv2d(up, t(w.transpose(0, 3, 1, 2)), t(b), padding=1)
    ref.backward(nchw(dy))
    np.testing.assert_allclose(L.up2_conv(x, Fw, b), nhwc(ref), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(L.up2_conv_dgrad(dy, Fw), nhwc(xt.grad), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(L.up2_conv_dgrad(dy, Fw), L.up2_bwd(L.conv2d_dgrad(dy, w)), rtol=1e-12,
                               atol=1e-12)


def test_up2_conv_fold_taps():
    """Each parity class's folded taps add up to the whole 3x3 filter; a single
    1 at tap (r, s) lands at the documented (t, u) = source offset - (a - 1)."""
    w = RNG.standard_normal((2, 3, 3, 3))
    Fw = L.up2_conv_fold(w)
    for a in range(2):
        for b in range(2):
            np.testing.assert_allclose(Fw[a, b].sum(axis=(1, 2)), w.sum(axis=(1, 2)), rtol=1e-13)
    one = np.zeros((1, 3, 3, 1))
    one[0, 0, 2, 0] = 1.0        # r = 0, s = 2
    Fo = L.up2_conv_fold(one)
    # a = 0: row offset -1 -> t = 0; a = 1: offset 0 -> t = 0.  b = 0: column
    # offset 0 -> u = 1; b = 1: offset +1 -> u = 1.
    for a in range(2):
        for b in range(2):
            nz = np.argwhere(Fo[a, b, 0, :, :, 0] != 0).tolist()
            assert nz == [[0, 1]], (a, b, nz)


def test_up2_conv_brute_force():
    x = RNG.standard_normal((1, 2, 3, 2))
    w = RNG.standard_normal((2, 3, 3, 2))
    up = np.zeros((1, 4, 6, 2))
    for h in range(4):
        for q in range(6):
            up[0, h, q] = x[0, h // 2, q // 2]
    ref = np.zeros((1, 4, 6, 2))
    for h in range(4):
        for q in range(6):
            for o in range(2):
                acc = 0.0
                for r in range(3):
                    for s in range(3):
                        hh, qq = h + r - 1, q + s - 1
                        if 0 <= hh < 4 and 0 <= qq < 6:
                            acc += float(up[0, hh, qq] @ w[o, r, s])
                ref[0, h, q, o] = acc
    np.testing.assert_allclose(L.up2_conv(x, L.up2_conv_fold(w)), ref, rtol=1e-13, atol=1e-13)


def test_pool2_conv_fold_equals_pooled_conv():
    """avgpool2(conv3x3(x)) as one stride-2 4x4 conv: equal to torch's pooled
    conv, forward and data gradient."""
    x = RNG.standard_normal((2, 6, 8, 3))
    w = RNG.standard_normal((5, 3, 3, 3))
    b = RNG.standard_normal(5)
    dy = RNG.standard_normal((2, 3, 4, 5))
    P = L.pool2_conv_fold(w)
    xt = nchw(x).requires_grad_()
    ref = F.avg_pool2d(F.conv2d(xt, t(w.transpose(0, 3, 1, 2)), t(b), padding=1), 2)
    ref.backward(nchw(dy))
    np.testing.assert_allclose(L.pool2_conv(x, P, b), nhwc(ref), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(L.pool2_conv_dgrad(dy, P), nhwc(xt.grad), rtol=1e-12, atol=1e-12)
    # the 4x4 taps sum to the 3x3 filter's total; the corners hold w / 4
    np.testing.assert_allclose(P.sum(axis=(1, 2)), w.sum(axis=(1, 2)), rtol=1e-13)
    np.testing.assert_allclose(P[:, 0, 0], w[:, 0, 0] / 4, rtol=1e-15)
    np.testing.assert_allclose(P[:, 3, 3], w[:, 2, 2] / 4, rtol=1e-15)


def test_fused_resample_conv_adjointness():
    x = RNG.standard_normal((2, 4, 6, 3))
    w = RNG.standard_normal((4, 3, 3, 3))
    d_up = RNG.standard_normal((2, 8, 12, 4))
    Fw = L.up2_conv_fold(w)
    lhs = (L.up2_conv(x, Fw) * d_up).sum()
    assert abs(lhs - (x * L.up2_conv_dgrad(d_up, Fw)).sum()) < 1e-10 * abs(lhs)
    d_pool = RNG.standard_normal((2, 2, 3, 4))
    P = L.pool2_conv_fold(w)
    lhs = (L.pool2_conv(x, P) * d_pool).sum()
    assert abs(lhs - (x * L.pool2_conv_dgrad(d_pool, P)).sum()) < 1e-10 * abs(lhs)


def test_maxpool_tie_rule():
    x = np.zeros((1, 2, 2, 3))
    x[0, :, :, 0] = [[1.0, 1.0], [1.0, 1.0]]      # all tied -> (0, 0)
    x[0, :, :, 1] = [[0.0, 2.0], [2.0, 0.0]]      # tie (0,1)/(1,0) -> (0, 1)
    x[0, :, :, 2] = [[0.0, 0.0], [0.0, 5.0]]
    y, arg = L.maxpool2(x)
    assert arg[0, 0, 0].tolist() == [0, 1, 3]
    g = L.maxpool2_bwd(np.ones((1, 1, 1, 3)), arg)
    assert g[0, 0, 0, 0] == 1 and g[0, 0, 1, 1] == 1 and g[0, 1, 1, 2] == 1
    assert g.sum() == 3


# --------------------------------------------------------------- batch norm
def test_bn_matches_torch_and_closed_form():
    x = RNG.standard_normal((3, 4, 5, 6)) * 3 + 7
    gain = np.ones((1, 6))
    bias = np.zeros((1, 6))
    y, _ = L.cbn_fwd(x, gain, bias, 1e-5)
    ref = F.batch_norm(nchw(x), None, None, training=True, eps=1e-5)
    np.testing.assert_allclose(y, nhwc(ref), rtol=1e-11, atol=1e-11)
    mean, var = L.bn_stats(x)
    np.testing.assert_allclose(y.mean(axis=(0, 1, 2)), 0, atol=1e-12)
    np.testing.assert_allclose(y.var(axis=(0, 1, 2)), var / (var + 1e-5), rtol=1e-12)
    np.testing.assert_allclose(var, np.var(x.reshape(-1, 6), axis=0), rtol=1e-12)


def _fd(f, x, idx, h=1e-6):
    xp = x.copy(); xp[idx] += h
    xm = x.copy(); xm[idx] -= h
    return (f(xp) - f(xm)) / (2 * h)


def test_cbn_backward_finite_differences():
    x = RNG.standard_normal((3, 2, 3, 4))
    gain = RNG.standard_normal((3, 4))
    bias = RNG.standard_normal((3, 4))
    r = RNG.standard_normal((3, 2, 3, 4))
    f = lambda xx, gg=gain, bb=bias: (L.cbn_fwd(xx, gg, bb, 1e-3)[0] * r).sum()
    y, cache = L.cbn_fwd(x, gain, bias, 1e-3)
    dx, dg, db = L.cbn_bwd(r, cache)
    for idx in [(0, 0, 0, 0), (1, 1, 2, 3), (2, 0, 1, 2)]:
        assert np.isclose(dx[idx], _fd(f, x, idx), rtol=1e-6, atol=1e-8)
    for idx in [(0, 0), (2, 3)]:
        assert np.isclose(dg[idx], _fd(lambda gg: f(x, gg), gain, idx), rtol=1e-6)
        assert np.isclose(db[idx], _fd(lambda bb: f(x, gain, bb), bias, idx), rtol=1e-6)
    # invariant: a per-channel gain leaves sum(dx) = 0, and at eps = 0 also
    # sum(dx * xhat) = 0 (sum xhat^2 = N var / (var + eps))
    g1 = RNG.standard_normal((1, 4))
    _, c1 = L.cbn_fwd(x, g1, np.zeros((1, 4)), 0.0)
    dx1, _, _ = L.cbn_bwd(r, c1)
    np.testing.assert_allclose(dx1.sum(axis=(0, 1, 2)), 0, atol=1e-10)
    np.testing.assert_allclose((dx1 * c1[0]).sum(axis=(0, 1, 2)), 0, atol=1e-10)


# ---------------------------------------------------------- spectral norm
def test_sn_converges_to_svd_sigma_and_is_monotone():
    w = RNG.standard_normal((12, 30))
    s1 = np.linalg.svd(w, compute_uv=False)[0]
    u = RNG.standard_normal(12)
    prev = 0.0
    for k in range(1, 60):
        _, _, s = L.sn_power_iter(w, u, k, 1e-12)
        assert s <= s1 * (1 + 1e-12)
        assert s >= prev * (1 - 1e-12)
        prev = s
    assert np.isclose(prev, s1, rtol=1e-9)


def test_sn_closed_forms():
    q, _ = np.linalg.qr(RNG.standard_normal((20, 8)))
    w = q.T                                           # orthonormal rows
    _, _, s = L.sn_power_iter(w, RNG.standard_normal(8), 1, 1e-12)
    assert np.isclose(s, 1.0, rtol=1e-12)
    w = RNG.standard_normal((6, 10))
    u = RNG.standard_normal(6)
    _, _, s = L.sn_power_iter(w, u, 3, 1e-12)
    _, _, s3 = L.sn_power_iter(-2.5 * w, u, 3, 1e-12)
    assert np.isclose(s3, 2.5 * s)                    # sigma(cW) = |c| sigma(W)
    perm = RNG.permutation(10)
    _, _, sp = L.sn_power_iter(w[:, perm], u, 3, 1e-12)
    assert np.isclose(sp, s)                          # column permutation
    un, v, _ = L.sn_power_iter(np.zeros((3, 4)), np.ones(3), 1, 1e-12)
    assert np.all(un == 0) and np.all(v == 0)         # eps guards the norm


def test_sn_backward_frozen_uv_fd_and_converged_svd():
    w = RNG.standard_normal((5, 7))
    u0 = RNG.standard_normal(5)
    un, v, s = L.sn_power_iter(w, u0, 1, 1e-12)
    r = RNG.standard_normal((5, 7))
    f = lambda ww: ((ww / float(un @ ww @ v)) * r).sum()
    dw = L.sn_bwd(r, w / s, un, v, s)
    for idx in [(0, 0), (3, 6), (4, 2)]:
        assert np.isclose(dw[idx], _fd(f, w, idx), rtol=1e-6)
    # converged power iteration: gradient of W / sigma_1(W) via LAPACK
    un, v, s = L.sn_power_iter(w, u0, 500, 1e-12)
    g = lambda ww: ((ww / np.linalg.svd(ww, compute_uv=False)[0]) * r).sum()
    dw = L.sn_bwd(r, w / s, un, v, s)
    for idx in [(0, 0), (3, 6), (4, 2)]:
        assert np.isclose(dw[idx], _fd(g, w, idx), rtol=1e-5)


# --------------------------------------------------------------- attention
def test_attention_core_matches_torch_and_invariants():
    q = RNG.standard_normal((2, 8, 3))
    k = RNG.standard_normal((2, 4, 3))
    v = RNG.standard_normal((2, 4, 5))
    o, p = L.attention_core_fwd(q, k, v)
    ref = torch.softmax(t(q) @ t(k).transpose(1, 2), dim=-1) @ t(v)
    np.testing.assert_allclose(o, ref.numpy(), rtol=1e-12)
    np.testing.assert_allclose(p.sum(axis=2), 1.0, rtol=1e-14)
    o0, _ = L.attention_core_fwd(np.zeros_like(q), k, v)   # uniform weights
    np.testing.assert_allclose(o0, np.broadcast_to(v.mean(axis=1, keepdims=True), o0.shape))


def test_attention_core_backward_fd():
    q = RNG.standard_normal((1, 6, 3))
    k = RNG.standard_normal((1, 4, 3))
    v = RNG.standard_normal((1, 4, 2))
    r = RNG.standard_normal((1, 6, 2))
    o, p = L.attention_core_fwd(q, k, v)
    dq, dk, dv = L.attention_core_bwd(r, q, k, v, p)
    f = lambda qq, kk, vv: (L.attention_core_fwd(qq, kk, vv)[0] * r).sum()
    for idx in [(0, 0, 0), (0, 5, 2)]:
        assert np.isclose(dq[idx], _fd(lambda z: f(z, k, v), q, idx), rtol=1e-6)
    for idx in [(0, 1, 1), (0, 3, 0)]:
        assert np.isclose(dk[idx], _fd(lambda z: f(q, z, v), k, idx), rtol=1e-6)
        assert np.isclose(dv[idx], _fd(lambda z: f(q, k, z), v, idx), rtol=1e-6)


# ------------------------------------------------------------ hinge, Adam
def test_hinge_closed_form():
    real = np.array([2.0, 0.5, 1.0, -1.0])
    fake = np.array([-2.0, -0.5, -1.0, 3.0])
    loss, dr, df = L.hinge_d(real, fake)
    assert np.isclose(loss, (0 + 0.5 + 0 + 2) / 4 + (0 + 0.5 + 0 + 4) / 4)
    np.testing.assert_array_equal(dr, [0, -0.25, 0, -0.25])    # kink at 1 -> 0
    np.testing.assert_array_equal(df, [0, 0.25, 0, 0.25])      # kink at -1 -> 0
    lg, dg = L.hinge_g(fake)
    assert np.isclose(lg, -(-2 - 0.5 - 1 + 3) / 4)
    np.testing.assert_array_equal(dg, -0.25)


def test_adam_closed_form_steps():
    p = np.array([1.0, -2.0, 0.5])
    g = np.array([0.3, -4e-7, 0.0])
    lr, eps = 1e-3, 1e-6
    # beta1 = 0: first step is lr * g / (|g| + eps)
    p1, m, v = L.adam(p, g, np.zeros(3), np.zeros(3), 1, lr, 0.0, 0.999, eps)
    np.testing.assert_allclose(p1, p - lr * g / (np.abs(g) + eps), rtol=1e-14)
    g2 = np.array([-0.1, 1e-6, 2.0])
    p2, _, _ = L.adam(p1, g2, m, v, 2, lr, 0.0, 0.999, eps)
    vhat = (0.999 * 0.001 * g ** 2 + 0.001 * g2 ** 2) / (1 - 0.999 ** 2)
    np.testing.assert_allclose(p2, p1 - lr * g2 / (np.sqrt(vhat) + eps), rtol=1e-12)
    # beta1 > 0: bias-corrected momentum, closed form at step 1 is the same
    p1b, _, _ = L.adam(p, g, np.zeros(3), np.zeros(3), 1, lr, 0.9, 0.999, eps)
    np.testing.assert_allclose(p1b, p1, rtol=1e-12)


def test_adabelief_worked_first_step():
    """Hand-computed first step from zero state: g = 2, beta1 = 1/2,
    beta2 = 3/4, eps = 0: m = 1, s = (1/4)(2 - 1)^2 = 1/4, mhat = 2,
    shat = 1, so the parameter moves by -2 lr."""
    p1, m, s = L.adabelief(np.array([5.0]), np.array([2.0]), np.zeros(1), np.zeros(1), 1, 0.1, 0.5, 0.75, 0.0)
    assert m[0] == 1.0 and s[0] == 0.25
    assert np.isclose(p1[0], 5.0 - 0.2, rtol=0, atol=1e-15)


def test_adabelief_constant_gradient_limit():
    """With a constant gradient the bias-corrected mean is exactly g at every
    step, the deviation g - m decays as beta1^t, so the second moment tends
    to eps / (1 - beta2) (the belief in a steady gradient): the step grows
    monotonically towards lr g / (sqrt(eps / (1 - beta2)) + eps)."""
    g, lr, b1, b2, eps = 0.3, 1e-3, 0.5, 0.9, 1e-8
    p, m, s = np.zeros(1), np.zeros(1), np.zeros(1)
    steps = []
    for t in range(1, 400):
        p_new, m, s = L.adabelief(p, np.array([g]), m, s, t, lr, b1, b2, eps)
        steps.append(float(p[0] - p_new[0]))
        p = p_new
        assert np.isclose(m[0] / (1 - b1 ** t), g, rtol=1e-12)
    assert all(b >= a * (1 - 1e-12) for a, b in zip(steps, steps[1:]))
    limit = lr * g / (np.sqrt(eps / (1 - b2)) + eps)
    assert np.isclose(steps[-1], limit, rtol=1e-6)


def test_adabelief_scale_invariant_without_eps():
    """At eps = 0 the step depends on the gradient's direction history, not
    its scale: m scales by k and (g - m)^2 by k^2."""
    rng = np.random.default_rng(5)
    gs = rng.standard_normal((6, 4))
    out = []
    for k in (1.0, 1e-3):
        p, m, s = np.zeros(4), np.zeros(4), np.zeros(4)
        for t, g in enumerate(gs, start=1):
            p, m, s = L.adabelief(p, k * g, m, s, t, 1e-2, 0.9, 0.999, 0.0)
        out.append(p)
    np.testing.assert_allclose(out[0], out[1], rtol=1e-10)
