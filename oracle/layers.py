"""Oracle layer primitives, float64, NHWC (test infrastructure only).

Each function states the definition it computes.  Backward functions are the
hand-derived adjoints of the forward ones; the tests pin them against
central finite differences, against a library routine where one exists
(torch's float64 CPU convolution, LAPACK's SVD) and against brute-force
loops on tiny inputs.

Shapes: activations are (N, H, W, C); convolution weights are
(Cout, R, S, Cin); linear weights are (out, in).
"""
import numpy as np


# --------------------------------------------------------------------------
# convolution: stride 1, zero padding (R-1)/2, bias
# --------------------------------------------------------------------------
def _pad(x, p):
    return np.pad(x, ((0, 0), (p, p), (p, p), (0, 0))) if p else x


def conv2d(x, w, b=None):
    """y[n,h,w,o] = b[o] + sum_{r,s,i} xpad[n,h+r,w+s,i] * w[o,r,s,i]."""
    n, h, wd, c = x.shape
    co, r_, s_, ci = w.shape
    assert ci == c and r_ == s_ and r_ % 2 == 1
    p = (r_ - 1) // 2
    xp = _pad(x, p)
    y = np.zeros((n, h, wd, co))
    for r in range(r_):
        for s in range(s_):
            y += xp[:, r:r + h, s:s + wd, :] @ w[:, r, s, :].T
    if b is not None:
        y += b
    return y


def conv2d_dgrad(dy, w):
    """Adjoint of conv2d in x: dx[n,h',w',i] = sum over taps of dy . w."""
    n, h, wd, co = dy.shape
    _, r_, s_, ci = w.shape
    p = (r_ - 1) // 2
    dxp = np.zeros((n, h + 2 * p, wd + 2 * p, ci))
    for r in range(r_):
        for s in range(s_):
            dxp[:, r:r + h, s:s + wd, :] += dy @ w[:, r, s, :]
    return dxp[:, p:p + h, p:p + wd, :]


def conv2d_wgrad(dy, x, ksize):
    """dw[o,r,s,i] = sum_{n,h,w} dy[n,h,w,o] * xpad[n,h+r,w+s,i]."""
    n, h, wd, co = dy.shape
    ci = x.shape[3]
    p = (ksize - 1) // 2
    xp = _pad(x, p)
    dw = np.zeros((co, ksize, ksize, ci))
    for r in range(ksize):
        for s in range(ksize):
            dw[:, r, s, :] = np.tensordot(dy, xp[:, r:r + h, s:s + wd, :],
                                          axes=([0, 1, 2], [0, 1, 2]))
    return dw


def bias_grad(dy):
    return dy.sum(axis=(0, 1, 2))


# --------------------------------------------------------------------------
# a 3x3 convolution fused with the 2x resampling next to it.  The 3x3 taps
# that meet the same input pixel are added first; in exact arithmetic this is
# the plain composition (the tests pin both identities).  Under bfloat16
# storage the folded filter, not the 3x3 one, is the stored weight operand.
# --------------------------------------------------------------------------
def up2_conv_fold(w):
    """Sub-pixel filters of conv3x3(up2(x), w).

    Output pixel (2i + a, 2j + b) with tap (r, s) reads the upsampled pixel
    (2i + a + r - 1, 2j + b + s - 1), i.e. the source pixel
    (i + (a + r - 1) // 2, j + (b + s - 1) // 2).  For parity a that row
    offset is a - 1 + t with t in {0, 1}.  Returns F of shape
    (2, 2, Cout, 2, 2, Cin): F[a, b][:, t, u, :] is the sum of the taps
    (r, s) whose source pixel is (i + a - 1 + t, j + b - 1 + u)."""
    co, r_, s_, ci = w.shape
    assert r_ == 3 and s_ == 3
    F = np.zeros((2, 2, co, 2, 2, ci))
    for a in range(2):
        for b in range(2):
            for r in range(3):
                for s in range(3):
                    t = (a + r - 1) // 2 - (a - 1)
                    u = (b + s - 1) // 2 - (b - 1)
                    F[a, b, :, t, u, :] += w[:, r, s, :]
    return F


def up2_conv(x, F, b=None):
    """y (N, 2H, 2W, Cout): y[n, 2i+a, 2j+b] = b + sum over t, u in {0, 1} of
    xpad[n, i+a+t, j+b+u] . F[a, b][:, t, u, :], xpad = x zero-padded by one
    pixel.  Equals conv2d(up2(x), w, b) for F = up2_conv_fold(w)."""
    n, h, wd, _ = x.shape
    co = F.shape[2]
    xp = _pad(x, 1)
    y = np.zeros((n, 2 * h, 2 * wd, co))
    for a in range(2):
        for bb in range(2):
            acc = np.zeros((n, h, wd, co))
            for t in range(2):
                for u in range(2):
                    acc += xp[:, a + t:a + t + h, bb + u:bb + u + wd, :] @ F[a, bb, :, t, u, :].T
            y[:, a::2, bb::2, :] = acc
    if b is not None:
        y += b
    return y


def up2_conv_dgrad(dy, F):
    """Adjoint of up2_conv in x: dx (N, H, W, Cin) from dy (N, 2H, 2W, Cout)."""
    n, h2, w2, _ = dy.shape
    h, wd = h2 // 2, w2 // 2
    ci = F.shape[-1]
    dxp = np.zeros((n, h + 2, wd + 2, ci))
    for a in range(2):
        for bb in range(2):
            g = dy[:, a::2, bb::2, :]
            for t in range(2):
                for u in range(2):
                    dxp[:, a + t:a + t + h, bb + u:bb + u + wd, :] += g @ F[a, bb, :, t, u, :]
    return dxp[:, 1:h + 1, 1:wd + 1, :]


def pool2_conv_fold(w):
    """Stride-2 4x4 filter of avgpool2(conv3x3(x, w)).

    Pooled pixel (i, j) averages the conv outputs (2i + a, 2j + b), whose
    tap (r, s) reads xpad[2i + a + r, 2j + b + s]; with t = a + r and
    u = b + s in 0..3, P[:, t, u, :] = 1/4 of the sum of w[:, t - a, u - b, :]
    over a, b in {0, 1} with the tap inside the 3x3 filter."""
    co, r_, s_, ci = w.shape
    assert r_ == 3 and s_ == 3
    P = np.zeros((co, 4, 4, ci))
    for a in range(2):
        for b in range(2):
            P[:, a:a + 3, b:b + 3, :] += w
    return 0.25 * P


def pool2_conv(x, P, b=None):
    """y (N, H/2, W/2, Cout): y[n, i, j] = b + sum over t, u in 0..3 of
    xpad[n, 2i+t, 2j+u] . P[:, t, u, :], xpad = x zero-padded by one pixel.
    Equals avgpool2(conv2d(x, w, b)) for P = pool2_conv_fold(w)."""
    n, h, wd, _ = x.shape
    ho, wo = h // 2, wd // 2
    co = P.shape[0]
    xp = _pad(x, 1)
    y = np.zeros((n, ho, wo, co))
    for t in range(4):
        for u in range(4):
            y += xp[:, t:t + 2 * ho:2, u:u + 2 * wo:2, :] @ P[:, t, u, :].T
    if b is not None:
        y += b
    return y


def pool2_conv_dgrad(dy, P):
    """Adjoint of pool2_conv in x: dx (N, 2Ho, 2Wo, Cin) from dy (N, Ho, Wo, Cout)."""
    n, ho, wo, _ = dy.shape
    ci = P.shape[-1]
    dxp = np.zeros((n, 2 * ho + 2, 2 * wo + 2, ci))
    for t in range(4):
        for u in range(4):
            dxp[:, t:t + 2 * ho:2, u:u + 2 * wo:2, :] += dy @ P[:, t, u, :]
    return dxp[:, 1:2 * ho + 1, 1:2 * wo + 1, :]


# --------------------------------------------------------------------------
# resampling
# --------------------------------------------------------------------------
def up2(x):
    """Nearest-neighbour 2x upsample: y[n,h,w,c] = x[n,h//2,w//2,c]."""
    return np.repeat(np.repeat(x, 2, axis=1), 2, axis=2)


def up2_bwd(dy):
    n, h, w, c = dy.shape
    return dy.reshape(n, h // 2, 2, w // 2, 2, c).sum(axis=(2, 4))


def avgpool2(x):
    """2x2 average pool, stride 2."""
    n, h, w, c = x.shape
    return x.reshape(n, h // 2, 2, w // 2, 2, c).mean(axis=(2, 4))


def avgpool2_bwd(dy):
    return up2(dy) * 0.25


def maxpool2(x):
    """2x2 max pool, stride 2.  Ties go to the first window element in
    (dh, dw) row-major order (a strict '>' scan).  Returns (y, argmax)."""
    n, h, w, c = x.shape
    win = x.reshape(n, h // 2, 2, w // 2, 2, c).transpose(0, 1, 3, 2, 4, 5)
    win = win.reshape(n, h // 2, w // 2, 4, c)
    arg = np.argmax(win, axis=3)              # first occurrence of the max
    y = np.take_along_axis(win, arg[:, :, :, None, :], axis=3)[:, :, :, 0, :]
    return y, arg


def maxpool2_bwd(dy, arg):
    n, h2, w2, c = dy.shape
    win = np.zeros((n, h2, w2, 4, c))
    np.put_along_axis(win, arg[:, :, :, None, :], dy[:, :, :, None, :], axis=3)
    win = win.reshape(n, h2, w2, 2, 2, c).transpose(0, 1, 3, 2, 4, 5)
    return win.reshape(n, 2 * h2, 2 * w2, c)


def relu(x):
    return np.maximum(x, 0.0)


# --------------------------------------------------------------------------
# batch normalisation (training-mode batch statistics, biased variance)
# --------------------------------------------------------------------------
def bn_stats(x):
    """Two-pass per-channel mean and biased variance over (N, H, W)."""
    cnt = x.shape[0] * x.shape[1] * x.shape[2]
    mean = x.sum(axis=(0, 1, 2)) / cnt
    var = ((x - mean) ** 2).sum(axis=(0, 1, 2)) / cnt
    return mean, var


def cbn_fwd(x, gain, bias, eps):
    """Conditional BN: y = gain[n,c] * (x - mean_c) / sqrt(var_c + eps) + bias[n,c].

    gain/bias are per-sample, per-channel (N, C); a plain affine BN passes
    (1, C) arrays.  Returns y and the cache for the backward pass."""
    mean, var = bn_stats(x)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mean) * rstd
    y = gain[:, None, None, :] * xhat + bias[:, None, None, :]
    return y, (xhat, rstd, gain)


def cbn_bwd(dy, cache):
    """Returns dx, dgain (N or 1, C), dbias (N or 1, C)."""
    xhat, rstd, gain = cache
    cnt = dy.shape[0] * dy.shape[1] * dy.shape[2]
    if gain.shape[0] == dy.shape[0]:
        dgain = (dy * xhat).sum(axis=(1, 2))
        dbias = dy.sum(axis=(1, 2))
    else:
        dgain = (dy * xhat).sum(axis=(0, 1, 2))[None, :]
        dbias = dy.sum(axis=(0, 1, 2))[None, :]
    dxhat = dy * gain[:, None, None, :]
    m1 = dxhat.sum(axis=(0, 1, 2)) / cnt
    m2 = (dxhat * xhat).sum(axis=(0, 1, 2)) / cnt
    dx = rstd * (dxhat - m1 - xhat * m2)
    return dx, dgain, dbias


# --------------------------------------------------------------------------
# spectral normalisation: one power iteration per training forward
# --------------------------------------------------------------------------
def _nrm(x, eps):
    return x / max(np.linalg.norm(x), eps)


def sn_power_iter(wmat, u, n_iter, eps):
    """v <- N(W^T u), u <- N(W v) repeated n_iter times; sigma = u^T W v.

    wmat is the weight viewed as (rows, cols) = (Cout, Cin*R*S); N(t) =
    t / max(||t||, eps).  Returns (u, v, sigma)."""
    for _ in range(n_iter):
        v = _nrm(wmat.T @ u, eps)
        u = _nrm(wmat @ v, eps)
    sigma = float(u @ (wmat @ v))
    return u, v, sigma


def sn_bwd(dwsn, wsn, u, v, sigma):
    """Gradient of W/sigma(W) with sigma = u^T W v and u, v held constant:
    dW = (dWsn - <dWsn, Wsn> u v^T) / sigma."""
    shp = dwsn.shape
    d = dwsn.reshape(shp[0], -1)
    s = wsn.reshape(shp[0], -1)
    dw = (d - float((d * s).sum()) * np.outer(u, v)) / sigma
    return dw.reshape(shp)


# --------------------------------------------------------------------------
# self-attention (non-local) block core
# --------------------------------------------------------------------------
def attention_core_fwd(q, k, v):
    """Per image: S = Q K^T (no scaling), P = softmax over keys, O = P V.

    q (N, Lq, dk), k (N, Lk, dk), v (N, Lk, dv)."""
    s = q @ k.transpose(0, 2, 1)
    s = s - s.max(axis=2, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=2, keepdims=True)
    return p @ v, p


def attention_core_bwd(do, q, k, v, p):
    dv = p.transpose(0, 2, 1) @ do
    dp = do @ v.transpose(0, 2, 1)
    ds = p * (dp - (dp * p).sum(axis=2, keepdims=True))
    dq = ds @ k
    dk = ds.transpose(0, 2, 1) @ q
    return dq, dk, dv


# --------------------------------------------------------------------------
# hinge loss and Adam
# --------------------------------------------------------------------------
def hinge_d(out_real, out_fake):
    """L_D = mean relu(1 - D(x_r)) + mean relu(1 + D(x_f)); the derivative
    at the kink is taken as 0.  Returns (loss, dL/dout_real, dL/dout_fake)."""
    br, bf = out_real.shape[0], out_fake.shape[0]
    loss = relu(1.0 - out_real).mean() + relu(1.0 + out_fake).mean()
    d_real = np.where(out_real < 1.0, -1.0 / br, 0.0)
    d_fake = np.where(out_fake > -1.0, 1.0 / bf, 0.0)
    return float(loss), d_real, d_fake


def hinge_g(out_fake):
    """L_G = -mean D(G(z))."""
    b = out_fake.shape[0]
    return float(-out_fake.mean()), np.full(out_fake.shape, -1.0 / b)


def adabelief(p, g, m, s, t, lr, beta1, beta2, eps):
    """AdaBelief step t (t >= 1), the optimiser the paper pairs with the
    generator (Numerical Optimizations, "Asymmetric Optimization Policy"),
    as its authors define it (Zhuang et al., NeurIPS 2020): the second
    moment tracks the squared deviation of the gradient from its running
    mean (the "belief"), eps inside the moment and in the denominator,
    bias-corrected, no weight decay."""
    m = beta1 * m + (1.0 - beta1) * g
    s = beta2 * s + (1.0 - beta2) * (g - m) ** 2 + eps
    mhat = m / (1.0 - beta1 ** t)
    shat = s / (1.0 - beta2 ** t)
    return p - lr * mhat / (np.sqrt(shat) + eps), m, s


def adam(p, g, m, v, t, lr, beta1, beta2, eps):
    """Bias-corrected Adam step t (t >= 1), no weight decay."""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    return p - lr * mhat / (np.sqrt(vhat) + eps), m, v
