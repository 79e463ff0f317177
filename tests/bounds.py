"""Element-wise bounds on what ambiguous ReLU decisions can change, computed
from the oracle alone (test infrastructure).

The GPU and the oracle evaluate the same bf16-storage arithmetic in
different summation orders (fp32 on the GPU, fp64 here).  Where a ReLU's
input lies within the summation error of zero, the two may take different
mask decisions, and the gradient behind that element then differs by its
whole value: a large, local change that no relative tolerance covers.  (The
other effect of summation order, a bf16 rounding going to the other
neighbour, changes a value by one spacing, 2^-8 of it: that is what the 2e-2
bar absorbs.  It enters here only by widening the band in which a ReLU
decision counts as ambiguous.)

For each block the functions below mark the ambiguous ReLU inputs from the
oracle's own values, compute for each of them the exact (signed) change of
every backward output when that mask alone reverses, and sum the absolute
values over the marked elements: the largest change any subset of flips can
cause, element by element.  A parity check then allows
|gpu - oracle| <= tol * max|oracle| + bound; elements no flip can reach get
no slack.

The bands are error estimates, not worst cases.  A worst-case bound on fp32
summation over K terms (about K/16 roundings of the accumulator) exceeds
bf16's half spacing for the sums here and would mark nearly every element;
the estimate instead models each accumulator rounding as an independent
error of at most 2^-24 of the running sum, whose total over n roundings has
standard deviation below 2^-24 sqrt(n) times the root-sum-square of the
terms.  SUM_EPS = 2^-19 takes 32 such standard deviations with n = K:
band = SUM_EPS * sqrt(K) * sqrt(sum of squared terms).  A BN output
gain * xhat + bias comes from fp32 statistics and tables after a handful of
roundings: BN_EPS = 2^-20 of its absolute terms.  The spectral norm sigma is
an fp32 power iteration on the GPU: SIGMA_EPS = 2^-16 of every value it
scales (a convolution's accumulated product, a conditional gain's and
bias's linear part).  The bf16 weight operands themselves are identical on
both sides: the master filter (or its exact fold) rounded once.
"""
import numpy as np

from oracle import layers as L

SUM_EPS = 2.0 ** -19
BN_EPS = 2.0 ** -20
SIGMA_EPS = 2.0 ** -16


def conv_band(l2sq, k):
    """Summation band of conv outputs whose k terms have squared sum l2sq."""
    return SUM_EPS * np.sqrt(k) * np.sqrt(l2sq)


def ulp_bf16(x):
    """Spacing of bfloat16 numbers at |x| (8 significant bits)."""
    ax = np.maximum(np.abs(np.asarray(x, np.float64)), 2.0 ** -126)
    return np.ldexp(1.0, np.floor(np.log2(ax)).astype(int) - 7)


def tie_ambiguous(v, band):
    """Where the exact value v lies within `band` of a bf16 rounding boundary
    (a midpoint between neighbouring bf16 numbers), so that a slightly
    different sum may round to the other neighbour."""
    v = np.abs(np.asarray(v, np.float64))
    u = ulp_bf16(v)
    q = v / u
    return np.abs(q - np.floor(q) - 0.5) * u <= band


def sn_bound(d_abs, proj_abs, st):
    """Bound on the change of the SN backward dW = (d - <d, Wsn> u v^T) / sigma
    given bounds on the change of d (element-wise, d_abs) and of <d, Wsn>
    (proj_abs, a scalar)."""
    un, v, sigma = st
    shp = d_abs.shape
    d = d_abs.reshape(shp[0], -1)
    return ((d + proj_abs * np.outer(np.abs(un), np.abs(v))) / sigma).reshape(shp)


def _bn_band(bn, xhat, gain):
    """Band of a BN output gain * xhat + bias computed from fp32 statistics
    and tables, gain - 1 and bias being SN-normalised linear maps."""
    g = gain[:, None, None, :]
    bias = np.abs(bn - g * xhat)
    return BN_EPS * (np.abs(g * xhat) + bias) + SIGMA_EPS * (np.abs((g - 1.0) * xhat) + bias)


def _pad1(x):
    return np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))


def _cbn_abs(ddy, xhat, rstd, gain):
    """Absolute-value map of the cBN backward for an output-gradient change
    bounded by ddy >= 0: bounds on the change of (dx, dgain, dbias)."""
    cnt = ddy.shape[0] * ddy.shape[1] * ddy.shape[2]
    gd = np.abs(gain)[:, None, None, :] * ddy
    ax = np.abs(xhat)
    m1 = gd.sum(axis=(0, 1, 2)) / cnt
    m2 = (gd * ax).sum(axis=(0, 1, 2)) / cnt
    return rstd * (gd + m1 + ax * m2), (ddy * ax).sum(axis=(1, 2)), ddy.sum(axis=(1, 2))


def _local_dgrad(F, ch, b, i, j, src_shape):
    """up2_conv_dgrad of a unit gradient at output pixel (b, i, j) of channel
    ch: at most four source pixels, as [(b, h, w, vector over Cin)]."""
    a, bb = i % 2, j % 2
    i0, j0 = i // 2, j // 2
    out = []
    for t in range(2):
        for u in range(2):
            h, w = i0 + a - 1 + t, j0 + bb - 1 + u
            if 0 <= h < src_shape[1] and 0 <= w < src_shape[2]:
                out.append((b, h, w, F[a, bb, ch, t, u, :]))
    return out


def gblock_bounds(p, cache, dy):
    """Bounds on |gpu - oracle| for the generator block's backward outputs in
    bf16 (the oracle's gradient names, plus "dx", "dcond" and "conv1.b_l1",
    the extra L1 mass of conv1.b's cancelling sum), and {"counts", "masks"}
    of the ambiguous ReLU decisions.  p: the block's parameters; cache: the
    oracle forward's; dy: the output gradient.

    A flip of cBN2's ReLU at e = (b, i, j, ch) moves dbn2 by da2[e] there,
    hence dh1 on channel ch by k (1_e - (1 + xh2 xh2[e]) / cnt): a local
    term and the spread through the batch means.  conv1's weight rows, the
    bn2 linears and every SN projection take each flip's exact response.
    Further down (conv1's data gradient, cBN1, the bn1 linears, dcond) the
    local term keeps its exact response and the spread terms, summed per
    channel, go through absolute-value maps."""
    c = cache
    xh1, rstd1, g1 = c["c1"]
    xh2, rstd2, g2 = c["c2"]
    bn1, bn2 = c["bn1"], c["bn2"]
    ws, st, cond = c["ws"], c["st"], c["cond"]
    B, H, W, Ci = bn1.shape
    H2, W2, Co = 2 * H, 2 * W, bn2.shape[3]
    cnt1, cnt2 = B * H * W, B * H2 * W2
    bias1 = (bn1 - g1[:, None, None, :] * xh1)[:, 0, 0, :]
    bias2 = (bn2 - g2[:, None, None, :] * xh2)[:, 0, 0, :]
    # --- ambiguous ReLU inputs
    band1 = _bn_band(bn1, xh1, g1)
    amb1 = np.abs(bn1) <= band1
    # a1 = bf16(relu(bn1)) may round the other way where bn1 is that close to
    # a rounding boundary, moving h1 by a spacing times the filter
    a1_flip = tie_ambiguous(bn1, band1) & (bn1 > 0)
    f1 = c["f1"] / c["s1"]                   # the effective (normalised) operands
    w2 = c["w2"] / c["s2"]
    f1a = np.abs(f1)
    acc1 = L.up2_conv(c["a1"], f1)
    h1_pre = acc1 + p["conv1.b"]
    band_h1 = (conv_band(L.up2_conv(c["a1"] ** 2, f1 ** 2), 4 * Ci) + SIGMA_EPS * np.abs(acc1) +
               L.up2_conv(ulp_bf16(bn1) * a1_flip, f1a))
    # h1 = bf16(...) may itself round the other way: one more spacing
    dh1_val = band_h1 + ulp_bf16(h1_pre) * tie_ambiguous(h1_pre, band_h1)
    band2 = np.abs(g2[:, None, None, :]) * rstd2 * dh1_val + _bn_band(bn2, xh2, g2)
    amb2 = np.abs(bn2) <= band2
    # --- the oracle's backward values the responses need
    da2 = L.conv2d_dgrad(dy, w2)
    dh1, _, _ = L.cbn_bwd(da2 * (bn2 > 0), c["c2"])
    da1 = L.up2_conv_dgrad(dh1, f1)
    A = L.up2(c["a1"])                       # conv1's operand at full resolution
    Ap = _pad1(A)
    Q = L.conv2d(A, ws["conv1.w"])           # <patch at a pixel, W1[c]> per pixel and c
    S0 = L.conv2d_wgrad(np.ones((B, H2, W2, 1)), A, 3)[0]        # (3, 3, Ci)
    S1 = L.conv2d_wgrad(xh2, A, 3)                               # (Co, 3, 3, Ci)
    sQ, sxQ, sx = Q.sum(axis=(0, 1, 2)), (xh2 * Q).sum(axis=(0, 1, 2)), xh2.sum(axis=(0, 1, 2))
    proj = {k: 0.0 for k in ("conv1.w", "bn1.gain", "bn1.bias", "bn2.gain", "bn2.bias")}
    row = {k: np.zeros(ws[k].shape) for k in ("conv1.w", "bn1.gain", "bn1.bias", "bn2.gain", "bn2.bias")}
    conv1b = np.zeros(Co)
    dx_b = np.zeros(bn1.shape)               # local parts of dx
    M1, M2 = np.zeros(Ci), np.zeros(Ci)      # their batch-mean spreads, summed
    dcond_b = np.zeros(cond.shape)
    spread = np.zeros(bn2.shape)             # per channel: sum over flips of the dh1 spread bound
    mask1 = (bn1 > 0).astype(np.float64)
    # dgain1 / dbias1 of the spread fields 1 and xh2 on channel ch, pushed
    # through conv1's data gradient: by adjointness, sums of the cBN1-side
    # factors (mask1 xh1, mask1) over the shifted source grid against the
    # fields on each parity class, one batched product per (class, tap)
    chans = np.unique(np.nonzero(amb2)[3])
    slot = {ch: n for n, ch in enumerate(chans)}
    Pg = np.zeros((2, B, len(chans), Ci))    # [field 1 / xh2][b, ch, ci] for dgain1
    Pb = np.zeros((2, B, len(chans), Ci))    # the same for dbias1
    if len(chans):
        Gg = _pad1(mask1 * xh1)
        Gb = _pad1(mask1)
        for a in range(2):
            for bb in range(2):
                X = xh2[:, a::2, bb::2, :][..., chans].reshape(B, H * W, len(chans))
                for t in range(2):
                    for u in range(2):
                        Fk = f1[a, bb][chans][:, t, u, :]               # (nch, Ci)
                        for n_, Gp in ((0, Gg), (1, Gb)):
                            Gs = Gp[:, a + t:a + t + H, bb + u:bb + u + W, :].reshape(B, H * W, Ci)
                            tgt = Pg if n_ == 0 else Pb
                            tgt[0] += Gs.sum(axis=1)[:, None, :] * Fk[None]
                            tgt[1] += np.matmul(X.transpose(0, 2, 1), Gs) * Fk[None]

    def through_cbn1(pts, scale, dg, db, rd):
        """A flip's change of dbn1: the points pts (vectors times scale) as
        local dx and its batch-mean moments, and the signed changes dg, db of
        dgain1 / dbias1 (B, Ci) into the bn1 linears and dcond (rd: dcond's
        change from the bn2 side of the same flip)."""
        m1, m2 = np.zeros(Ci), np.zeros(Ci)
        for (b, h, w, vec) in pts:
            v = scale * vec
            # where cBN1's own mask is ambiguous the change may pass or not
            vp = v * mask1[b, h, w]
            va = np.abs(v) * amb1[b, h, w]
            dx_b[b, h, w] += np.abs(rstd1 * g1[b] * vp) + rstd1 * np.abs(g1[b]) * va
            m1 += g1[b] * vp / cnt1
            m2 += g1[b] * vp * xh1[b, h, w] / cnt1
            M1[...] += np.abs(g1[b]) * va / cnt1
            M2[...] += np.abs(g1[b]) * va * np.abs(xh1[b, h, w]) / cnt1
            dg[b] += vp * xh1[b, h, w]
            db[b] += vp
            if va.any():
                row["bn1.gain"][...] += np.outer(va * np.abs(xh1[b, h, w]), np.abs(cond[b]))
                row["bn1.bias"][...] += np.outer(va, np.abs(cond[b]))
                dcond_b[b] += (va * np.abs(xh1[b, h, w])) @ np.abs(ws["bn1.gain"]) + va @ np.abs(ws["bn1.bias"])
        M1[...] += np.abs(m1)
        M2[...] += np.abs(m2)
        row["bn1.gain"] += np.abs(dg.T @ cond)
        row["bn1.bias"] += np.abs(db.T @ cond)
        proj["bn1.gain"] += abs(float((dg * (g1 - 1.0)).sum()))      # cond . Wg1[c] = gain - 1
        proj["bn1.bias"] += abs(float((db * bias1).sum()))
        dcond_b[...] += np.abs(rd + dg @ ws["bn1.gain"] + db @ ws["bn1.bias"])

    # --- flips of cBN2's ReLU: dbn2 moves by da2 at e (sign unknown)
    for (b, i, j, ch) in zip(*np.nonzero(amb2)):
        D = abs(da2[b, i, j, ch])
        xe = xh2[b, i, j, ch]
        k = rstd2[ch] * g2[b, ch] * D
        row["conv1.w"][ch] += np.abs(k * (Ap[b, i:i + 3, j:j + 3, :] - (S0 + xe * S1[ch]) / cnt2))
        proj["conv1.w"] += abs(k * (Q[b, i, j, ch] - (sQ[ch] + xe * sxQ[ch]) / cnt2))
        conv1b[ch] += abs(k * (1.0 - (cnt2 + xe * sx[ch]) / cnt2))
        spread[..., ch] += abs(k) * (1.0 + abs(xe) * np.abs(xh2[..., ch])) / cnt2
        # the bn2 side: dgain2 and dbias2 of (b, ch) move by D xe and D
        row["bn2.gain"][ch] += np.abs(D * xe * cond[b])
        row["bn2.bias"][ch] += np.abs(D * cond[b])
        proj["bn2.gain"] += abs(D * xe * (g2[b, ch] - 1.0))
        proj["bn2.bias"] += abs(D * bias2[b, ch])
        rd = np.zeros(cond.shape)
        rd[b] = D * xe * ws["bn2.gain"][ch] + D * ws["bn2.bias"][ch]
        n_ = slot[ch]
        dg = -k * (Pg[0, :, n_] + xe * Pg[1, :, n_]) / cnt2
        db = -k * (Pb[0, :, n_] + xe * Pb[1, :, n_]) / cnt2
        through_cbn1(_local_dgrad(f1, ch, b, i, j, bn1.shape), k, dg, db, rd)
    # --- flips of cBN1's ReLU: dbn1 moves by da1 at e
    for (b, i, j, ch) in zip(*np.nonzero(amb1)):
        vec = np.zeros(Ci)
        vec[ch] = da1[b, i, j, ch]
        dx_b[b, i, j, ch] += abs(rstd1[ch] * g1[b, ch] * vec[ch])
        M1[ch] += abs(g1[b, ch] * vec[ch]) / cnt1
        M2[ch] += abs(g1[b, ch] * vec[ch] * xh1[b, i, j, ch]) / cnt1
        dg, db = np.zeros((B, Ci)), np.zeros((B, Ci))
        dg[b, ch], db[b, ch] = vec[ch] * xh1[b, i, j, ch], vec[ch]
        through_cbn1([], 1.0, dg, db, np.zeros(cond.shape))
    # --- the spread's share of dx (and of dgain1 / dbias1 where cBN1's own
    # mask is ambiguous) in absolute value
    dsp_in = L.up2_conv_dgrad(spread, f1a)
    dsp, _, _ = _cbn_abs(dsp_in * ((bn1 > 0) | amb1), xh1, rstd1, g1)
    _, dga, dba = _cbn_abs(dsp_in * amb1, xh1, rstd1, g1)
    ca = np.abs(cond)
    row["bn1.gain"] += dga.T @ ca
    row["bn1.bias"] += dba.T @ ca
    proj["bn1.gain"] += float((dga * np.abs(g1 - 1.0)).sum())
    proj["bn1.bias"] += float((dba * np.abs(bias1)).sum())
    out = {"conv1.w": sn_bound(row["conv1.w"], proj["conv1.w"], st["conv1.w"]),
           "conv1.b_l1": conv1b,
           "dx": dx_b + rstd1 * (M1 + np.abs(xh1) * M2) + dsp,
           "dcond": dcond_b + dga @ np.abs(ws["bn1.gain"]) + dba @ np.abs(ws["bn1.bias"])}
    for k in ("bn1.gain", "bn1.bias", "bn2.gain", "bn2.bias"):
        out[k] = sn_bound(row[k], proj[k], st[k])
    info = {"counts": {"amb_bn1": int(amb1.sum()), "amb_bn2": int(amb2.sum()), "round_a1": int(a1_flip.sum())},
            "masks": {"bn1": amb1, "bn2": amb2}}
    return out, info


def dblock_bounds(cache, dy, down, preact):
    """Bounds for the discriminator block's backward in bf16: where conv1's
    output h lies within the summation band of zero its ReLU mask may flip,
    moving dh by |conv2^T dy| there (no batch coupling: each flip's change is
    local).  Returns ({"conv1.w", "conv1.b", "dx"}, {"counts", "masks"})."""
    c = cache
    w1, w2 = c["w1"] / c["s1"], c["w2"] / c["s2"]     # the effective (normalised) operands
    da = L.pool2_conv_dgrad(dy, w2) if down else L.conv2d_dgrad(dy, w2)
    k1 = 9 * c["a0"].shape[3]
    band = conv_band(L.conv2d(c["a0"] ** 2, w1 ** 2), k1) + SIGMA_EPS * np.abs(L.conv2d(c["a0"], w1))
    amb = np.abs(c["h"]) <= band
    ddh = np.abs(da) * amb
    proj = float((ddh * np.abs(L.conv2d(c["a0"], c["ws"]["conv1.w"]))).sum())
    out = {"conv1.w": sn_bound(L.conv2d_wgrad(ddh, np.abs(c["a0"]), 3), proj, c["st"]["conv1.w"]),
           "conv1.b": ddh.sum(axis=(0, 1, 2))}
    ddx = L.conv2d_dgrad(ddh, np.abs(w1))
    if preact:
        ddx = ddx * (c["x"] > 0)
    out["dx"] = ddx
    return out, {"counts": {"amb_h": int(amb.sum())}, "masks": {"h": amb}}
