"""Shared helpers for the GPU parity tests: tolerances and device setup.

Tolerances (the bar for this hot path):
* fp32 path: max_i |g_i - r_i| / max(|r_i|, 1e-2 max|r|) <= 1e-4 per tensor
  (elementwise relative error, floored at 1% of the tensor's scale: below
  that, fp32 accumulation over hundreds of terms and two convolutions
  cannot resolve a value, and a 1e-4 relative bar there would demand
  sub-ulp agreement);
* bf16 path: max |g - r| / max |r| <= 2e-2 per tensor, against the oracle
  in bf16-storage emulation (so the two differ only by summation order and
  the rare bf16 rounding flip that order causes).
"""
import numpy as np
import pytest

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def rel_err_f32(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    floor = 1e-2 * np.abs(r).max() if r.size else 0.0
    den = np.maximum(np.abs(r), max(floor, 1e-30))
    return float((np.abs(g - r) / den).max()) if r.size else 0.0


def norm_maxabs(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    m = np.abs(r).max() if r.size else 0.0
    return float(np.abs(g - r).max() / max(m, 1e-30)) if r.size else 0.0


class Report:
    """Collects per-tensor errors; fails at the end with every error shown."""

    def __init__(self):
        self.err = {}
        self.bad = []

    def add(self, name, e, tol):
        self.err[name] = e
        if not (e <= tol):
            self.bad.append("%s: error %.3g > %.3g" % (name, e, tol))

    def done(self):
        print("errors", {k: "%.2e" % v for k, v in self.err.items()}, flush=True)
        assert not self.bad, "; ".join(self.bad)


def check(name, g, r, bf16, report):
    assert np.all(np.isfinite(g)), name + ": non-finite GPU values"
    e = norm_maxabs(g, r) if bf16 else rel_err_f32(g, r)
    report.add(name, e, TOL_BF16 if bf16 else TOL_F32)
    return e


def rel_l2(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    return float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))


def kink_pixels(pre, rel=1e-6, radius=1):
    """(N,H,W) mask of pixels within `radius` of an element of the oracle's
    pre-activation `pre` (N,H,W,C) so close to 0 (|v| <= rel * max|pre|)
    that fp32 and fp64 summation may disagree on its sign, i.e. where the
    ReLU mask may legitimately differ.  Derived from the oracle alone."""
    near = (np.abs(pre) <= rel * np.abs(pre).max()).any(axis=3)
    out = near.copy()
    n, h, w = near.shape
    for dh in range(-radius, radius + 1):
        for dw in range(-radius, radius + 1):
            sh = np.zeros_like(near)
            sh[:, max(dh, 0):h + min(dh, 0), max(dw, 0):w + min(dw, 0)] = \
                near[:, max(-dh, 0):h + min(-dh, 0), max(-dw, 0):w + min(-dw, 0)]
            out |= sh
    return out


def check_kinked(name, g, r, excl, bf16, report):
    """Normalised max-abs (or fp32 relative) error outside the kink pixels
    `excl` (N,H,W), and relative L2 error over everything."""
    assert np.all(np.isfinite(g)), name + ": non-finite GPU values"
    keep = ~excl
    tol = TOL_BF16 if bf16 else TOL_F32
    gm, rm = np.asarray(g)[keep], np.asarray(r)[keep]
    e = norm_maxabs(gm, rm) * np.abs(rm).max() / max(np.abs(r).max(), 1e-30) if bf16 else rel_err_f32(gm, rm)
    report.add(name, e, tol)
    report.add(name + ".l2", rel_l2(g, r), tol)
    report.err[name + ".kink_px"] = float(excl.sum())
    return e


def check_with_bound(name, g, r, bound, bf16, report):
    """|g - r| <= tol * scale + bound, elementwise, where `bound` is what
    legitimately ambiguous decisions (ReLU masks of values within fp32
    summation error of zero) can change, computed from the oracle alone.
    Reported error: max of (|g - r| - bound) / scale."""
    assert np.all(np.isfinite(g)), name + ": non-finite GPU values"
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    scale = max(np.abs(r).max(), 1e-30)
    e = float((np.maximum(np.abs(g - r) - bound, 0.0)).max() / scale)
    report.add(name, e, TOL_BF16 if bf16 else TOL_F32)
    report.err[name + ".raw"] = norm_maxabs(g, r)
    report.err[name + ".bound_max"] = float(np.abs(bound).max() / scale)
    return e


def check_cancelling_sum(name, g, r, l1, bf16, report):
    """For a gradient that is a sum whose exact value cancels (e.g. the bias
    in front of a batch-statistics BN, identically zero): compare the
    difference against the L1 mass of the summed terms, per element."""
    e = float((np.abs(np.asarray(g) - np.asarray(r)) / np.maximum(l1, 1e-30)).max())
    report.add(name, e, TOL_BF16 if bf16 else TOL_F32)
    return e


def need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paragan_2411_03999_amd import lib
    lib.load()              # fails loudly when the library is missing
    return torch
