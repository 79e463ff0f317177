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


# kernel-template instances (profiler names) launched by the parity tests of
# this session, for the coverage check of the benchmark's instances
SEEN = set()


def context():
    """A library context whose convolution, weight-gradient and attention
    launches are recorded by name (harvest() collects them)."""
    from paragan_2411_03999_amd import lib
    ctx = lib.Context()
    lib.paragan_profile(ctx, 1)
    return ctx


def harvest(ctx):
    from paragan_2411_03999_amd import lib
    for st in lib.paragan_profile_read(ctx):
        SEEN.add(st["name"])


def optim(spec):
    """lib.Optim of an oracle OptSpec."""
    from paragan_2411_03999_amd import lib
    return lib.Optim({"adam": lib.ADAM, "adabelief": lib.ADABELIEF}[spec.kind], spec.lr, spec.beta1, spec.beta2,
                     spec.eps)


def biggan_desc(a, B, hp):
    """The C descriptor of an oracle architecture and hyper-parameters."""
    from paragan_2411_03999_amd import lib
    d = lib.BigganDesc()
    d.img, d.ch, d.n_g, d.n_d = a.img, a.ch, a.n_g, len(a.d_mult)
    for i, m in enumerate(a.g_mult):
        d.g_mult[i] = m
    for j, (m, dn) in enumerate(zip(a.d_mult, a.d_down)):
        d.d_mult[j], d.d_down[j] = m, dn
    d.attn_res, d.n_classes, d.dz, d.shared_dim, d.B = a.attn_res, a.n_classes, a.dz, a.shared_dim, B
    d.n_power_iter, d.bn_eps, d.sn_eps = hp.n_power_iter, hp.bn_eps, hp.sn_eps
    d.opt_g, d.opt_d = optim(hp.opt_g), optim(hp.opt_d)
    return d
