"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module generates numbers only; it holds none of the BigGAN arithmetic.
Every tensor comes from its own PCG64 stream, `SeedSequence(seed).spawn()`
in the order the tensors are requested, so a given (seed, request order)
always yields the same values on every machine.

ImageNet (the paper's dataset, Evaluation "Experiment Setup") is not used:
real images are uniform in [-1, 1], latents are N(0, 1), labels are uniform
over the classes.
"""
import numpy as np


class Stream:
    """Hands out independent PCG64 generators in request order."""

    def __init__(self, seed):
        self._ss = np.random.SeedSequence(seed)

    def rng(self):
        return np.random.default_rng(self._ss.spawn(1)[0])

    def normal(self, shape, scale=1.0):
        return self.rng().standard_normal(shape) * scale

    def uniform(self, shape, lo=-1.0, hi=1.0):
        return self.rng().uniform(lo, hi, shape)

    def labels(self, n, n_classes):
        return self.rng().integers(0, n_classes, n).astype(np.int32)

    def orthogonal(self, shape, gain=1.0):
        """Orthogonal init on the (shape[0], prod(shape[1:])) view: QR of a
        Gaussian matrix with the signs fixed by diag(R) (Saxe et al.)."""
        rows = shape[0]
        cols = int(np.prod(shape[1:]))
        a = self.rng().standard_normal((max(rows, cols), min(rows, cols)))
        q, r = np.linalg.qr(a)
        q = q * np.sign(np.diag(r))
        if rows < cols:
            q = q.T
        return (gain * q[:rows, :cols]).reshape(shape)


def init_params(layout, stream, weights="orthogonal", gain_noise=0.1,
                attn_gamma=0.5):
    """Initial values for a {name: shape} layout.

    Weight matrices/kernels (>= 2-D): orthogonal, or Gaussian N(0, 1/fan_in)
    with weights="gaussian" (orthogonal weights have sigma = 1 exactly,
    which would hide a missing spectral normalisation).  Biases: U(+-1/sqrt
    fan_in) so that bias bugs show.  BN gains 1 + noise, BN biases noise.
    Attention gamma is set non-zero so that the attention path matters."""
    out = {}
    fan = {}
    for name, shape in layout.items():
        if len(shape) >= 2:
            fan[name.rsplit(".", 1)[0]] = int(np.prod(shape[1:]))
    for name, shape in layout.items():
        base = name.rsplit(".", 1)[0]
        if name.endswith("gamma"):
            out[name] = np.full(shape, attn_gamma)
        elif len(shape) >= 2:
            if weights == "orthogonal":
                out[name] = stream.orthogonal(shape)
            else:
                out[name] = stream.normal(shape, 1.0 / np.sqrt(np.prod(shape[1:])))
        elif name.endswith("out_bn.gain"):
            out[name] = 1.0 + stream.normal(shape, gain_noise)
        elif name.endswith("out_bn.bias"):
            out[name] = stream.normal(shape, gain_noise)
        else:
            f = fan.get(base, shape[0])
            out[name] = stream.uniform(shape, -1.0 / np.sqrt(f), 1.0 / np.sqrt(f))
    return out


def init_u(layout, sn_keys, stream):
    """Persistent power-iteration vectors u ~ N(0, 1), one per SN weight."""
    return {k: stream.normal((layout[k][0],)) for k in sn_keys}
