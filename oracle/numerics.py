"""bfloat16 storage emulation for the oracle (test infrastructure only).

The paper trains with bfloat16 activations and keeps the last generator and
discriminator layers in fp32 (Design, "System Optimizations"; Implementation,
"Mixed-Precision Training").  bfloat16 keeps fp32's 8 exponent bits and 8
significant bits (7 stored).  `bf16` rounds a float64 array to the nearest
bfloat16 value, ties to even, directly from float64 (no double rounding via
fp32); overflow goes to +-inf, NaN stays NaN, subnormals keep a fixed quantum
of 2**-133.
"""
import numpy as np

_BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127      # largest finite bfloat16
_OVERFLOW = (2.0 - 2.0 ** -8) * 2.0 ** 127      # rounds up to inf at/after this


def bf16(x):
    """Round float64 values to bfloat16 (round to nearest, ties to even)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    ax = np.abs(x)
    finite = np.isfinite(x)
    normal = finite & (ax >= 2.0 ** -126)
    # normal range: x = m * 2**e with 0.5 <= |m| < 1; keep 8 significant bits
    m, e = np.frexp(np.where(normal, x, 1.0))
    q = np.round(m * 256.0)                      # numpy rounds half to even
    out[...] = np.ldexp(q, e - 8)
    # subnormal range: fixed quantum 2**-133
    sub = finite & ~normal
    out[sub] = np.round(x[sub] * 2.0 ** 133) * 2.0 ** -133
    over = finite & (ax >= _OVERFLOW)
    out[over] = np.copysign(np.inf, x[over])
    out[~finite] = x[~finite]
    return out


def identity(x):
    return np.asarray(x, dtype=np.float64)


def rounder(emulate_bf16):
    """Storage rounding used at every point where the GPU path stores bf16."""
    return bf16 if emulate_bf16 else identity
