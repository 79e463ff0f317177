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
    """Round float64 values to bfloat16 (round to nearest, ties to even).

    A normal bfloat16 keeps 8 significant bits, i.e. the top 7 of float64's
    52 stored fraction bits: rounding to nearest even at bit 45 of the
    float64 pattern (add half the dropped range, minus one unless the kept
    last bit is odd, then clear the dropped bits) gives it exactly, a carry
    into the exponent included.  Below 2**-126 bfloat16 has a fixed quantum
    of 2**-133; from _OVERFLOW on the result is +-inf; NaN stays NaN."""
    x = np.asarray(x, dtype=np.float64)
    bits = np.ascontiguousarray(x).view(np.uint64)
    odd = (bits >> np.uint64(45)) & np.uint64(1)
    r = (bits + (np.uint64((1 << 44) - 1) + odd)) & ~np.uint64((1 << 45) - 1)
    out = r.view(np.float64).reshape(x.shape)
    ax = np.abs(x)
    sub = ax < 2.0 ** -126
    if sub.any():
        out = out.copy()
        out[sub] = np.round(x[sub] * 2.0 ** 133) * 2.0 ** -133
    big = ~(ax < _OVERFLOW)                      # overflow, inf and NaN
    if big.any():
        out = out.copy() if not sub.any() else out
        out[big] = np.where(np.isnan(x[big]), x[big], np.copysign(np.inf, x[big]))
    return out


def identity(x):
    return np.asarray(x, dtype=np.float64)


def rounder(emulate_bf16):
    """Storage rounding used at every point where the GPU path stores bf16."""
    return bf16 if emulate_bf16 else identity
