"""Plain CPU oracle for ParaGAN's per-replica BigGAN hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link anything in this package; only
the tests, the smoke check and the CPU-baseline leg of the benchmark use it.

Everything here is slow, obvious numpy in float64, written from the
definitions: direct per-tap convolution sums, two-pass batch statistics,
explicit softmax over all keys, spectral-norm power iteration exactly as
defined, hand-derived backward passes.  Where the GPU path stores bfloat16
the oracle rounds to bfloat16 (round-to-nearest-even) at the same point, so
that the two differ only by summation order.

Modules
-------
numerics  bfloat16 rounding emulation
layers    convolution, resampling, batch norm, spectral norm, attention,
          hinge loss, Adam (forward and backward)
blocks    BigGAN generator / discriminator residual blocks
biggan    parameter layout, full networks, the G+D train step
"""
