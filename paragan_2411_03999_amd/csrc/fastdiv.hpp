// Division by a run-time invariant divisor with one multiply-high, the
// round-up method of Granlund and Montgomery ("Division by Invariant
// Integers using Multiplication", PLDI 1994, Fig. 4.1, N = 32):
//   l = ceil(log2 d),  m = floor(2^32 (2^l - d) / d) + 1,
//   n / d = (mulhi(m, n) + n) >> l.
// Valid for 1 <= d < 2^31 and 0 <= n < 2^31 (then mulhi + n < 2^32).
// Plain C++ so that host tests can compile it; the kernels include it
// through ops.hpp.
#pragma once
#include <cstdint>

#if defined(__HIP__)
#define PG_HD __host__ __device__ __forceinline__
#else
#define PG_HD inline
#endif

namespace pg {

struct FastDiv {
  uint32_t d, mul, shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while (l < 32 && (1ull << l) < d) ++l;
  const uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
  return FastDiv{d, (uint32_t)m, l};
}

PG_HD uint32_t fdiv(uint32_t n, const FastDiv& f) {
  const uint32_t hi = (uint32_t)(((uint64_t)n * f.mul) >> 32);
  return (hi + n) >> f.shift;
}

}  // namespace pg
