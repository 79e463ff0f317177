"""Host-side logic of the native library, checked on the CPU.

The index decoding of the weight-gradient kernels divides pixel indices by
the grid width and height with a multiply-high (Granlund and Montgomery,
1994).  The header is plain C++: compile it with g++ and compare against
integer division over edge cases and random pairs.
"""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paragan_2411_03999_amd", "csrc")

DRIVER = r"""
#include <cstdio>
#include "fastdiv.hpp"
int main() {
  unsigned d, n;
  unsigned long long bad = 0, cnt = 0;
  while (std::scanf("%u %u", &d, &n) == 2) {
    const pg::FastDiv f = pg::make_fastdiv(d);
    ++cnt;
    if (pg::fdiv(n, f) != n / d) {
      ++bad;
      if (bad < 5) std::printf("mismatch d=%u n=%u got %u\n", d, n, pg::fdiv(n, f));
    }
  }
  std::printf("checked %llu bad %llu\n", cnt, bad);
  return bad != 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_fastdiv_matches_integer_division():
    rng = np.random.default_rng(7)
    pairs = []
    divisors = [1, 2, 3, 4, 5, 7, 8, 9, 16, 31, 32, 33, 63, 64, 65, 96, 127, 128, 129, 192, 255, 256, 288,
                384, 1023, 1024, 1536, 4096, 65535, 65536, 1 << 20, (1 << 31) - 1]
    limit = (1 << 31) - 1
    for d in divisors:
        for n in [0, 1, d - 1, d, d + 1, 2 * d - 1, 2 * d, limit, limit - 1, limit - d]:
            if 0 <= n <= limit:
                pairs.append((d, n))
        for n in rng.integers(0, limit, 200):
            pairs.append((d, int(n)))
    for d, n in zip(rng.integers(1, 1 << 31, 5000), rng.integers(0, 1 << 31, 5000)):
        pairs.append((int(d), int(n)))
    with tempfile.TemporaryDirectory() as tmp:
        src = os.path.join(tmp, "drv.cpp")
        exe = os.path.join(tmp, "drv")
        open(src, "w").write(DRIVER)
        subprocess.run(["g++", "-O2", "-std=c++17", "-I", CSRC, src, "-o", exe], check=True)
        inp = "\n".join("%d %d" % p for p in pairs)
        r = subprocess.run([exe], input=inp, capture_output=True, text=True)
        assert r.returncode == 0, r.stdout
        assert ("checked %d bad 0" % len(pairs)) in r.stdout
