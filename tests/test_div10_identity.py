"""The simulation kernels divide the fp32 gap EMA by 10 with one product and
one residual step instead of an IEEE division, inside [2^-64, 2^64].  This
checks, for every float of that window, that the result equals the
correctly rounded quotient, which is what the oracle's division computes
(eq. (ema)).  Plain C on the host: glibc's fmaf is the fused operation."""
import os
import subprocess
import tempfile

import pytest

SRC = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
int main(void) {
  const float lo = 0x1p-64f, hi = 0x1p64f;
  uint32_t a, b;
  memcpy(&a, &lo, 4);
  memcpy(&b, &hi, 4);
  unsigned long long n = 0, bad = 0;
  for (uint32_t u = a; u <= b; ++u) {
    float s;
    memcpy(&s, &u, 4);
    volatile float want = s / 10.0f;
    float q0 = s * 0.1f;
    float r = fmaf(-q0, 10.0f, s);
    float q = fmaf(r, 0.1f, q0);
    float w = want;
    if (memcmp(&q, &w, 4) != 0) bad++;
    n++;
  }
  printf("%llu %llu\n", n, bad);
  return 0;
}
"""


def test_residual_division_by_ten_is_exact_on_its_window():
    with tempfile.TemporaryDirectory() as d:
        c, exe = os.path.join(d, "div10.c"), os.path.join(d, "div10")
        open(c, "w").write(SRC)
        try:
            subprocess.run(["gcc", "-O2", "-ffp-contract=off", c, "-o", exe, "-lm"], check=True)
        except (OSError, subprocess.CalledProcessError) as e:
            pytest.skip("no C compiler: %s" % e)
        n, bad = map(int, subprocess.run([exe], check=True, capture_output=True, text=True,
                                         timeout=300).stdout.split())
    assert n == 128 * (1 << 23) + 1   # 128 binades of 2^23 floats, and 2^64 itself
    assert bad == 0
