"""The group-scale division of the scaled formats (E4M3, INT8, INT4), exhaustively.

The kernels compute s = fl32(m / qmax) as fma(m, zh, fl32(m zl)) with
zh = fl32(1 / qmax), zl = fl32(1 / qmax - zh) for m in [2^-112, FLT_MAX]
(Brisebarre, Muller and Raina, "Accelerating correctly rounded floating-point
division when the divisor is known in advance", 2004). The identity is a
property of IEEE fp32 arithmetic (fused multiply-add and division both
correctly rounded), so it is checked here on the host for every fp32 value in
that range (every exponent from -112 to 127, all 2^23 mantissas) and each of the
three qmax values, with the constants the device code uses. The device side of
the scale (the division on the device and the reciprocal) is checked, also
exhaustively, by tests/test_gpu_scale_math.py.
"""
import os
import subprocess
import tempfile

import pytest

SRC = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
static float bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
int main(void) {
  const float qmax[3] = {448.0f, 127.0f, 7.0f};
  const float zh[3] = {0x1.24924ap-9f, 0x1.020408p-7f, 0x1.24924ap-3f};
  const float zl[3] = {-0x1.b6db6ep-34f, 0x1.020408p-35f, -0x1.b6db6ep-28f};
  long bad = 0, n = 0;
  for (int t = 0; t < 3; ++t) {
    if (zh[t] != 1.0f / qmax[t]) { printf("zh\n"); return 2; }
    if ((double)zl[t] != (double)(float)(1.0 / qmax[t] - (double)zh[t])) { printf("zl\n"); return 2; }
    #pragma omp parallel for reduction(+ : bad, n) schedule(dynamic)
    for (int e = -112; e <= 127; ++e) {
      long b = 0;
      for (uint32_t m = 0; m < (1u << 23); ++m) {
        const float x = bits(((uint32_t)(e + 127) << 23) | m);
        const float q = fmaf(x, zh[t], x * zl[t]);
        b += (q != x / qmax[t]);
      }
      bad += b;
      n += 1L << 23;
    }
  }
  printf("%ld %ld\n", n, bad);
  return bad != 0;
}
"""


def test_fma_division_by_qmax_is_correctly_rounded():
    with tempfile.TemporaryDirectory() as d:
        c, exe = os.path.join(d, "div.c"), os.path.join(d, "div")
        with open(c, "w") as f:
            f.write(SRC)
        r = subprocess.run(["gcc", "-O3", "-march=native", "-fopenmp", "-ffp-contract=off",
                            "-fno-fast-math", "-o", exe, c, "-lm"], capture_output=True, text=True)
        if r.returncode != 0:
            pytest.skip("no C compiler: " + r.stderr[-200:])
        out = subprocess.run([exe], capture_output=True, text=True, timeout=600)
        n, bad = map(int, out.stdout.split())
        # 3 divisors x 240 binades x 2^23 mantissas
        assert out.returncode == 0 and bad == 0 and n == 3 * 240 * (1 << 23), out.stdout
