"""The group-scale division of the scaled formats (E4M3, INT8, INT4).

The kernels compute s = fl32(m / qmax) as fma(m, zh, fl32(m zl)) with
zh = fl32(1 / qmax), zl = fl32(1 / qmax - zh) for m in [2^-112, FLT_MAX]
(Brisebarre, Muller and Raina, 2004). The identity is a property of IEEE fp32
arithmetic (fused multiply-add and division both correctly rounded), so it is
checked here on the host: every mantissa at several exponents, and a stride
through all the others. The constants are the ones the device code uses.
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
  const int full[7] = {-112, -64, -1, 0, 1, 100, 127};
  long bad = 0, n = 0;
  for (int t = 0; t < 3; ++t) {
    if (zh[t] != 1.0f / qmax[t]) { printf("zh\n"); return 2; }
    for (int e = -112; e <= 127; ++e) {
      int all = 0;
      for (int i = 0; i < 7; ++i) all |= (full[i] == e);
      const uint32_t step = all ? 1u : 4099u;
      for (uint32_t m = 0; m < (1u << 23); m += step) {
        const float x = bits(((uint32_t)(e + 127) << 23) | m);
        const float q = fmaf(x, zh[t], x * zl[t]);
        ++n;
        if (q != x / qmax[t]) ++bad;
      }
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
        r = subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", exe, c, "-lm"],
                           capture_output=True, text=True)
        if r.returncode != 0:
            pytest.skip("no C compiler: " + r.stderr[-200:])
        out = subprocess.run([exe], capture_output=True, text=True, timeout=300)
        n, bad = map(int, out.stdout.split())
        assert out.returncode == 0 and bad == 0 and n > 100_000_000, out.stdout
