"""The scale's division by L = 2^b - 1 is computed as q0 = d*RN(1/L) followed
by one fma residual step.  This CPU check runs the same sequence with IEEE
fp32 fma on a strided sample of all non-negative finite fp32 dividends (every
pattern with HG_EXHAUSTIVE=1) and compares with the IEEE quotient.  The GPU
test test_gpu_arith.py repeats it exhaustively with the kernels' helper."""
import os
import subprocess
import tempfile

SRC = r'''
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
int main(int argc, char** argv) {
  unsigned stride = (unsigned)atoi(argv[1]);
  const float Ls[3] = {3.0f, 7.0f, 15.0f};
  const float ys[3] = {0x1.555556p-2f, 0x1.24924ap-3f, 0x1.111112p-4f};
  unsigned long long bad = 0, checked = 0;
  for (int i = 0; i < 3; ++i) {
    if (ys[i] != 1.0f / Ls[i]) { printf("bad constant %d\n", i); return 2; }
    for (uint64_t u = 0; u < 0x7F800000ull; u += stride) {
      float d; uint32_t b = (uint32_t)u; memcpy(&d, &b, 4);
      volatile float ref = d / Ls[i];
      float q0 = d * ys[i];
      float r = fmaf(-q0, Ls[i], d);
      float q1 = fmaf(r, ys[i], q0);
      checked++;
      if (q1 != ref) bad++;
    }
  }
  printf("%llu %llu\n", checked, bad);
  return bad != 0;
}
'''


def test_division_by_levels_sampled():
    stride = 1 if os.environ.get("HG_EXHAUSTIVE") else 61
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "div.c"), os.path.join(d, "div")
        open(src, "w").write(SRC.replace("#include <string.h>", "#include <string.h>\n#include <stdlib.h>"))
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-o", exe, src, "-lm"])
        out = subprocess.run([exe, str(stride)], capture_output=True, text=True, timeout=1200)
        checked, bad = map(int, out.stdout.split())
        assert out.returncode == 0 and bad == 0 and checked > 0
