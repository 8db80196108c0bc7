"""The launch-time-invariant division used by the kernels (csrc/fastdiv.h)
equals integer division for every numerator below 2^31: compiled for the
CPU from the same header and checked on edge cases and random values."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SRC = r'''
#include <stdio.h>
#include <stdlib.h>
#include "fastdiv.h"
int main(void) {
  unsigned long long bad = 0, n = 0;
  unsigned s = 12345;
  for (uint32_t d = 1; d <= 5000; ++d) {
    FastDiv f = make_fastdiv(d);
    uint32_t xs[] = {0, 1, d - 1, d, d + 1, 2 * d - 1, 2 * d, 0x7FFFFFFFu, 0x7FFFFFFEu, 0x7FFFFFFFu - d};
    for (int i = 0; i < 10; ++i) { uint32_t x = xs[i] & 0x7FFFFFFFu; n++; bad += fdiv(x, f) != x / d; }
    for (uint32_t x = 0; x < 3000; ++x) { n++; bad += fdiv(x, f) != x / d; }
    for (int i = 0; i < 300; ++i) { s = s * 1103515245u + 12345u; uint32_t x = s & 0x7FFFFFFFu; n++; bad += fdiv(x, f) != x / d; }
  }
  for (int i = 0; i < 300000; ++i) {
    s = s * 1103515245u + 12345u; uint32_t d = (s & 0x7FFFFFFFu) | 1u;
    s = s * 1103515245u + 12345u; uint32_t x = s & 0x7FFFFFFFu;
    FastDiv f = make_fastdiv(d); n++; bad += fdiv(x, f) != x / d;
  }
  printf("%llu %llu\n", n, bad);
  return bad != 0;
}
'''


def test_fastdiv_exact(tmp_path):
    c = tmp_path / "fd.c"
    c.write_text(SRC)
    exe = tmp_path / "fd"
    subprocess.check_call(["gcc", "-O2", "-I", os.path.join(ROOT, "paper_2609_35481_amd", "csrc"),
                           "-o", str(exe), str(c)])
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout
    n, bad = map(int, out.stdout.split())
    assert n > 10**7 and bad == 0
