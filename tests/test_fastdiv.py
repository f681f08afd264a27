"""Host check of the launch-time integer division used in kernel index math
(multiply-high + add + shift): exhaustive over small numerators and divisors,
sampled up to 2^31 - 1, against plain integer division."""
import os
import subprocess
import tempfile

SRC = r"""
#include "fastdiv.h"
#include <cstdio>
#include <initializer_list>
#include <cstdint>
int main() {
  unsigned long long bad = 0, n_checked = 0;
  uint64_t x = 88172645463325252ull;
  for (uint32_t d = 1; d <= 4096; ++d) {
    cf::FastDiv f = cf::make_fastdiv(d);
    for (int n = 0; n < 20000; ++n, ++n_checked) bad += cf::fdiv_host(n, f) != n / (int)d;
    for (int k = 0; k < 20000; ++k, ++n_checked) {
      x ^= x << 13; x ^= x >> 7; x ^= x << 17;
      int n = (int)(x & 0x7fffffffu);
      bad += cf::fdiv_host(n, f) != n / (int)d;
    }
    bad += cf::fdiv_host(0x7fffffff, f) != 0x7fffffff / (int)d;
  }
  for (uint32_t d : {65535u, 65536u, 65537u, 1000003u, 1u << 30, 0x7fffffffu}) {
    cf::FastDiv f = cf::make_fastdiv(d);
    for (int k = 0; k < 100000; ++k, ++n_checked) {
      x ^= x << 13; x ^= x >> 7; x ^= x << 17;
      int n = (int)(x & 0x7fffffffu);
      bad += cf::fdiv_host(n, f) != n / (int)d;
    }
  }
  printf("%llu %llu\n", bad, n_checked);
  return bad != 0;
}
"""


def test_fastdiv_matches_integer_division():
    inc = os.path.join(os.path.dirname(__file__), "..", "paper_1808_04728_amd", "csrc")
    with tempfile.TemporaryDirectory() as td:
        src = os.path.join(td, "t.cpp")
        exe = os.path.join(td, "t")
        open(src, "w").write(SRC)
        subprocess.run(["g++", "-O2", "-std=c++17", "-I", inc, src, "-o", exe], check=True)
        r = subprocess.run([exe], capture_output=True, text=True)
        bad, checked = map(int, r.stdout.split())
        assert r.returncode == 0 and bad == 0, r.stdout
        assert checked > 100_000_000
