"""The decoder's log1p for arguments in [0, 1] (the two-score log-sum-exp of
the recombination step: m + log1p(exp(-d)), d >= 0), compiled for the host
from the same header the kernels include and checked against the C
library's 80-bit long double log1p: never more than 0.75 ulp off and
correctly rounded in at least 98 % of a million seeded arguments, exact at 0
and at 1, and the log-sum-exp built on it within 3 ulp of the one built on
the C library's double log1p (the oracle's; the two differ by up to 2 ulp
where m is small and cancels).  Dropping the quotient's low part fails all
three bounds.  No GPU is needed."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_14002_amd", "csrc")

HARNESS = r"""
#include "lb_device.h"
#include <cmath>
#include <cstdint>
#include <cstdio>

static uint64_t state = 0x9E3779B97F4A7C15ull;
static double uniform() {  // SplitMix64 stream -> [0, 1)
  uint64_t z = (state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  return static_cast<double>(z >> 11) * 0x1p-53;
}
static double ulp_of(double x) {
  int e;
  std::frexp(x, &e);
  return std::ldexp(1.0, e - 53);
}
int main() {
  const long n = 1000000;
  long exact = 0;
  double worst = 0.0, worst_lse = 0.0;
  for (long i = 0; i < n; ++i) {
    // d spread over [0, 2) and [0, 60): e = exp(-d) covers (0, 1]
    const double d = (i & 1) ? 60.0 * uniform() : 2.0 * uniform();
    const double e = std::exp(-d);
    const long double ref = std::log1p(static_cast<long double>(e));
    const double got = lb::log1p_unit(e);
    if (got == static_cast<double>(ref)) ++exact;
    const double cr = static_cast<double>(ref);
    if (cr != 0.0) {
      const double err = static_cast<double>(std::fabs(static_cast<long double>(got) - ref)) / ulp_of(cr);
      if (err > worst) worst = err;
    }
    const double m = -std::ldexp(1.0 + uniform(), static_cast<int>(i % 12));
    const double a = m + got, b = m + std::log1p(e);
    const double el = std::fabs(a - b) / ulp_of(b);
    if (el > worst_lse) worst_lse = el;
  }
  std::printf("%.6f %.6f %.6f %.17g %.17g\n", static_cast<double>(exact) / n, worst, worst_lse,
              lb::log1p_unit(0.0), lb::log1p_unit(1.0));
  return 0;
}
"""


def test_log1p_unit_matches_an_80_bit_log1p(tmp_path):
    hipcc = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)
    if hipcc is None:
        pytest.skip("hipcc not found")
    src = tmp_path / "log1p_unit.cpp"
    src.write_text(HARNESS)
    exe = tmp_path / "log1p_unit"
    inc = os.path.join(ROOT, "include")
    subprocess.run([hipcc, "-O2", "-ffp-contract=off", "-I", CSRC, "-I", inc, "-o", str(exe), str(src)],
                   check=True, capture_output=True, timeout=300)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=120).stdout.split()
    frac_exact, worst, worst_lse, at0, at1 = (float(x) for x in out)
    assert frac_exact >= 0.98, frac_exact
    assert worst <= 0.75, worst
    assert worst_lse <= 3.0, worst_lse
    assert at0 == 0.0
    assert at1 == 0.6931471805599453  # log(2), correctly rounded
