"""Integer helpers of the split planner, checked on the host.

The planner divides every tile's page count by each candidate unit size; the
device does this with a multiply-high by a per-divisor magic number
(`udiv_make` / `udiv` in splash_common.hpp, shared verbatim by host and
device).  This test compiles that header with the host compiler and compares
the result with plain integer division: exhaustively over every divisor the
planner can use (1 .. 1024 pages, plus a margin) for all numerators below
2^17, and over numerators next to multiples of the divisor across the whole
32-bit range.  It also checks the candidate part counts of the geometric
continuation against the recurrence they are defined by.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2609_37626_amd", "csrc")

PROGRAM = r"""
#include <stdio.h>
#include <stdint.h>
#include "splash_common.hpp"
using namespace splash;
int main() {
  long bad = 0, checked = 0;
  for (uint32_t d = 1; d <= 1100; ++d) {
    const UDiv u = udiv_make(d);
    for (uint32_t n = 0; n < (1u << 17); ++n, ++checked)
      if (udiv(n, u) != n / d) { if (bad++ < 5) printf("d=%u n=%u got %u\n", d, n, udiv(n, u)); }
    // numerators next to multiples of d across the 32-bit range
    for (uint64_t k = 1; k * d <= 0xffffffffull; k = k * 3 + 7) {
      for (int64_t e = -2; e <= 2; ++e) {
        const int64_t n = (int64_t)(k * d) + e;
        if (n < 0 || n > 0xffffffffll) continue;
        ++checked;
        if (udiv((uint32_t)n, u) != (uint32_t)n / d) { if (bad++ < 5) printf("d=%u n=%lld\n", d, (long long)n); }
      }
    }
    ++checked;
    if (udiv(0xffffffffu, u) != 0xffffffffu / d) bad++;
  }
  // divisors across the whole supported range
  for (uint64_t d = 2; d <= 0x80000000ull; d = d * 5 / 3 + 1) {
    const UDiv u = udiv_make((uint32_t)d);
    for (uint64_t n = 0; n <= 0xffffffffull; n += 0x10001ull * 7 + d) {
      ++checked;
      if (udiv((uint32_t)n, u) != (uint32_t)(n / d)) { if (bad++ < 5) printf("d=%llu n=%llu\n", (unsigned long long)d, (unsigned long long)n); }
    }
  }
  // part counts: k + 1 below 64, then parts_k = parts_{k-1} + parts_{k-1} / 8
  int32_t parts = 64;
  for (int k = 0; k < kNumCandidates; ++k) {
    if (k >= 64) parts += parts / 8;
    const int32_t want = k < 64 ? k + 1 : parts;
    if (plan_candidate_parts(k) != want) { bad++; printf("parts k=%d\n", k); }
  }
  printf("checked %ld bad %ld\n", checked, bad);
  return bad != 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host C++ compiler")
def test_magic_division_and_candidate_parts(tmp_path):
    src = tmp_path / "udiv_check.cpp"
    exe = tmp_path / "udiv_check"
    src.write_text(PROGRAM)
    subprocess.run(["g++", "-O2", "-std=c++17", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    print(res.stdout)
    assert res.returncode == 0, res.stdout
