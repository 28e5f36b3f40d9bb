"""Host-side checks of two pure helpers of the kernels (compiled from the
kernels' own header with hipcc for the host; no GPU needed):

* fastmod: the multiply-only remainder must equal n mod d for every 32-bit n
  and d >= 1 (exhaustive over small d, random over the full range);
* cdf_search: the 8-way search of a CDF row must return the smallest s in
  1..cap-1 with w2 < T[s], else cap (the definition of an output-length draw),
  on random nondecreasing rows with ties, saturation and boundary values of
  w2, for every row length up to 70 and sampled lengths up to 4100; and so
  must the search narrowed by the row's 64-bucket guide (cdf_guide_entry,
  cdf_search_in), as the Nested WAIT kernel draws.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2504_11320_amd", "csrc")
INC = os.path.join(ROOT, "include")

PROG = r'''
#include "sim_common.h"
#include <cstdio>
#include <random>
#include <vector>
using namespace wsim;
static int32_t linear(const uint32_t *row, int32_t cap, uint32_t w2) {
  for (int32_t s = 1; s < cap; ++s) if (w2 < row[s - 1]) return s;
  return cap;
}
int main() {
  std::mt19937_64 g(2026);
  long bad = 0, n_ = 0;
  for (uint32_t d = 1; d <= 3000; ++d) {
    const uint64_t M = fastmod_magic(d);
    const uint32_t edge[4] = {0u, 0xffffffffu, d - 1u, d};
    for (int q = 0; q < 600; ++q) {
      const uint32_t n = q < 4 ? edge[q] : (q % 2 ? (uint32_t)g() : (uint32_t)(g() % 200000));
      ++n_; bad += fastmod(n, M, d) != n % d;
    }
  }
  for (int q = 0; q < 2000000; ++q) {
    uint32_t d = (uint32_t)g() >> (g() % 32);
    if (d == 0) d = 1;
    const uint32_t n = (uint32_t)g();
    ++n_; bad += fastmod(n, fastmod_magic(d), d) != n % d;
  }
  std::printf("fastmod %ld checked, %ld wrong\n", n_, bad);
  long bad2 = 0, n2 = 0;
  for (int cap = 1; cap <= 4100; cap += (cap < 70 ? 1 : 97)) {
    for (int rep = 0; rep < 12; ++rep) {
      std::vector<uint32_t> row(cap > 1 ? cap - 1 : 1, 0u);
      uint64_t v = (rep % 3 == 0) ? 0 : g() % 1000;
      for (int s = 0; s < cap - 1; ++s) {
        if (g() % 4) v += g() % (1ull << (3 * rep % 33));
        if (v > 0xffffffffull) v = 0xffffffffull;
        row[s] = (uint32_t)v;
      }
      for (int q = 0; q < 200; ++q) {
        uint32_t w2;
        switch (q % 5) {
          case 0: w2 = (uint32_t)g(); break;
          case 1: w2 = cap > 1 ? row[g() % (cap - 1)] : 7u; break;
          case 2: w2 = cap > 1 ? row[g() % (cap - 1)] - 1u : 0u; break;
          case 3: w2 = (q & 1) ? 0u : 0xffffffffu; break;
          default: w2 = (uint32_t)(g() % 2000);
        }
        const int32_t want = linear(row.data(), cap, w2);
        ++n2; bad2 += cdf_search(row.data(), cap, w2) != want;
        const int b = (int)(w2 >> 26);
        const int32_t glo = cdf_guide_entry(row.data(), cap, b);
        const int32_t ghi = cdf_guide_entry(row.data(), cap, b + 1);
        ++n2; bad2 += cdf_search_in(row.data(), glo, ghi, w2) != want;
      }
    }
  }
  std::printf("cdf_search %ld checked, %ld wrong\n", n2, bad2);
  return (bad || bad2) ? 1 : 0;
}
'''


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


def test_fastmod_and_cdf_search(tmp_path):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not available")
    src = tmp_path / "helpers.hip"
    src.write_text(PROG)
    exe = tmp_path / "helpers"
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O2", "-std=c++17", "-I", CSRC, "-I", INC,
                    "-o", str(exe), str(src)], check=True, capture_output=True, timeout=300)
    p = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    print(p.stdout)
    assert p.returncode == 0, p.stdout + p.stderr
    assert "0 wrong" in p.stdout.splitlines()[0] and "0 wrong" in p.stdout.splitlines()[1]
