"""The video kernel's work partition (ws_kernels.hpp: VideoPartition), on the
CPU: the host, the attention kernel and the merge kernel all call the same
header functions, compiled here with the host compiler.

- The 32-bit form of the lookups gives the same integers as the 64-bit form
  wherever video_fits32 holds.
- The shares tile the (head, page) units: group g takes units
  [lo(g), lo(g + 1)), lo(0) = 0, lo(groups) = heads * pages, lo is
  non-decreasing, and group_of(x) is the g whose share holds x.
- A share meets at most ceil(pages_per_group / pages) + 1 heads, and a head
  is split over at most ceil(groups / heads) + 1 ranges (the bound the host
  sizes the split-KV workspace with)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_04443_amd", "csrc")

PROGRAM = r"""
#include "ws_kernels.hpp"
#include <cstdio>
#include <cstdlib>

static int fail(const char* what, long long h, long long pg, long long c, long long g, long long at) {
  std::printf("FAIL %s heads=%lld pages=%lld cost=%lld groups=%lld at=%lld\n", what, h, pg, c, g, at);
  return 1;
}

int main() {
  const long long heads_set[] = {1, 3, 12, 40, 64};
  const long long pages_set[] = {1, 2, 5, 15, 64, 133, 139, 499};
  const long long cost_set[] = {0, 1, 6};
  long long checked = 0;
  for (long long heads : heads_set)
    for (long long pages : pages_set)
      for (long long cost : cost_set)
        for (long long groups = 1; groups <= 4 * heads + 8 && groups <= 300; ++groups) {
          const ws::VideoPartition p{heads, pages, cost, groups};
          if (!ws::video_fits32(p)) return fail("fits32", heads, pages, cost, groups, -1);
          const long long units = heads * pages;
          long long prev = -1;
          for (long long g = 0; g <= groups; ++g) {
            const long long lo = ws::video_group_lo(p, g);
            if (lo != ws::video_group_lo_wide(p, g)) return fail("lo32", heads, pages, cost, groups, g);
            if (lo < prev) return fail("lo monotone", heads, pages, cost, groups, g);
            if (g == 0 && lo != 0) return fail("lo(0)", heads, pages, cost, groups, g);
            if (g == groups && lo != units) return fail("lo(G)", heads, pages, cost, groups, g);
            prev = lo;
          }
          for (long long x = 0; x < units; ++x) {
            const long long g = ws::video_group_of(p, x);
            if (g != ws::video_group_of_wide(p, x)) return fail("of32", heads, pages, cost, groups, x);
            if (g < 0 || g >= groups) return fail("of range", heads, pages, cost, groups, x);
            if (!(ws::video_group_lo(p, g) <= x && x < ws::video_group_lo(p, g + 1)))
              return fail("of/lo", heads, pages, cost, groups, x);
            ++checked;
          }
          for (long long h = 0; h < heads; ++h) {
            const long long r = ws::video_group_of(p, h * pages + pages - 1) - ws::video_group_of(p, h * pages) + 1;
            if (r > (groups + heads - 1) / heads + 1) return fail("ranges", heads, pages, cost, groups, h);
          }
        }
  // past the 32-bit range the lookups take the 64-bit form
  const ws::VideoPartition big{64, 40000000, 6, 256};
  if (ws::video_fits32(big)) return fail("big fits32", 64, 40000000, 6, 256, -1);
  if (ws::video_group_lo(big, 256) != 64LL * 40000000) return fail("big lo(G)", 64, 40000000, 6, 256, 256);
  std::printf("ok %lld\n", checked);
  return 0;
}
"""


def test_partition_lookups_tile_the_units(tmp_path):
    src = tmp_path / "partition.cpp"
    exe = tmp_path / "partition"
    src.write_text(PROGRAM)
    try:
        subprocess.run(["g++", "-std=c++17", "-O1", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                        "-I", CSRC, str(src), "-o", str(exe)], check=True, capture_output=True, text=True)
    except FileNotFoundError:
        pytest.skip("no host C++ compiler")
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok")
