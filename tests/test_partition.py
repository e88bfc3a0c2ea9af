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


GROUPS_PROGRAM = r"""
#include "ws_kernels.hpp"
#include <cstdio>

int main() {
  // the shapes the benchmark times: 40 heads x 4 query tiles over 139 pages
  // (8-unit history), 19 pages (single unit) and 479 pages (32 units); 12
  // heads x 1 tile over 13 pages (v0.1)
  struct { long long h, qt, p, want; } pinned[] = {{40, 4, 139, 64}, {40, 4, 19, 40}, {40, 4, 479, 64},
                                                   {12, 1, 13, 84}};
  for (auto& c : pinned) {
    const long long g = ws::video_group_count(c.h, c.qt, c.p, 256);
    if (g != c.want) { std::printf("FAIL pinned h=%lld p=%lld got %lld\n", c.h, c.p, g); return 1; }
  }
  long long n = 0;
  for (long long h : {1, 3, 8, 12, 40, 64, 80, 160})
    for (long long qt : {1, 2, 4})
      for (long long p : {0, 1, 2, 5, 13, 19, 64, 139, 479})
        for (long long cus : {4, 20, 85, 256}) {
          const long long g = ws::video_group_count(h, qt, p, cus);
          if (p == 0) {
            if (g != h) { std::printf("FAIL empty\n"); return 1; }
            continue;
          }
          if (g < 1 || g > h * p) { std::printf("FAIL range h=%lld p=%lld g=%lld\n", h, p, g); return 1; }
          // every head meets at most kMaxVideoSplits ranges
          if ((g + h - 1) / h + 1 > ws::kMaxVideoSplits) { std::printf("FAIL ranges h=%lld g=%lld\n", h, g); return 1; }
          // a group count that divides the head count splits no head, and the
          // partition then gives each head to exactly one group
          if (!ws::video_heads_split(h, g)) {
            const ws::VideoPartition part{h, p, 6, g};
            for (long long x = 0; x < h; ++x)
              if (ws::video_group_of(part, x * p) != ws::video_group_of(part, x * p + p - 1)) {
                std::printf("FAIL aligned h=%lld p=%lld g=%lld head=%lld\n", h, p, g, x);
                return 1;
              }
          }
          ++n;
        }
  std::printf("ok %lld\n", n);
  return 0;
}
"""


def test_group_count_model(tmp_path):
    """The host's video group count (ws_kernels.hpp: video_group_count): the
    counts it picks for the benchmark's shapes (one round of 256 workgroups
    at 8 and 32 history units; one head per group, so no merge, for a single
    unit; seven key ranges per head at v0.1), and over a grid of shapes: at
    least one group and at most one per (head, page) unit, at most
    kMaxVideoSplits ranges per head, and whenever no head is split
    (video_heads_split false) each head lies in one group's share."""
    src = tmp_path / "groups.cpp"
    exe = tmp_path / "groups"
    src.write_text(GROUPS_PROGRAM)
    try:
        subprocess.run(["g++", "-std=c++17", "-O1", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                        "-I", CSRC, str(src), "-o", str(exe)], check=True, capture_output=True, text=True)
    except FileNotFoundError:
        pytest.skip("no host C++ compiler")
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok")
