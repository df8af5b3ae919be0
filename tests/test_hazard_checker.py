"""The plan generator's hazard proof has teeth.

plan.cpp refuses a schedule in which one work item of a launch writes a
location (buffer, rank, block) that another item reads or writes.  Here a
C++ program (host code only, g++) builds real schedules, checks that every
one of them passes, and then plants the mistakes a buffer assignment could
make -- an in-place doubling step, a reduce that reads and writes one
scratch buffer, two ranges writing the same placement, a copy reading
what another item writes -- and checks that each is refused.
"""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2004_09362_amd", "csrc")

PROG = r"""
#include <cstdio>
#include <string>
#include "ar_internal.hpp"
using namespace ar;

static int fails = 0;
static void expect(bool ok, const char* what) {
  if (!ok) { std::printf("FAIL: %s\n", what); ++fails; }
}
static Schedule make(int32_t P, int32_t k, int32_t group, int32_t sched) {
  Schedule s;
  const std::string e = build_schedule_ex(P, 1000, k, group, sched, &s);
  if (!e.empty()) { std::printf("build failed P=%d k=%d: %s\n", P, k, e.c_str()); ++fails; }
  return s;
}

int main() {
  // every real schedule passes
  int built = 0;
  for (int32_t P = 1; P <= 128; ++P) {
    int32_t L = 0;
    while ((1 << L) < P) ++L;
    for (int32_t k = L; k <= 2 * L; ++k) {
      Schedule s = make(P, k, kGroupCyclic, kSchedButterfly);
      expect(check_hazards(s).empty(), "cyclic schedule refused");
      ++built;
      if ((P & (P - 1)) == 0) {
        Schedule x = make(P, k, kGroupXor, kSchedButterfly);
        expect(check_hazards(x).empty(), "xor schedule refused");
        ++built;
      }
    }
    Schedule r = make(P, 2 * (P - 1), kGroupCyclic, kSchedRing);
    expect(check_hazards(r).empty(), "ring schedule refused");
    ++built;
  }

  // planted mistakes
  {  // XOR doubling step made in place: peers read what is rewritten
    Schedule s = make(8, 4, kGroupXor, kSchedButterfly);  // r = 2: two doubling steps via scratch
    bool planted = false;
    for (Launch& l : s.launches)
      for (Range& rg : l.ranges)
        if (!planted && rg.kind == kReduce && rg.dst != kBufU && rg.own == rg.src) {
          rg.dst = rg.src;
          planted = true;
        }
    expect(planted, "no doubling step to plant into");
    expect(!check_hazards(s).empty(), "in-place doubling step accepted");
  }
  {  // cyclic shifted step writing its primed sums into the buffer it reads
     // from peers (P = 7, k = 4: placements 1..3 read X at p + 2 and would
     // overwrite X at p)
    Schedule s = make(7, 4, kGroupCyclic, kSchedButterfly);
    bool planted = false;
    for (Launch& l : s.launches)
      for (Range& rg : l.ranges)
        if (!planted && rg.kind == kReduce2 && rg.dst != rg.src) {
          rg.dst = rg.src;
          planted = true;
        }
    expect(planted, "no dual reduce to plant into");
    expect(!check_hazards(s).empty(), "reduce reading and writing one scratch buffer accepted");
  }
  {  // two ranges writing the same placement
    Schedule s = make(24, 10, kGroupCyclic, kSchedButterfly);
    Launch& l = s.launches[0];
    Range dup = l.ranges[0];
    dup.count = 1;
    l.ranges.push_back(dup);
    expect(!check_hazards(s).empty(), "duplicate writer accepted");
  }
  {  // Ring reduction step widened to two placements: rank x + 1 reads
     // placement 1 of rank x, which that rank now rewrites in the same step
    Schedule s = make(5, 8, kGroupCyclic, kSchedRing);
    s.launches[1].ranges[0].p0 = 1;
    s.launches[1].ranges[0].count = 2;
    expect(!check_hazards(s).empty(), "ring step writing the read placement accepted");
  }
  {  // distribution copy widened onto placements that are read in the same launch
    Schedule s = make(7, 6, kGroupCyclic, kSchedButterfly);
    Launch& l = s.launches.back();
    l.ranges[0].p0 = 0;
    l.ranges[0].count = 7;
    expect(!check_hazards(s).empty(), "copy over its own sources accepted");
  }
  std::printf("%d schedules, %d failures\n", built, fails);
  return fails != 0;
}
"""


def test_hazard_checker_accepts_real_schedules_and_refuses_planted_hazards(tmp_path):
    src = tmp_path / "hz.cpp"
    src.write_text(PROG)
    exe = tmp_path / "hz"
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", CSRC, "-o", str(exe), str(src),
                    os.path.join(CSRC, "plan.cpp")], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "0 failures" in res.stdout
