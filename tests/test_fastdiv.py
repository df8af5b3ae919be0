"""The precomputed 32-bit divisions used by the kernels' work decomposition
(host references of the same arithmetic: the step and column kernels' form,
and the broadcast's branch-free form) against exact division, including
edge divisors and numerators."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PROG = r"""
#include <cstdio>
#include <cstdint>
#include <random>
#include "ar_internal.hpp"
int main() {
  std::mt19937_64 g(12345);
  uint64_t bad = 0, checks = 0;
  const uint32_t edge_n[] = {0u, 1u, 2u, 3u, 255u, 256u, 65535u, 65536u, 0x7fffffffu, 0x80000000u, 0xfffffffeu, 0xffffffffu};
  auto check = [&](uint32_t n, uint32_t d) {
    ar::FastDiv f = ar::make_fastdiv(d);
    ar::StreamDiv s = ar::stream_div(d);
    ++checks;
    if (ar::fastdiv_host(n, f) != n / d) { if (bad < 5) printf("n=%u d=%u\n", n, d); ++bad; }
    if (ar::stream_div_host(n, s) != n / d || s.d != d) { if (bad < 5) printf("stream n=%u d=%u\n", n, d); ++bad; }
  };
  for (uint32_t d = 1; d <= 5000; ++d) {
    for (uint32_t n : edge_n) check(n, d);
    for (int i = 0; i < 200; ++i) check(uint32_t(g()), d);
    for (uint32_t k = 1; k < 40; ++k) { check(k * d - 1, d); check(k * d, d); check(k * d + 1, d); }
  }
  for (int i = 0; i < 2000000; ++i) {
    uint32_t d = uint32_t(g() >> (32 + (g() % 32)));
    if (d == 0) d = 1;
    check(uint32_t(g()), d);
  }
  for (uint32_t n : edge_n) for (uint32_t d : edge_n) if (d) check(n, d);
  printf("%llu %llu\n", (unsigned long long)checks, (unsigned long long)bad);
  return bad != 0;
}
"""


def test_fastdiv_matches_exact_division(tmp_path):
    src = tmp_path / "fd.cpp"
    src.write_text(PROG)
    exe = tmp_path / "fd"
    subprocess.run(["g++", "-O2", "-std=c++17", "-I", os.path.join(ROOT, "paper_2004_09362_amd", "csrc"),
                    "-o", str(exe), str(src)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout
    checks, bad = map(int, res.stdout.split()[-2:])
    assert bad == 0 and checks > 3000000
