"""Host-side check of the closed-form decode-run walk (csrc/cf_run.h).

run_walk must return exactly what one IEEE binary64 addition per step
returns.  The header is compiled with g++ (-O2 -ffp-contract=off) into a
small driver that compares it with the plain loop on seeded random cases:
realistic times and durations, durations that make every step a rounding tie (from even and from odd
significands, and entering a binade from the finer grid below it),
runs that cross binades, durations below half an ulp, and stop times inside
and outside the run.
"""
import os
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "paper_2512_14098_amd", "csrc", "cf_run.h")

DRIVER = r"""
#include <cmath>
#include <cstdio>
#include <cstring>
#include "cf_run.h"

static uint64_t sm = 0x9E3779B97F4A7C15ull;
static uint64_t next64() {  // splitmix64
  uint64_t z = (sm += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static double unif() { return (double)(next64() >> 11) * 0x1p-53; }

static long bad = 0, cases = 0, ties = 0, crossings = 0, stopped = 0;

static void check(double e, double d, uint32_t n, double stop) {
  double r = e;
  uint32_t k = 0;
  bool tie = false, cross = false;
  while (r < stop && k < n) {
    const double nr = r + d;
    if (std::ilogb(nr) != std::ilogb(r)) cross = true;
    // a tie: the exact sum lies halfway between two neighbours
    const long double ex = (long double)r + (long double)d;
    if ((long double)nr != ex && std::fabs((long double)nr - ex) * 2 == (long double)(std::nextafter(nr, INFINITY) - nr)) tie = true;
    r = nr;
    k++;
  }
  uint32_t k2 = 12345;
  const double r2 = cf::run_walk(e, d, n, stop, &k2);
  cases++;
  ties += tie;
  crossings += cross;
  stopped += (k < n);
  if (k2 != k || std::memcmp(&r, &r2, 8) != 0) {
    if (bad < 10) std::printf("MISMATCH e=%a d=%a n=%u stop=%a: loop %a %u, walk %a %u\n", e, d, n, stop, r, k, r2, k2);
    bad++;
  }
}

int main() {
  // floor_div53 against integer division
  for (int i = 0; i < 2000000; i++) {
    const uint64_t a = next64() >> (11 + (next64() % 53)), b = (next64() >> (11 + (next64() % 53))) | 1u;
    if (cf::floor_div53(a, b) != a / b) { if (bad < 10) std::printf("DIV %llu %llu\n", (unsigned long long)a, (unsigned long long)b); bad++; }
  }
  for (int i = 0; i < 300000; i++) {
    const int kind = i % 8;
    double e = 0, d = 0, stop = INFINITY;
    uint32_t n = (uint32_t)(next64() % 400);
    if (kind == 0) {  // decode runs of the workloads: times up to 1e4 s, steps of ms
      e = unif() * std::pow(10.0, (double)(next64() % 9) - 4);
      d = 0.004 + unif() * 0.05;
    } else if (kind == 1) {  // every step a rounding tie: d = (f + 1/2) ulp(e) with few bits
      e = std::ldexp(1.0 + std::ldexp((double)(next64() % 64), -6), (int)(next64() % 40) - 20);
      const double u = std::nextafter(e, INFINITY) - e;
      d = ((double)(next64() % 8) + 0.5) * u * (double)(1u << (next64() % 3));
      n = (uint32_t)(next64() % 3000);
    } else if (kind == 2) {  // runs that cross binades
      e = std::ldexp(1.0, (int)(next64() % 30) - 10) * (1.0 - unif() * 0.01);
      d = e * unif() * 0.02;
    } else if (kind == 3) {  // steps below half an ulp, and tiny starts
      e = unif() * 1e3;
      d = (next64() & 1) ? e * 0x1p-60 : std::nextafter(0.0, 1.0) * (double)(next64() % 5);
    } else if (kind == 4) {  // long runs
      e = unif() * 100;
      d = 1e-3 + unif() * 1e-2;
      n = (uint32_t)(next64() % 20000);
    } else if (kind == 5) {  // arbitrary significands
      e = std::ldexp(unif(), (int)(next64() % 60) - 30);
      d = std::ldexp(unif(), (int)(next64() % 60) - 40);
    } else if (kind == 6) {  // ties from an odd significand inside a binade
      const int E = (int)(next64() % 40) - 20;
      e = std::ldexp(1.0 + std::ldexp((double)((next64() >> 12) | 1u), -52), E);
      const double u = std::ldexp(1.0, E - 52);
      d = ((double)(next64() % 1000) + 0.5) * u * (double)(1u << (next64() % 4));
      n = (uint32_t)(next64() % 3000);
    } else {  // ties relative to the binade above, from just below it (odd landing)
      const int E = (int)(next64() % 40) - 20;
      e = std::ldexp(1.0 - std::ldexp((double)((next64() % 4000) + 1), -52), E);
      const double u = std::ldexp(1.0, E - 52);
      d = ((double)(next64() % 1000) + 0.5) * u;
      n = (uint32_t)(next64() % 3000);
    }
    const int sk = (int)(next64() % 4);
    if (sk == 1) stop = e + d * (double)n * unif() * 1.2;
    else if (sk == 2) stop = e + d * (double)(next64() % 8);
    else if (sk == 3) stop = e;
    check(e, d, n, stop);
  }
  std::printf("cases %ld ties %ld crossings %ld stopped %ld bad %ld\n", cases, ties, crossings, stopped, bad);
  return bad != 0;
}
"""


def test_run_walk_matches_one_addition_per_step():
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "walk.cpp"), os.path.join(d, "walk")
        with open(src, "w") as f:
            f.write(DRIVER)
        subprocess.check_call(["g++", "-O2", "-std=c++20", "-ffp-contract=off", "-I",
                               os.path.dirname(HDR), src, "-o", exe])
        p = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    print(p.stdout)
    assert p.returncode == 0, p.stdout
    last = p.stdout.strip().splitlines()[-1].split()
    stats = dict(zip(last[0::2], map(int, last[1::2])))
    assert stats["bad"] == 0
    # the generator reached the cases the closed form treats specially
    assert stats["ties"] > 10000 and stats["crossings"] > 10000 and stats["stopped"] > 10000


if __name__ == "__main__":
    pytest.main([__file__, "-q", "-s"])
