// cf_run.h -- the step ends of a decode run without one addition per step.
//
// A decode run repeats one iteration of fixed duration d: the end of step j
// is e_j = fl(e_{j-1} + d), one IEEE binary64 addition per step, which is
// what the step-by-step rules compute.  run_walk gives the same values
// without performing every addition.
//
// Inside one binade [2^E, 2^(E+1)) of normal numbers every sum that stays in
// the binade is rounded to the grid of spacing u = 2^(E-52).  Write q = d/u.
//   - If q is not an odd multiple of 1/2, a step from significand m gives
//     m + round(q), whatever m is.
//   - If it is (a rounding tie), the sum goes to the even neighbour, so a
//     step from any grid point lands on an even significand, and from an
//     even significand the increment is whichever of floor(q), floor(q) + 1
//     is even.
// So once a step has been taken from a point of the binade's grid (or from
// a point with an even significand), the increment D (in units of u) is the
// same for every later step of the binade, and a step from m lands on
// m + D as long as m + D is still inside the binade (the exact sum is then
// below 2^(E+1), so the grid does not change).  The first step into a
// binade starts from the finer grid below it, so it may leave an odd
// significand with a tie: one more step inside the binade settles that.
// The steps of a segment inside a binade are therefore computed in integer
// units of u: at most three single additions per binade (entering it,
// settling the parity, measuring D), then one jump.  Non-normal values are
// taken one addition at a time.
// The functions are constexpr (usable from device code and from host-side
// tests) and use only IEEE binary64 addition, division and conversions.
#pragma once
#include <stdint.h>

namespace cf {

// floor(a / b) for 0 <= a < 2^53 and 1 <= b < 2^53.  The correctly rounded
// quotient is at most one above the true floor.
constexpr uint64_t floor_div53(uint64_t a, uint64_t b) {
  uint64_t q = (uint64_t)((double)a / (double)b);
  if (q * b > a) q--;
  return q;
}

// From e >= 0, the end of a step of a run whose steps last d >= 0, takes at
// most n further steps and stops after the first step whose end is >= stop.
// Returns the end reached and stores the steps taken in *taken.  Same
// result as
//     k = 0; while (e < stop && k < n) { e = e + d; k++; }
constexpr double run_walk(double e, double d, uint32_t n, double stop, uint32_t *taken) {
  constexpr uint64_t kMant = (1ull << 52) - 1;
  uint32_t k = 0;
  while (k < n && e < stop) {
    e = e + d;
    k++;
    if (k >= n || !(e < stop)) break;
    uint64_t b1 = __builtin_bit_cast(uint64_t, e);
    const uint64_t ex = b1 >> 52;  // e >= 0: the sign bit is clear
    if (ex == 0 || ex >= 0x7FF) continue;
    if (b1 & 1u) {
      // an odd significand may have come from the finer grid below: one
      // step from this grid point fixes the increment
      e = e + d;
      k++;
      if (k >= n || !(e < stop)) break;
      b1 = __builtin_bit_cast(uint64_t, e);
      if ((b1 >> 52) != ex) continue;
    }
    e = e + d;
    k++;
    if (k >= n || !(e < stop)) break;
    const uint64_t b2 = __builtin_bit_cast(uint64_t, e);
    if ((b2 >> 52) != ex) continue;
    const uint64_t m2 = b2 & kMant, D = m2 - (b1 & kMant);
    uint64_t j = n - k;
    if (D > 0) {
      // the steps that stay in the binade (no division when all of them do)
      uint64_t span = 0;
      if (__builtin_mul_overflow(j, D, &span) || span > kMant - m2) j = floor_div53(kMant - m2, D);
      const uint64_t bs = __builtin_bit_cast(uint64_t, stop);
      if ((bs >> 52) == ex) {
        // stop lies in this binade above e: the ends m2 + i D reach it from
        // i = ceil((ms - m2) / D)
        const uint64_t is = floor_div53((bs & kMant) - m2 - 1, D) + 1;
        j = is < j ? is : j;
      }
    }
    e = __builtin_bit_cast(double, (b2 & ~kMant) | (m2 + j * D));
    k += (uint32_t)j;
  }
  *taken = k;
  return e;
}

}  // namespace cf
