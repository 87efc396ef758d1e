/* Exhaustive host check of the reciprocal-and-correction quotient that the
 * row quantizer uses in place of a divide.  With s = amax / 448 (fp32,
 * correctly rounded) and r = 1 / s (likewise), the kernel forms
 *   y = x r,  q = copysign(fma(fma(-y, s, x), r, y), y)
 * for every element x of a group whose bf16 amax is finite and >= 2^-64.
 * This program walks every such amax and every bf16 x with |x| <= amax, both
 * signs, and counts the cases where q differs from the correctly rounded
 * x / s: bit for bit where either quotient is >= 2^-12 in magnitude (where
 * an E4M3 code can be nonzero under either rounding), by sign elsewhere
 * (both encode to a signed zero).  Exit status 0 iff there are none.
 * Build: gcc -O2 -fopenmp -ffp-contract=off (IEEE fp32, no contraction). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float bf16(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static uint32_t bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}

int main(void) {
  long long pairs = 0, bad = 0, groups = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(+ : pairs, bad, groups)
  for (int ab = 1; ab < 0x7F80; ++ab) {
    const float amax = bf16((uint16_t)ab);
    if (!(amax >= 0x1p-64f)) continue;
    groups++;
    const float s = amax / 448.0f, r = 1.0f / s;
    for (int xb = 0; xb < 0x7F80; ++xb) {
      const float ax = bf16((uint16_t)xb);
      if (ax > amax) break;
      for (int neg = 0; neg < 2; ++neg) {
        const float x = neg ? -ax : ax;
        const float q = x / s;
        const float y = x * r;
        const float q2 = copysignf(fmaf(fmaf(-y, s, x), r, y), y);
        const int big = fabsf(q) >= 0x1p-12f || fabsf(q2) >= 0x1p-12f;
        pairs++;
        if (big ? bits(q) != bits(q2) : signbit(q) != signbit(q2)) bad++;
      }
    }
  }
  printf("amax values %lld, (amax, x) pairs %lld, mismatches %lld\n", groups, pairs, bad);
  return bad != 0;
}
