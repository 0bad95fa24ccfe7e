/* Exhaustive check that the quantizer's division shortcut equals IEEE fp32
 * division for every pair of a finite fp16 activation x and a positive finite
 * fp16 scale s.
 *
 * The shortcut (per row, once) r = RN(1/s), rh = r / 2, s2 = 2 s; (per
 * element) h0 = fma(x, rh, +0), e = fma(-h0, s2, x), h = fma(e, rh, h0).
 * Claim: h == RN(x / s) / 2 exactly (as values: +0 and -0 compare equal).
 * This is the quotient correction of Markstein's division with a correctly
 * rounded reciprocal, applied to the half quotient (scaling by 2 commutes
 * with rounding: no value here is subnormal or overflows in fp32).
 *
 * Prints "pairs <n> mismatches <m>" and, for a mismatch, the first pair.
 * Built with -DSKIP_CORRECTION it checks the uncorrected product instead,
 * which must fail. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float half_to_float(uint16_t h) {
  const int sign = h >> 15, exp = (h >> 10) & 31, man = h & 1023;
  float v = exp == 0 ? ldexpf((float)man, -24) : ldexpf((float)(man | 1024), exp - 25);
  return sign ? -v : v;
}

int main(void) {
  long long mismatches = 0, pairs = 0;
  unsigned first_x = 0, first_s = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(+ : mismatches, pairs)
  for (int sb = 1; sb < 0x7C00; ++sb) {
    const float s = half_to_float((uint16_t)sb);
    const float r = 1.0f / s;
    const float rh = r * 0.5f, s2 = s * 2.0f;
    long long bad = 0;
    unsigned bad_x = 0;
    for (int xb = 0; xb < 0x10000; ++xb) {
      if ((xb & 0x7C00) == 0x7C00) continue;  /* infinities and NaNs */
      const float x = half_to_float((uint16_t)xb);
      const float h0 = fmaf(x, rh, 0.0f);
      const float e = fmaf(-h0, s2, x);
#ifdef SKIP_CORRECTION /* a planted mistake: the plain product x (1/s) / 2 */
      const float h = h0 + 0.0f * e;
#else
      const float h = fmaf(e, rh, h0);
#endif
      const float want = (x / s) * 0.5f;
      ++pairs;
      if (h != want && bad++ == 0) bad_x = (unsigned)xb;
    }
    mismatches += bad;
    if (bad) {
#pragma omp critical
      if (first_s == 0 || (unsigned)sb < first_s) { first_x = bad_x; first_s = (unsigned)sb; }
    }
  }
  printf("pairs %lld mismatches %lld\n", pairs, mismatches);
  if (mismatches) printf("first x=0x%04x s=0x%04x\n", first_x, first_s);
  return mismatches != 0;
}
