/* Host check of the lookup's mean division: for a float32 sum a and a bag
 * length L (as float fl), the kernel computes y = RN(1/fl), q = RN(a*y),
 * r = fma(-q, fl, a) and fma(r, y, q) when 2^-64 <= |a| <= FLT_MAX, and
 * claims the result equals the IEEE binary32 quotient RN(a/fl) (Markstein's
 * correction theorem).  This program compares the two on every significand
 * of several binades for a set of divisors, on random dividend/divisor pairs
 * up to 2^31, and on exact quotients; it prints the number of mismatches and
 * exits non-zero when there is one. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static uint64_t state = 88172645463325252ull;
static uint64_t next(void) { state ^= state << 13; state ^= state >> 7; state ^= state << 17; return state; }
static float from_bits(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint32_t to_bits(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

static long checked = 0, mismatches = 0;
static void check(float a, uint32_t L) {
  volatile float fl = (float)L;
  volatile float y = 1.0f / fl;
  volatile float q = a * y;
  volatile float r = fmaf(-q, fl, a);
  volatile float got = fmaf(r, y, q);
  volatile float want = a / fl;
  ++checked;
  if (to_bits(got) != to_bits(want)) {
    if (mismatches < 5) printf("mismatch a=%a L=%u: %a vs %a\n", a, L, got, want);
    ++mismatches;
  }
}

int main(int argc, char** argv) {
  const long random_pairs = argc > 1 ? atol(argv[1]) : 2000000;
  const uint32_t sig_step = argc > 2 ? (uint32_t)atol(argv[2]) : 7;
  const uint32_t divisors[] = {3, 7, 10, 11, 27, 255, 1000, 65535, 16777215, 16777217, 2147483647u, 1431655765u};
  const uint32_t exps[] = {63, 64, 127, 200, 254};   /* biased exponents: 2^-64, 2^-63, 1, 2^73, 2^127 */
  for (unsigned i = 0; i < sizeof divisors / sizeof divisors[0]; ++i)
    for (unsigned j = 0; j < sizeof exps / sizeof exps[0]; ++j)
      for (uint32_t m = 0; m < (1u << 23); m += sig_step) check(from_bits(exps[j] << 23 | m), divisors[i]);
  for (long i = 0; i < random_pairs; ++i) {
    uint32_t L = (i & 1) ? 1 + (uint32_t)(next() % 300) : 1 + (uint32_t)(next() % 2147483647u);
    uint32_t e = 63 + (uint32_t)(next() % 192), m = (uint32_t)next() & 0x7fffff, s = (uint32_t)next() & 1;
    if (i % 7 == 0) m = 0x7fffff - ((uint32_t)next() & 15);   /* significands near all ones */
    if (i % 11 == 0) m = (uint32_t)next() & 15;               /* near powers of two */
    check(from_bits(s << 31 | e << 23 | m), L);
  }
  for (uint32_t L = 1; L < 2000; ++L)
    for (uint32_t k = 1; k < 400; k += 13) check((float)L * (float)k * 0x1p-20f, L);
  printf("checked %ld, mismatches %ld\n", checked, mismatches);
  return mismatches != 0;
}
