/* Exhaustive check of the quantiser's step size: for the divisors L = 3, 15
 * and 255 (2^b - 1 at b = 2, 4, 8) and every finite binary32 value x >= 0,
 *     q0 = x * r,  r = RN(1/L);   q = fma(fma(-q0, L, x), r, q0)
 * equals the correctly rounded quotient x / L.  Prints one line per divisor
 * with the number of mismatches.  Build without contraction. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

int main(void) {
  const float Ls[] = {3.0f, 15.0f, 255.0f};
  for (int li = 0; li < 3; ++li) {
    const float L = Ls[li], r = 1.0f / L;
    unsigned long long bad = 0;
    for (uint32_t hi = 0; hi < 0x7f80u; ++hi) {
      for (uint32_t lo = 0; lo < 0x10000u; ++lo) {
        const uint32_t u = (hi << 16) | lo;
        float x;
        memcpy(&x, &u, 4);
        const float ref = x / L;
        const float q0 = x * r;
        const float q = fmaf(fmaf(-q0, L, x), r, q0);
        uint32_t a, c;
        memcpy(&a, &ref, 4);
        memcpy(&c, &q, 4);
        bad += a != c;
      }
    }
    printf("%g %llu\n", L, bad);
  }
  return 0;
}
