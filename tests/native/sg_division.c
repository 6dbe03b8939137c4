/* Host check of the tensor-scale division used by the encoders: for binary32
 * a >= 2^-100, q = a * y with y the binary32 nearest to 1/2688, then
 * q + (a - 2688 q) y with both steps as fused multiply-adds, equals the correctly
 * rounded a / 2688.  Usage: sg_division STRIDE; checks every STRIDE-th bit pattern
 * from 2^-100 to the largest finite value and every pattern of four whole binades;
 * prints the number of mismatches. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float f_of(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t u_of(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

static int check(uint32_t u, float b, float y) {
  const float a = f_of(u);
  const float q = a * y;
  const float q2 = fmaf(fmaf(-q, b, a), y, q);
  return u_of(q2) != u_of(a / b);
}

int main(int argc, char** argv) {
  const uint32_t stride = argc > 1 ? (uint32_t)strtoul(argv[1], NULL, 10) : 1u;
  volatile float bv = 2688.0f;
  const float b = bv, y = 1.0f / b;
  if (u_of(y) != 0x39c30c31u) { printf("reciprocal %08x\n", u_of(y)); return 2; }
  unsigned long long bad = 0, n = 0;
  for (uint32_t u = 0x0D800000u; u < 0x7F800000u; u += stride, ++n) bad += check(u, b, y);
  const uint32_t binades[4] = {0x0D800000u, 0x2F000000u, 0x3F800000u, 0x7F000000u};
  for (int k = 0; k < 4; ++k)
    for (uint32_t u = binades[k]; u < binades[k] + 0x800000u; ++u, ++n) bad += check(u, b, y);
  printf("%llu %llu\n", bad, n);
  return 0;
}
