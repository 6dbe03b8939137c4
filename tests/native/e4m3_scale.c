/* Host checks of the E4M3 scale arithmetic of the encoders.
 *
 * 1. Rounding from the bits: for v >= 2^-6 the E4M3 value nearest to v (ties to the
 *    even code) is v's binary32 pattern rounded at bit 20 (ties to even) with the 20
 *    bits below cleared; below 2^-6 it is rint(v * 512) / 512.  Checked for every
 *    binary32 v in [0, 448] against the nearest point of the 127-value grid, found by
 *    search.
 * 2. The quotient shortcut: v = min(bmax * r, 448), r within one ulp of 1/den, may
 *    stand in for min(fl32(bmax / den), 448) whenever v >= 2^-6 and the 20 bits below
 *    its 3-bit mantissa are at least 16 away from 0x80000.  Checked on random and on
 *    midpoint-seeking (bmax, den) pairs with r = RN(1/den) and its two neighbours.
 * Prints "<mismatches in 1> <mismatches in 2> <pairs tried in 2>". */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float f_of(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t u_of(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

static float grid[127];   /* E4M3FN values 0 .. 448, code order = value order */

static void make_grid(void) {
  for (int c = 0; c < 127; ++c) {
    const int e = c >> 3, m = c & 7;
    grid[c] = e == 0 ? (float)m / 512.0f : ldexpf(1.0f + m / 8.0f, e - 7);
  }
}

static float round_bits(float v) {
  const uint32_t b = u_of(v);
  const float sn = f_of((b + 0x7FFFFu + ((b >> 20) & 1u)) & 0xFFF00000u);
  const float ss = rintf(v * 512.0f) / 512.0f;
  return v < 0.015625f ? ss : sn;
}

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next32(void) {
  rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
  return (uint32_t)(rng >> 11);
}

int main(void) {
  make_grid();
  unsigned long long bad1 = 0, bad2 = 0, tried = 0;
  /* 1: every binary32 in [0, 448]; the search walks the grid monotonically */
  int lo = 0;
  for (uint32_t u = 0; u <= 0x43E00000u; ++u) {
    const float v = f_of(u);
    while (lo + 1 < 127 && grid[lo + 1] <= v) ++lo;
    float ref;
    if (grid[lo] == v || lo == 126) ref = grid[lo];
    else {
      const double dl = (double)v - grid[lo], dh = (double)grid[lo + 1] - v;
      ref = dl < dh ? grid[lo] : dh < dl ? grid[lo + 1] : ((lo & 1) ? grid[lo + 1] : grid[lo]);
    }
    if (u_of(round_bits(v)) != u_of(ref)) ++bad1;
  }
  /* 2: the shortcut */
  for (int it = 0; it < 4000000; ++it) {
    const float den = f_of(0x28000000u + next32() % 0x2A000000u);   /* ~1e-14 .. ~1e11 */
    float bmax;
    if (it & 1) {
      /* aim at an E4M3 midpoint: bmax ~ mid * den */
      const int c = next32() % 126;
      const float mid = 0.5f * (grid[c] + grid[c + 1]);
      bmax = f_of(u_of(mid * den) + (next32() % 64) - 32);
    } else {
      bmax = den * ldexpf(1.0f + (next32() % 1000) / 1000.0f, (int)(next32() % 20) - 8);
    }
    if (!(bmax > 0) || !isfinite(bmax)) continue;
    const float exact = fminf(bmax / den, 448.0f);
    const float want = round_bits(exact);
    const float r0 = 1.0f / den;
    const float rs[3] = {r0, nextafterf(r0, 0.0f), nextafterf(r0, INFINITY)};
    for (int k = 0; k < 3; ++k) {
      const float v = fminf(bmax * rs[k], 448.0f);
      const uint32_t rem = u_of(v) & 0xFFFFFu;
      if (v >= 0.015625f && rem - 0x7FFF0u >= 32u) {
        ++tried;
        if (u_of(round_bits(v)) != u_of(want)) ++bad2;
      }
    }
  }
  printf("%llu %llu %llu\n", bad1, bad2, tried);
  return 0;
}
