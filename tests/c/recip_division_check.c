/* Exhaustive check of the division the fused on-the-fly mode uses in its on-chip quantization.
 *
 * The quantization rule divides x by the block scale d = RN(absmax / 127) in FP32.  On chip the
 * quotient is formed as q0 = RN(x * r), q = RN(q0 + RN(x - q0 * d) * r) with r = RN(1 / d)
 * (two fused multiply-adds).  For every positive finite FP16 absmax and every FP16 x with
 * |x| <= absmax (both signs and zero) this program compares q with RN(x / d) bit for bit and
 * also checks |RN(x / d)| < 127.5, so that rounding never needs the clamp to [-127, 127].
 * Prints the counts; exits 1 on any mismatch.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float fp16_value(uint16_t h) {
  const uint32_t e = (h >> 10) & 31u, m = h & 1023u;
  const float v = e == 0 ? ldexpf((float)m, -24) : ldexpf((float)(m | 1024u), (int)e - 25);
  return (h >> 15) ? -v : v;
}

int main(void) {
  static float pos[0x7C00];
  int n = 0;
  for (uint32_t h = 1; h < 0x7C00u; ++h) pos[n++] = fp16_value((uint16_t)h);   /* ascending */
  long long pairs = 0, mismatches = 0, out_of_range = 0;
  for (int ia = 0; ia < n; ++ia) {
    const volatile float d = pos[ia] / 127.0f;
    const volatile float r = 1.0f / d;
    for (int ix = -1; ix <= ia; ++ix) {
      for (int sign = 0; sign < 2; ++sign) {
        const float x = ix < 0 ? 0.0f : (sign ? -pos[ix] : pos[ix]);
        const float q0 = fmaf(x, r, 0.0f);
        const float q = fmaf(fmaf(-q0, d, x), r, q0);
        const float want = x / d;
        ++pairs;
        if (memcmp(&q, &want, sizeof q) != 0) ++mismatches;
        if (!(fabsf(want) < 127.5f)) ++out_of_range;
      }
    }
  }
  printf("pairs %lld mismatches %lld out_of_range %lld\n", pairs, mismatches, out_of_range);
  return (mismatches || out_of_range) ? 1 : 0;
}
