/*
 * quotient_check.c -- checks, on the CPU, that a multiply-and-correct
 * sequence gives the correctly rounded fp32 quotient a / Q for the constants
 * Q = 127 and Q = 448 of the INT8 and FP8 row scales:
 *
 *     q0 = RN(a * R),  R = RN(1 / Q),   q = RN(q0 + RN(a - q0 * Q) * R)   (two fmas)
 *
 * For each tested a it forms e = a - q * Q exactly in long double and accepts
 * q iff the true quotient a / Q = q + e / Q lies within half a gap of q
 * (gap above: ulp(q); gap below: ulp(q) / 2 when q is a normal power of
 * two), ties going to the even significand.  Inputs: every finite a >= 0
 * whose bit pattern is a multiple of STRIDE, plus every pattern in windows
 * around the subnormal/normal boundary and around Q * 2^-126.  STRIDE = 1
 * checks all 2^31 inputs.
 *
 * Output, one line per Q: "Q <checked> <fails_normal> <fails_subnormal>",
 * counting inputs whose quotient is normal or subnormal.  Exit status 0.
 * Build: cc -O2 -mfma -ffp-contract=off quotient_check.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float f_of(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t u_of(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

static int exact(float a, float Q, float q) {
  const uint32_t qu = u_of(q);
  const int qexp = (int)((qu >> 23) & 0xFF);
  const long double ulp = qexp == 0 ? ldexpl(1.0L, -149) : ldexpl(1.0L, qexp - 150);
  const long double below = (qexp > 1 && (qu & 0x7FFFFF) == 0) ? ulp / 2 : ulp;
  const long double e = (long double)a - (long double)q * (long double)Q;
  const long double hi = ulp * Q / 2, lo = -below * Q / 2;
  if (e < hi && e > lo) return 1;
  if (e == hi || e == lo) return (qu & 1) == 0;
  return 0;
}

static void check(float Q, uint32_t u, uint64_t *n, uint64_t *bad_norm, uint64_t *bad_sub) {
  const float R = 1.0f / Q;
  const float a = f_of(u);
  const float q0 = a * R;
  const float q = fmaf(fmaf(-q0, Q, a), R, q0);
  ++*n;
  if (!exact(a, Q, q)) {
    if (((u_of(q) >> 23) & 0xFF) == 0) ++*bad_sub; else ++*bad_norm;
  }
}

int main(int argc, char **argv) {
  const uint32_t stride = argc > 1 ? (uint32_t)strtoul(argv[1], NULL, 10) : 4099u;
  const float qs[2] = {127.0f, 448.0f};
  for (int t = 0; t < 2; ++t) {
    const float Q = qs[t];
    uint64_t n = 0, bad_norm = 0, bad_sub = 0;
    for (uint64_t u = 0; u < 0x7F800000u; u += stride) check(Q, (uint32_t)u, &n, &bad_norm, &bad_sub);
    if (stride > 1) {
      /* dense windows: the subnormal/normal input boundary and Q * 2^-126 */
      const uint32_t centers[2] = {0x00800000u, u_of(Q * 0x1p-126f)};
      for (int c = 0; c < 2; ++c)
        for (uint32_t u = centers[c] - (1u << 20); u < centers[c] + (1u << 20); ++u)
          check(Q, u, &n, &bad_norm, &bad_sub);
    }
    printf("%g %llu %llu %llu\n", Q, (unsigned long long)n, (unsigned long long)bad_norm,
           (unsigned long long)bad_sub);
  }
  return 0;
}
