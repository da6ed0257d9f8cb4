/*
 * OCP e4m3fn encoder in plain C, for exhaustive sweeps (oracle; test
 * infrastructure only -- nothing in the product path links this file).
 *
 * Same definition as oracle/e4m3.py (the FP8 format read for the paper's
 * Sec. 3.4, Eq. 7): keep the sign, saturate |v| >= 448 to 0x7E, otherwise
 * round |v| to the nearest point of the e4m3 grid with ties to the even code.
 * The grid step in the binade [2^e, 2^(e+1)) is 2^(e-3); below 2^-6 the step
 * stays 2^-9 (subnormals). The quotient |v| / step is exact in double and
 * nearbyint() rounds it half-to-even in the default rounding mode.
 *
 * Built by the repository's build step with gcc (no -ffast-math).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static uint8_t code_of_grid_value(double q) {
  /* q is a non-negative point of the e4m3 grid, q <= 448 */
  if (q < 0.015625) /* 2^-6: subnormal codes 0x00..0x07 count units of 2^-9 */
    return (uint8_t)(q * 512.0);
  int ex;
  double f = frexp(q, &ex); /* q = f * 2^ex, f in [0.5, 1) */
  int e = ex - 1;           /* q = (1 + m/8) * 2^e */
  int m = (int)((f * 2.0 - 1.0) * 8.0);
  return (uint8_t)(((e + 7) << 3) | m);
}

uint8_t oracle_e4m3_encode_one(float v) {
  double x = (double)v;
  uint8_t sign = signbit(x) ? 0x80 : 0x00;
  double a = fabs(x);
  if (a >= 448.0) return sign | 0x7E;
  int ex;
  frexp(a, &ex);
  int e = ex - 1;
  if (e < -6) e = -6;
  double step = ldexp(1.0, e - 3);
  double n = nearbyint(a / step);
  return sign | code_of_grid_value(n * step);
}

void oracle_e4m3_encode_f32(const float* v, uint8_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_e4m3_encode_one(v[i]);
}

/*
 * codes[i] is a device encoding of the fp32 value with bit pattern first + i.
 * Returns the number of finite inputs whose code differs from the oracle's;
 * *first_bad receives the bit pattern of the first such input (unchanged if
 * none). Non-finite inputs are outside the quantizer's contract and skipped.
 */
int64_t oracle_e4m3_sweep_check(const uint8_t* codes, uint32_t first, int64_t n, uint32_t* first_bad) {
  int64_t bad = 0;
  for (int64_t i = 0; i < n; ++i) {
    uint32_t bits = first + (uint32_t)i;
    if ((bits & 0x7F800000u) == 0x7F800000u) continue;
    float v;
    memcpy(&v, &bits, sizeof v);
    if (codes[i] != oracle_e4m3_encode_one(v)) {
      if (bad == 0 && first_bad) *first_bad = bits;
      ++bad;
    }
  }
  return bad;
}
