/* Exhaustive check of the bfloat16 packing rule over all 2^32 binary32 bit
 * patterns (test infrastructure, host only).
 *
 * The rule checked is the one the oracle and the kernels both state: round to
 * nearest with ties to even, NaN packed as the quiet NaN 0x7FC0, infinities
 * kept, finite values past the largest bfloat16 rounded to infinity,
 * subnormals kept.  It is written here twice, independently:
 *   - the integer form: (u + 0x7FFF + ((u >> 16) & 1)) >> 16, NaN -> 0x7FC0;
 *   - the definition: of the two bfloat16 values that bracket x (its truncation
 *     toward zero and the next value away from zero, 2^128 standing for the
 *     step past the largest finite one), take the nearer in exact arithmetic,
 *     and on a tie the one with an even last bit.
 * The program counts the patterns where the two disagree and prints
 * "mismatches <count> checked <count>"; exit status 0 only for zero.
 * `bf16_exhaustive sample STRIDE COUNT` instead prints, one per line in hex,
 * the definition's result for the patterns k * STRIDE (mod 2^32), k < COUNT,
 * for comparison with other implementations of the rule.
 * Built with -DPLANT_TRUNCATION the integer form truncates instead of rounding,
 * a planted mistake the exhaustive run must report. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float f_of(uint32_t u) {
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

static uint16_t by_integer_form(uint32_t u) {
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
#ifdef PLANT_TRUNCATION
  return (uint16_t)(u >> 16);
#else
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
#endif
}

static uint16_t by_definition(uint32_t u) {
  const float x = f_of(u);
  if (isnan(x)) return 0x7FC0u;
  if (isinf(x)) return (uint16_t)(u >> 16);
  const uint32_t sign = u & 0x80000000u;
  const uint32_t mag = u & 0x7FFFFFFFu;
  const uint32_t lo = mag & 0xFFFF0000u;          /* truncation toward zero */
  const uint32_t hi = lo + 0x10000u;              /* next value away from zero */
  const double ax = fabs((double)x);
  const double vlo = (double)f_of(lo);
  const double vhi = (hi >= 0x7F800000u) ? ldexp(1.0, 128) : (double)f_of(hi);
  const double dlo = ax - vlo, dhi = vhi - ax;    /* both exact in double */
  uint32_t pick;
  if (dlo < dhi) pick = lo;
  else if (dhi < dlo) pick = hi;
  else pick = ((lo >> 16) & 1u) ? hi : lo;         /* tie: even last bit */
  if (pick > 0x7F800000u) pick = 0x7F800000u;      /* (never above infinity) */
  return (uint16_t)((sign | pick) >> 16);
}

int main(int argc, char** argv) {
  if (argc == 4 && strcmp(argv[1], "sample") == 0) {
    const uint32_t stride = (uint32_t)strtoul(argv[2], NULL, 0);
    const unsigned long count = strtoul(argv[3], NULL, 0);
    for (unsigned long k = 0; k < count; ++k) printf("%04x\n", by_definition((uint32_t)(k * stride)));
    return 0;
  }
  unsigned long long bad = 0, checked = 0;
#pragma omp parallel for reduction(+ : bad, checked) schedule(static)
  for (long long hi16 = 0; hi16 < 65536; ++hi16) {
    for (uint32_t lo16 = 0; lo16 < 65536u; ++lo16) {
      const uint32_t u = ((uint32_t)hi16 << 16) | lo16;
      bad += by_integer_form(u) != by_definition(u);
      ++checked;
    }
  }
  printf("mismatches %llu checked %llu\n", bad, checked);
  return bad == 0 && checked == 4294967296ull ? 0 : 1;
}
