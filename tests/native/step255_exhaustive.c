/* Exhaustive check of the level spacing of 8-bit linear norms used by the decode and attention
 * kernels: for every finite fp32 x, the product q = RN(x * RN(1/255)) corrected once by its
 * exact residual, RN(q + RN(x - 255 q) * RN(1/255)) (two fused multiply-adds), equals the
 * IEEE fp32 quotient RN(x / 255).  Non-finite x is passed through by the kernels and is not
 * checked here, nor is x = -0: R'max - R'min rounds to -0 only for R'max = -0, R'min = +0,
 * which compare equal, and equal norms take the kernels' zero spacing instead.  Prints the number of mismatching inputs; exit status 0 when there are none.
 * Build: gcc -O2 -fopenmp -ffp-contract=off -mfma (IEEE fp32 with denormals, as the kernels
 * run: no flush-to-zero). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float from_bits(uint32_t u) {
  float x;
  memcpy(&x, &u, 4);
  return x;
}

static uint32_t to_bits(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return u;
}

int main(void) {
  volatile float c_in = 255.0f;
  const float c = c_in;
  const float inv = 1.0f / c;
  unsigned long long bad = 0, checked = 0;
#pragma omp parallel for reduction(+ : bad, checked) schedule(static)
  for (long long i = 0; i <= 0xffffffffll; ++i) {
    const float x = from_bits((uint32_t)i);
    if (!isfinite(x) || (uint32_t)i == 0x80000000u) continue;
    const float want = x / c;
    const float q = x * inv;
    const float got = fmaf(fmaf(-q, c, x), inv, q);
    ++checked;
    if (to_bits(want) != to_bits(got)) ++bad;
  }
  printf("checked %llu finite inputs, mismatches %llu\n", checked, bad);
  return bad != 0;
}
