/*
 * Oracle of the lossy 32 -> 16-bit conversion of section 5.5 (test
 * infrastructure only: nothing in the product library links this file).
 *
 * The paper's converter keeps an fp32 value's sign, exponent and top 7
 * fraction bits and drops the other 16 fraction bits. Written here from the
 * arithmetic of that operation rather than from the bit layout: a finite
 * value is rounded toward zero to 8 significant bits (normal range) or to a
 * multiple of 2^-133 (below 2^-126, the 16-bit format's subnormal quantum).
 * Infinities and signed zeros are kept. NaN has no arithmetic meaning; the
 * reading used throughout is that it becomes the quiet NaN 0x7FC0 with its
 * sign (so that no NaN turns into an infinity). The result is returned as the
 * 16-bit pattern of the exactly representable value.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static uint16_t pattern_of(float t) { /* t is exactly representable in 16 bits */
  uint32_t u;
  memcpy(&u, &t, sizeof u);
  return (uint16_t)(u >> 16);
}

uint16_t oracle_trunc16_one(float x) {
  if (isnan(x)) return signbit(x) ? 0xFFC0u : 0x7FC0u;
  if (isinf(x) || x == 0.0f) return pattern_of(x);
  const float a = fabsf(x);
  float t;
  if (a >= 0x1p-126f) {
    int e;
    const float m = frexpf(a, &e);            /* a = m * 2^e, 0.5 <= m < 1 */
    t = ldexpf(truncf(m * 256.0f), e - 8);    /* 8 significant bits, toward zero */
  } else {
    t = ldexpf(truncf(ldexpf(a, 133)), -133); /* multiple of 2^-133, toward zero */
  }
  return pattern_of(copysignf(t, x));
}

/* out[i] = converter(x[i]) for n values. */
void oracle_trunc16(const float* x, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_trunc16_one(x[i]);
}

/* out[i] = converter(the fp32 whose bit pattern is first + i), i < count:
 * lets a test walk all 2^32 inputs in slices. */
void oracle_trunc16_range(uint32_t first, int64_t count, uint16_t* out) {
  for (int64_t i = 0; i < count; ++i) {
    const uint32_t u = first + (uint32_t)i;
    float x;
    memcpy(&x, &u, sizeof x);
    out[i] = oracle_trunc16_one(x);
  }
}
