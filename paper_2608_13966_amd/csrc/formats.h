// formats.h -- E2M1 (FP4) and E4M3 (FP8) rounding used by the NVFP4 kernel
// (Sec. 4.2: E2M1 codes, E4M3 block scale).  Written as __host__ __device__
// so the library's own host-side unit check can exercise the exact code that
// runs on the GPU.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

namespace quasar {

__host__ __device__ inline uint32_t fbits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}
__host__ __device__ inline float bitsf(uint32_t u) {
  float f;
  memcpy(&f, &u, 4);
  return f;
}

// Nearest E2M1 value to y (magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6), ties to the
// even mantissa bit, saturating at 6; the sign follows y (a zero result may be
// -0; the emitted code is always +0).  The spacing of E2M1 is 2^(E-1) on
// [2^E, 2^(E+1)) with E clamped below at 0, so adding and subtracting
// 1.5 * 2^(E+22) rounds |y| to that spacing in one IEEE addition (RNE).
__host__ __device__ inline float e2m1_round(float y) {
  const uint32_t ub = fbits(y);
  const float a = bitsf(ub & 0x7fffffffu);
  uint32_t e = ub & 0x7f800000u;
  e = e > 0x3f800000u ? e : 0x3f800000u;
  const float C = bitsf(e + (22u << 23) + 0x00400000u);
  float q = (a + C) - C;
  q = fminf(q, 6.0f);
  return bitsf(fbits(q) | (ub & 0x80000000u));
}

// 4-bit code of an E2M1 value produced by e2m1_round: (sign << 3) | index.
__host__ __device__ inline uint32_t e2m1_code_of(float q) {
  const uint32_t ub = fbits(q);
  const float a = bitsf(ub & 0x7fffffffu);
  uint32_t idx;
  if (a >= 1.0f) {
    const uint32_t ex = ((ub >> 23) & 0xffu) - 127u;  // 0, 1, 2
    idx = ((ex + 1u) << 1) | ((ub >> 22) & 1u);
  } else {
    idx = (a == 0.5f) ? 1u : 0u;
  }
  return idx == 0u ? 0u : (idx | ((ub >> 28) & 8u));
}

// Nearest non-negative E4M3FN value to x (RNE, saturating at 448, subnormal
// step 2^-9); returns the value and stores the byte in *code.
__host__ __device__ inline double e4m3_round(double x, uint32_t* code) {
  if (!(x > 0.0)) {
    *code = 0;
    return 0.0;
  }
  if (x >= 448.0) {
    *code = 0x7e;
    return 448.0;
  }
  int e2;
  (void)frexp(x, &e2);
  int E = e2 - 1;
  if (E < -6) E = -6;
  const double n = rint(ldexp(x, 3 - E));  // exact scaling by a power of two
  const double val = ldexp(n, E - 3);
  if (val < 0.015625) {  // below 2^-6: subnormal, val = k * 2^-9
    *code = (uint32_t)ldexp(val, 9);
  } else {
    int ev;
    const double mv = frexp(val, &ev);
    *code = (uint32_t)((ev - 1 + 7) << 3) | (uint32_t)((mv * 2.0 - 1.0) * 8.0);
  }
  return val;
}

// Nearest non-negative E4M3FN value to an fp32 x (RNE, saturating at 448,
// subnormal step 2^-9); returns the value and stores the byte in *code.
// Normal range: round the fp32 mantissa to 3 bits in integer arithmetic;
// subnormal range: one IEEE addition of 1.5 * 2^14 rounds to a multiple of 2^-9.
__host__ __device__ inline float e4m3_round_f32(float x, uint32_t* code) {
  const uint32_t xb = fbits(x);
  const uint32_t rn = (xb + 0x7ffffu + ((xb >> 20) & 1u)) & 0xfff00000u;
  const float vs = (x + 24576.0f) - 24576.0f;
  float v = (x >= 0.015625f) ? bitsf(rn) : vs;
  v = (x >= 448.0f) ? 448.0f : v;
  v = (x > 0.0f) ? v : 0.0f;  // also maps NaN to 0
  const uint32_t vb = fbits(v);
  const uint32_t cn = ((((vb >> 23) & 0xffu) - 120u) << 3) | ((vb >> 20) & 7u);
  const uint32_t cs = (uint32_t)(v * 512.0f);
  *code = (v >= 0.015625f) ? cn : cs;
  return v;
}

}  // namespace quasar
