/*
 * quasar_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, sequential CPU implementation of QUASAR's per-step
 * loss-aware reconstruction (arXiv 2608.13966), written from the paper's
 * definitions.  It exists to check the GPU library; nothing in the product
 * path may link, load or call it.  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg use it.  It shares no code, header, table
 * or constant generator with the HIP library.
 *
 * What it computes, per quantisation group (INT) or 16-element block (NVFP4):
 *   - optional saliency EMA  v' = beta2*v + (1-beta2)*g^2       (Sec. 4.1.1;
 *     App. A.2 keeps this EMA explicitly when the optimiser has no v)
 *   - Algorithm 1 (Sec. 4.1.2): centre/half-range from min/max, then for every
 *     clip factor f: RTN codes on [c - f*rho, c + f*rho] (Eq. rtn), the
 *     saliency-weighted least-squares dequantiser (Eq. ridgefit), its score
 *     S(f) = sum h (s q + z - w)^2 (Eq. fisher-obj); keep the argmin.
 *   - NVFP4 (Sec. 4.2): fp32 tensor scale from the tensor absmax (not
 *     optimised), per block: candidate search scales give E2M1 codes, the
 *     E4M3 block scale is fitted to minimise the same objective, argmin kept.
 *   - variants: saliency weighting h, h^2 (App. A.3) or 1 (Table 5), and the
 *     INT dequantiser deployed in fp16/bf16 (rounded before r and the score).
 *   - symmetric INT-b groups: signed codes on [-f m, f m] (m = group absmax),
 *     the scale-only weighted fit (the symmetric closed form Sec. 4.1.2
 *     mentions beside Eq. ridgefit), same objective and selection.
 *   - Rubin INT3 LUT (App. B, Eq. rubin-fit): 8x64 blocks, for each clip the
 *     INT3 codes of the range, an 8-entry E4M3 codebook of saliency-weighted
 *     code means, the candidate with the lowest score kept.
 *   - one AdamW step (the optimiser every method trains with, Sec. 6.1, whose
 *     second moment is the saliency, Sec. 4.1.1) followed by the
 *     reconstruction of the updated weights.
 *
 * Precision (the paper fixes none):
 *   - every step that decides an integer (codes, E2M1 value, E4M3 value,
 *     bf16 rounding of r) is written as explicit fp32 operations, identical on
 *     both implementations, so that discrete outcomes are comparable bit for
 *     bit;
 *   - the fit and the score are evaluated in fp64, sequentially, in the
 *     paper's own form (weighted means, centred sums).
 *   - a "literal fp32" mode replaces the fp64 fit/score with single-pass fp32
 *     accumulation; it is a reported diagnostic only.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared -lm
 * (no contraction, no fast-math, denormals kept; fmaf/rintf from libm are
 * the IEEE-754 operations).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include "quasar_oracle.h"

/* ------------------------------------------------------------------------ */
/* bf16 <-> fp32                                                             */
/* ------------------------------------------------------------------------ */

static float bf16_bits_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* Round-to-nearest-even fp32 -> bf16; NaN stays NaN (quiet). */
static uint16_t f32_to_bf16_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

uint16_t qor_f32_to_bf16(float f) { return f32_to_bf16_bits(f); }

/* Round-to-nearest-even fp32 -> IEEE binary16 value (returned as a float):
 * 10 explicit mantissa bits, exponent range 2^-14 .. 2^15, subnormal steps of
 * 2^-24, values at or beyond 65520 overflow to infinity (as the IEEE
 * conversion does); NaN stays NaN. */
static float f32_round_f16(float f) {
  if (f != f) return f;
  float a = fabsf(f);
  if (a >= 65520.0f) return copysignf(INFINITY, f);
  if (a == 0.0f) return f;
  int e2;
  (void)frexpf(a, &e2);                /* a in [2^(e2-1), 2^e2) */
  int E = e2 - 1;
  if (E < -14) E = -14;                /* subnormals share the 2^-24 step */
  double step = ldexp(1.0, E - 10);
  double n = nearbyint((double)a / step); /* exact quotient (power of two); RNE */
  return copysignf((float)(n * step), f);
}

float qor_f32_round_f16(float f) { return f32_round_f16(f); }

/* The deployed precision of the dequantiser (s, z): 0 fp32, 1 fp16, 2 bf16. */
static float round_param(float x, int param_dtype) {
  if (param_dtype == 1) return f32_round_f16(x);
  if (param_dtype == 2) return bf16_bits_to_f32(f32_to_bf16_bits(x));
  return x;
}

/* ------------------------------------------------------------------------ */
/* E2M1 (FP4): 1 sign, 2 exponent, 1 mantissa bit (Sec. 4.2).               */
/* Magnitudes by index 0..7: 0, 0.5, 1, 1.5, 2, 3, 4, 6.                     */
/* ------------------------------------------------------------------------ */

static const float kE2M1[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};

/* Nearest E2M1 magnitude to |y|, ties to the even mantissa bit (that is,
 * to the even index), saturating at 6.  The decision boundaries are the
 * midpoints 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5; a value exactly on a
 * midpoint goes to the neighbour whose index is even.  Returns the 4-bit
 * code: bit 3 = sign (set only for a non-zero negative value), bits 0-2 =
 * magnitude index.  Zero is always +0. */
static int e2m1_code(float y) {
  float a = fabsf(y);
  static const float mid[7] = {0.25f, 0.75f, 1.25f, 1.75f, 2.5f, 3.5f, 5.0f};
  int idx = 0;
  while (idx < 7) {
    if (a > mid[idx]) {
      idx++;
    } else if (a == mid[idx]) {
      /* tie between idx and idx+1: keep the even one */
      if ((idx & 1) != 0) idx++;
      break;
    } else {
      break;
    }
  }
  if (idx == 0) return 0;
  return ((y < 0.0f) ? 8 : 0) | idx;
}

static float e2m1_value(int code) {
  float m = kE2M1[code & 7];
  return (code & 8) ? -m : m;
}

int qor_e2m1_code(float y) { return e2m1_code(y); }

/* ------------------------------------------------------------------------ */
/* E4M3 (OCP FP8 E4M3FN): 1 sign, 4 exponent (bias 7), 3 mantissa bits.     */
/* Max finite 448; subnormals m * 2^-9; no infinity.                          */
/* ------------------------------------------------------------------------ */

/* Nearest non-negative E4M3 value to x >= 0 (round half to even, saturate at
 * 448).  Returns the byte code (sign bit clear). */
static int e4m3_code_nonneg(double x) {
  if (!(x > 0.0)) return 0;            /* also maps NaN to 0 */
  if (x >= 448.0) return 0x7e;         /* 0 1111 110 */
  int e2;
  (void)frexp(x, &e2);                 /* x = m * 2^e2, m in [0.5, 1) */
  int E = e2 - 1;                      /* x in [2^E, 2^(E+1)) */
  if (E < -6) E = -6;                  /* subnormal range shares 2^-9 steps */
  double step = ldexp(1.0, E - 3);     /* 3 mantissa bits */
  double n = nearbyint(x / step);      /* exact quotient (power of two); RNE */
  double val = n * step;
  if (val > 448.0) val = 448.0;
  /* encode val */
  if (val == 0.0) return 0;
  int ev;
  double mv = frexp(val, &ev);         /* val = mv * 2^ev */
  int Ev = ev - 1;
  if (Ev < -6) {                       /* subnormal: val = k * 2^-9 */
    int k = (int)(val / ldexp(1.0, -9));
    return k & 7;
  }
  int mant = (int)((mv * 2.0 - 1.0) * 8.0 + 0.5); /* exact: 0..7 */
  return ((Ev + 7) << 3) | mant;
}

static double e4m3_value(int code) {
  int e = (code >> 3) & 15, m = code & 7;
  double v = (e == 0) ? ldexp((double)m, -9) : ldexp(1.0 + m / 8.0, e - 7);
  return (code & 0x80) ? -v : v;
}

int qor_e4m3_code(double x) { return e4m3_code_nonneg(x); }
double qor_e4m3_value(int code) { return e4m3_value(code); }

/* ------------------------------------------------------------------------ */
/* Saliency EMA (Sec. 4.1.1 / App. A.2): v' = beta2 * v + (1 - beta2) * g^2   */
/* fp32, fixed order: t = g*g; u = (1-beta2)*t; v' = fmaf(beta2, v, u).      */
/* ------------------------------------------------------------------------ */

static float ema_one(float v, float g, float beta2) {
  float omb2 = 1.0f - beta2;
  float t = g * g;
  float u = omb2 * t;
  return fmaf(beta2, v, u);
}

/* ------------------------------------------------------------------------ */
/* INT-b asymmetric group (Sec. 3.1 Eq. rtn; Sec. 4.1.2 Alg. 1, Eq. ridgefit) */
/* ------------------------------------------------------------------------ */

typedef struct {
  double score;     /* S(f) of the emitted (fp32) dequantiser */
  float a, b;       /* fp32 scale s and offset z */
  int degenerate;   /* 0 regular, 1 zero saliency, 2 rank-deficient */
} int_fit;

/* Codes of clip factor f (Alg. 1: range [c - f rho, c + f rho]).
 * fp32 realisation of q = clamp(round((w - lo)/s)) with lo = c - f rho,
 * s = 2 f rho / qmax:
 *   u   = fmaf(w, 1/rho, -(c/rho))        normalised position, ~[-1, 1]
 *   x   = fmaf(u, qmax/(2f), qmax/2)      ( = (w - lo)/s in exact math)
 *   q   = min(max(rint(x), 0), qmax)      round half to even, clamp. */
static void int_codes(const float* u, int n, float alpha, float beta, float qmaxf, float* q) {
  for (int i = 0; i < n; i++) {
    float x = fmaf(u[i], alpha, beta);
    float r = rintf(x);
    if (r < 0.0f) r = 0.0f;
    if (r > qmaxf) r = qmaxf;
    q[i] = r + 0.0f; /* +0 for a rounded -0 */
  }
}

/* Eq. ridgefit written out in fp64: weighted means, centred sums. */
static int_fit int_fit_fp64(const float* w, const float* h, const float* q, int n, double qmax,
                            float s_rtn, float lo, int param_dtype) {
  int_fit out;
  double sh = 0.0, shq = 0.0, shw = 0.0;
  for (int i = 0; i < n; i++) {
    sh += (double)h[i];
    shq += (double)h[i] * (double)q[i];
    shw += (double)h[i] * (double)w[i];
  }
  double a, b;
  if (sh == 0.0) {
    /* no saliency information: keep the RTN dequantiser of this range */
    a = s_rtn;
    b = lo;
    out.degenerate = 1;
  } else {
    double qbar = shq / sh, wbar = shw / sh;
    double sqq = 0.0, sqw = 0.0;
    for (int i = 0; i < n; i++) {
      double dq = (double)q[i] - qbar;
      double dw = (double)w[i] - wbar;
      sqq += (double)h[i] * dq * dq;
      sqw += (double)h[i] * dq * dw;
    }
    if (sqq <= 1e-12 * sh * qmax * qmax) {
      /* all saliency on one code: slope undetermined, keep the RTN step,
       * fit the offset (weighted mean) */
      a = s_rtn;
      out.degenerate = 2;
    } else {
      a = sqw / sqq;
      out.degenerate = 0;
    }
    b = wbar - a * qbar;
  }
  /* fp32, then the deployed precision; the score is that of the dequantiser
   * actually emitted */
  out.a = round_param((float)a, param_dtype);
  out.b = round_param((float)b, param_dtype);
  /* Eq. fisher-obj for the dequantiser actually emitted */
  double s = 0.0;
  for (int i = 0; i < n; i++) {
    double e = (double)out.a * (double)q[i] + (double)out.b - (double)w[i];
    s += (double)h[i] * e * e;
  }
  out.score = s;
  return out;
}

/* Literal fp32 reading: raw single-pass moments and solve in fp32. */
static int_fit int_fit_fp32(const float* w, const float* h, const float* q, int n, float qmax,
                            float s_rtn, float lo, int param_dtype) {
  int_fit out;
  float sh = 0.f, shq = 0.f, shqq = 0.f, shw = 0.f, shqw = 0.f;
  for (int i = 0; i < n; i++) {
    float hq = h[i] * q[i];
    sh += h[i];
    shq += hq;
    shqq += hq * q[i];
    shw += h[i] * w[i];
    shqw += hq * w[i];
  }
  float a, b;
  if (sh == 0.f) {
    a = s_rtn;
    b = lo;
    out.degenerate = 1;
  } else {
    float d = sh * shqq - shq * shq;
    if (d <= 1e-12f * sh * sh * qmax * qmax) {
      a = s_rtn;
      out.degenerate = 2;
    } else {
      a = (sh * shqw - shq * shw) / d;
      out.degenerate = 0;
    }
    b = (shw - a * shq) / sh;
  }
  out.a = a = round_param(a, param_dtype);
  out.b = b = round_param(b, param_dtype);
  float s = 0.f;
  for (int i = 0; i < n; i++) {
    float e = fmaf(a, q[i], b) - w[i];
    s += h[i] * e * e;
  }
  out.score = (double)s;
  return out;
}

/* One INT group.  w, h: n values.  Outputs: codes (n bytes), a, b, r32 (n
 * fp32 values a*q+b), best clip, its score; scores[k] for every clip when
 * non-NULL; diag[0..3] = { S_RTN(f=1 min-max), S_LS(first clip), unused,
 * degenerate flag of the chosen fit } when non-NULL. */
static void int_group(const float* w, const float* h, int n, int bits, const float* clips, int K,
                      int fp32_mode, int param_dtype, uint8_t* codes, float* a_out, float* b_out,
                      float* r32, int* best_out, double* err_out, double* scores, double* diag) {
  const int qmax = (1 << bits) - 1;
  const float qmaxf = (float)qmax;
  float mn = w[0], mx = w[0];
  for (int i = 1; i < n; i++) {
    if (w[i] < mn) mn = w[i];
    if (w[i] > mx) mx = w[i];
  }
  if (diag) diag[0] = diag[1] = diag[2] = diag[3] = 0.0;
  if (mx == mn) {
    /* constant group: every code 0, s = 0, z = w in the deployed precision
     * (exact reconstruction at fp32) */
    const float z = round_param(mn, param_dtype);
    double s = 0.0;
    for (int i = 0; i < n; i++) {
      codes[i] = 0;
      r32[i] = z;
      const double d = (double)z - (double)w[i];
      s += (double)h[i] * d * d;
    }
    *a_out = 0.0f;
    *b_out = z;
    *best_out = 0;
    *err_out = s;
    if (scores)
      for (int k = 0; k < K; k++) scores[k] = s;
    return;
  }
  /* Alg. 1, first line: centre and half-range */
  const float c = 0.5f * (mx + mn);
  const float rho = 0.5f * (mx - mn);
  const float rrho = 1.0f / rho;
  const float nc = -(c * rrho);
  float u[QOR_MAX_GROUP], q[QOR_MAX_GROUP], qbest[QOR_MAX_GROUP];
  for (int i = 0; i < n; i++) u[i] = fmaf(w[i], rrho, nc);
  const float beta = 0.5f * qmaxf;

  int best = 0;
  int_fit fbest = {0};
  for (int k = 0; k < K; k++) {
    const float f = clips[k];
    const float alpha = qmaxf / (2.0f * f);
    int_codes(u, n, alpha, beta, qmaxf, q);
    /* the RTN dequantiser of this range (used only by the degenerate cases) */
    const float fr = f * rho;
    const float s_rtn = (2.0f * fr) / qmaxf;
    const float lo = c - fr;
    int_fit fk = fp32_mode ? int_fit_fp32(w, h, q, n, qmaxf, s_rtn, lo, param_dtype)
                           : int_fit_fp64(w, h, q, n, (double)qmax, s_rtn, lo, param_dtype);
    if (scores) scores[k] = fk.score;
    if (diag && k == 0) diag[1] = fk.score;
    if (k == 0 || fk.score < fbest.score) { /* strict: ties keep the lowest index */
      best = k;
      fbest = fk;
      memcpy(qbest, q, sizeof(float) * (size_t)n);
    }
  }
  for (int i = 0; i < n; i++) {
    codes[i] = (uint8_t)qbest[i];
    r32[i] = fmaf(fbest.a, qbest[i], fbest.b);
  }
  *a_out = fbest.a;
  *b_out = fbest.b;
  *best_out = best;
  *err_out = fbest.score;
  if (diag) {
    /* Standard QAT (Sec. 3.1): min-max range, its own (s, z), no fit.
     * Codes by the same fp32 recipe at f = 1. */
    const float s1 = (2.0f * rho) / qmaxf;
    const float lo1 = c - rho;
    int_codes(u, n, qmaxf / 2.0f, beta, qmaxf, q);
    double s = 0.0;
    for (int i = 0; i < n; i++) {
      double e = (double)s1 * (double)q[i] + (double)lo1 - (double)w[i];
      s += (double)h[i] * e * e;
    }
    diag[0] = s;
    diag[3] = (double)fbest.degenerate;
  }
}

/* ------------------------------------------------------------------------ */
/* Symmetric INT-b group: r = s q, q in [-Q, Q], Q = 2^(b-1) - 1              */
/* ------------------------------------------------------------------------ */

/* Codes of clip f: q = clamp(rint(w / (f m / Q)), -Q, Q), realised in fp32 as
 * (w * (1/m)) * (Q/f); the scale minimising Eq. fisher-obj for fixed codes is
 * s* = sum h q w / sum h q^2 (fp64; the RTN scale f m / Q when sum h q^2 = 0),
 * rounded to fp32 and then to the deployed precision; the score is that of the
 * emitted s.  An all-zero group has codes 0 and s = 0. */
static void sym_group(const float* w, const float* h, int n, int bits, const float* clips, int K,
                      int param_dtype, uint8_t* codes, float* s_out, float* r32, int* best_out, double* err_out,
                      double* scores) {
  const int Q = (1 << (bits - 1)) - 1;
  const float Qf = (float)Q;
  float m = 0.0f;
  for (int i = 0; i < n; i++) {
    const float a = fabsf(w[i]);
    if (a > m) m = a;
  }
  if (m == 0.0f) {
    for (int i = 0; i < n; i++) {
      codes[i] = 0;
      r32[i] = 0.0f;
    }
    *s_out = 0.0f;
    *best_out = 0;
    *err_out = 0.0;
    if (scores)
      for (int k = 0; k < K; k++) scores[k] = 0.0;
    return;
  }
  const float rm = 1.0f / m;
  float u[QOR_MAX_GROUP], q[QOR_MAX_GROUP], qbest[QOR_MAX_GROUP];
  for (int i = 0; i < n; i++) u[i] = w[i] * rm;
  int best = 0;
  double sbest = 0.0;
  float abest = 0.0f;
  for (int k = 0; k < K; k++) {
    const float cq = Qf / clips[k];
    double sqq = 0.0, sqw = 0.0;
    for (int i = 0; i < n; i++) {
      float x = rintf(u[i] * cq);
      if (x < -Qf) x = -Qf;
      if (x > Qf) x = Qf;
      q[i] = x + 0.0f;
      sqq += (double)h[i] * (double)q[i] * (double)q[i];
      sqw += (double)h[i] * (double)q[i] * (double)w[i];
    }
    const double sstar = sqq == 0.0 ? (double)((clips[k] * m) / Qf) : sqw / sqq;
    const float a = round_param((float)sstar, param_dtype);
    double sc = 0.0;
    for (int i = 0; i < n; i++) {
      const double d = (double)a * (double)q[i] - (double)w[i];
      sc += (double)h[i] * d * d;
    }
    if (scores) scores[k] = sc;
    if (k == 0 || sc < sbest) {
      best = k;
      sbest = sc;
      abest = a;
      memcpy(qbest, q, sizeof(float) * (size_t)n);
    }
  }
  for (int i = 0; i < n; i++) {
    codes[i] = (uint8_t)((int)qbest[i] & ((1 << bits) - 1)); /* two's complement in b bits */
    r32[i] = abest * qbest[i];
  }
  *s_out = abest;
  *best_out = best;
  *err_out = sbest;
}

/* ------------------------------------------------------------------------ */
/* NVFP4 block (Sec. 4.2)                                                    */
/* ------------------------------------------------------------------------ */

/* One 16-element block.  st: fp32 tensor scale (amax / (6*448)). */
static void nvfp4_block(const float* w, const float* h, int n, float st, const float* clips, int K,
                        int fp32_mode, uint8_t* codes, uint8_t* e_out, float* r32, int* best_out,
                        double* err_out, double* scores, double* diag) {
  float m = 0.0f;
  for (int i = 0; i < n; i++) {
    float a = fabsf(w[i]);
    if (a > m) m = a;
  }
  if (diag) diag[0] = diag[1] = diag[2] = diag[3] = 0.0;
  if (m == 0.0f || st == 0.0f) {
    for (int i = 0; i < n; i++) {
      codes[i] = 0;
      r32[i] = 0.0f;
    }
    *e_out = 0;
    *best_out = 0;
    double s = 0.0;
    for (int i = 0; i < n; i++) s += (double)h[i] * (double)w[i] * (double)w[i];
    *err_out = s;
    if (scores)
      for (int k = 0; k < K; k++) scores[k] = s;
    return;
  }
  /* candidate search scale sigma_f = f*m/6; y = w / sigma_f, realised as
   * (w * (1/m)) * (6/f) in fp32 */
  const float rm = 1.0f / m;
  float u[16], qv[16];
  int qc[16], qbest[16];
  for (int i = 0; i < n; i++) u[i] = w[i] * rm;

  int best = 0, ebest = 0;
  double sbest = 0.0, xbest = 0.0;
  float sblk_best = 0.0f;
  for (int k = 0; k < K; k++) {
    const float ck = 6.0f / clips[k];
    for (int i = 0; i < n; i++) {
      qc[i] = e2m1_code(u[i] * ck);
      qv[i] = e2m1_value(qc[i]);
    }
    /* scale-only weighted least squares: s* = sum h q w / sum h q^2 */
    double x;
    if (fp32_mode) {
      float sqq = 0.f, sqw = 0.f;
      for (int i = 0; i < n; i++) {
        sqq += h[i] * qv[i] * qv[i];
        sqw += h[i] * qv[i] * w[i];
      }
      float sstar = (sqq == 0.f) ? clips[k] * m / 6.0f : sqw / sqq;
      x = (double)(sstar / st);
    } else {
      double sqq = 0.0, sqw = 0.0;
      for (int i = 0; i < n; i++) {
        sqq += (double)h[i] * (double)qv[i] * (double)qv[i];
        sqw += (double)h[i] * (double)qv[i] * (double)w[i];
      }
      double sstar = (sqq == 0.0) ? (double)clips[k] * (double)m / 6.0 : sqw / sqq;
      x = sstar / (double)st;
    }
    /* the objective is a parabola in the scale, so the best E4M3 value is
     * the one nearest to s_star / S_t */
    const int e = e4m3_code_nonneg(x);
    const float sblk = st * (float)e4m3_value(e);
    double s = 0.0;
    if (fp32_mode) {
      float sf = 0.f;
      for (int i = 0; i < n; i++) {
        float d = sblk * qv[i] - w[i];
        sf += h[i] * d * d;
      }
      s = (double)sf;
    } else {
      for (int i = 0; i < n; i++) {
        double d = (double)sblk * (double)qv[i] - (double)w[i];
        s += (double)h[i] * d * d;
      }
    }
    if (scores) scores[k] = s;
    if (k == 0 || s < sbest) {
      best = k;
      sbest = s;
      ebest = e;
      xbest = x;
      sblk_best = sblk;
      memcpy(qbest, qc, sizeof(int) * (size_t)n);
    }
  }
  for (int i = 0; i < n; i++) {
    codes[i] = (uint8_t)qbest[i];
    r32[i] = sblk_best * e2m1_value(qbest[i]);
  }
  *e_out = (uint8_t)ebest;
  *best_out = best;
  *err_out = sbest;
  if (diag) {
    /* Standard NVFP4 QAT: codes from sigma_1 = m/6, RTN block scale
     * E4M3(m / 6 / S_t), no fit */
    const int ertn = e4m3_code_nonneg(((double)m / 6.0) / (double)st);
    const float srtn = st * (float)e4m3_value(ertn);
    double s = 0.0;
    for (int i = 0; i < n; i++) {
      float qq = e2m1_value(e2m1_code(u[i] * 6.0f));
      double d = (double)srtn * (double)qq - (double)w[i];
      s += (double)h[i] * d * d;
    }
    diag[0] = s;
    diag[2] = xbest;
  }
}

/* ------------------------------------------------------------------------ */
/* Code packing (layout definitions; the paper prescribes none)              */
/*   INT4 / NVFP4: two codes per byte, even element in the low nibble.       */
/*   INT2: four per byte, element 4k+j at bits 2j.                           */
/*   INT3: per group a little-endian bit stream, code i at bits [3i, 3i+3).  */
/* Groups follow each other in row-major order.                              */
/* ------------------------------------------------------------------------ */

void qor_pack_group(const uint8_t* codes, int n, int bits, uint8_t* out) {
  int nbytes = (n * bits) / 8;
  memset(out, 0, (size_t)nbytes);
  for (int i = 0; i < n; i++) {
    int bit = i * bits;
    for (int t = 0; t < bits; t++, bit++) {
      if ((codes[i] >> t) & 1) out[bit >> 3] |= (uint8_t)(1u << (bit & 7));
    }
  }
}

void qor_unpack_group(const uint8_t* in, int n, int bits, uint8_t* codes) {
  for (int i = 0; i < n; i++) {
    int v = 0;
    int bit = i * bits;
    for (int t = 0; t < bits; t++, bit++) v |= ((in[bit >> 3] >> (bit & 7)) & 1) << t;
    codes[i] = (uint8_t)v;
  }
}

/* ------------------------------------------------------------------------ */
/* Tensor-level driver                                                       */
/* ------------------------------------------------------------------------ */

static float load_w(const void* W, int w_bf16, int64_t idx) {
  return w_bf16 ? bf16_bits_to_f32(((const uint16_t*)W)[idx]) : ((const float*)W)[idx];
}

float qor_absmax(const void* W, int w_bf16, int64_t n) {
  float m = 0.0f;
  for (int64_t i = 0; i < n; i++) {
    float a = fabsf(load_w(W, w_bf16, i));
    if (a > m) m = a;
  }
  return m;
}

int qor_reconstruct(const qor_desc* d, int64_t row0, int64_t row1, const void* W, const float* v,
                    const void* g, float tensor_amax, float* v_out, uint8_t* codes_packed,
                    uint8_t* codes_unpacked, float* scale, float* zero, uint8_t* e4m3, void* r,
                    uint8_t* best_clip, float* err, double* scores, double* diag) {
  const int G = d->nvfp4 == 1 ? 16 : d->group;
  if (d->nvfp4 < 0 || d->nvfp4 > 2) return -4;
  if (G <= 0 || G > QOR_MAX_GROUP || d->cols % G != 0) return -2;
  if (d->n_clips < 1 || d->n_clips > QOR_MAX_CLIPS) return -1;
  if (d->nvfp4 != 1 && (d->bits < 2 || d->bits > 4)) return -4;
  if (d->weighting < 0 || d->weighting > 2) return -1;
  if (d->param_dtype < 0 || d->param_dtype > 2 || (d->nvfp4 == 1 && d->param_dtype != 0)) return -4;
  const int bits = d->nvfp4 == 1 ? 4 : d->bits;
  const int64_t gpr = d->cols / G; /* groups per row */
  const int K = d->n_clips;
  const float st = tensor_amax / 2688.0f; /* 6 * 448: E2M1 max times E4M3 max */
  float w[QOR_MAX_GROUP], h[QOR_MAX_GROUP], r32[QOR_MAX_GROUP];
  uint8_t codes[QOR_MAX_GROUP];
  for (int64_t row = row0; row < row1; row++) {
    for (int64_t j = 0; j < gpr; j++) {
      const int64_t gid = row * gpr + j;
      const int64_t base = gid * G;
      for (int i = 0; i < G; i++) {
        w[i] = load_w(W, d->w_bf16, base + i);
        float vi = v[base + i];
        if (g) {
          float gi = d->g_bf16 ? bf16_bits_to_f32(((const uint16_t*)g)[base + i])
                               : ((const float*)g)[base + i];
          vi = ema_one(vi, gi, d->beta2);
          if (v_out) v_out[base + i] = vi;
        }
        /* saliency weighting: h (Sec. 4.1.1), h^2 (App. A.3), or none, h = 1
         * (the scale-search-only ablation of Table 5) */
        h[i] = d->weighting == 1 ? vi * vi : d->weighting == 2 ? 1.0f : vi;
      }
      int best = 0;
      double e = 0.0;
      double* sc = scores ? scores + gid * K : NULL;
      double* dg = diag ? diag + gid * 4 : NULL;
      if (d->nvfp4 == 2) {
        float a = 0.f;
        sym_group(w, h, G, bits, d->clips, K, d->param_dtype, codes, &a, r32, &best, &e, sc);
        if (scale) scale[gid] = a;
        if (zero) zero[gid] = 0.0f;
      } else if (d->nvfp4) {
        uint8_t eb = 0;
        nvfp4_block(w, h, G, st, d->clips, K, d->fp32_mode, codes, &eb, r32, &best, &e, sc, dg);
        if (e4m3) e4m3[gid] = eb;
      } else {
        float a = 0.f, b = 0.f;
        int_group(w, h, G, bits, d->clips, K, d->fp32_mode, d->param_dtype, codes, &a, &b, r32, &best, &e,
                  sc, dg);
        if (scale) scale[gid] = a;
        if (zero) zero[gid] = b;
      }
      if (codes_packed) qor_pack_group(codes, G, bits, codes_packed + gid * (G * bits / 8));
      if (codes_unpacked) memcpy(codes_unpacked + base, codes, (size_t)G);
      if (r) {
        for (int i = 0; i < G; i++) {
          if (d->w_bf16)
            ((uint16_t*)r)[base + i] = f32_to_bf16_bits(r32[i]);
          else
            ((float*)r)[base + i] = r32[i];
        }
      }
      if (best_clip) best_clip[gid] = (uint8_t)best;
      if (err) err[gid] = (float)e;
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* AdamW step, then reconstruction of the updated weights                    */
/* ------------------------------------------------------------------------ */

/* Host-side constants of one AdamW step (fp64, then fp32). */
void qor_adamw_constants(const qor_adamw* o, float* omb1, float* omb2, float* decay, float* step_size,
                         float* rbc2) {
  *omb1 = 1.0f - o->beta1;
  *omb2 = 1.0f - o->beta2;
  *decay = (float)(1.0 - (double)o->lr * (double)o->weight_decay);
  const double bc1 = 1.0 - pow((double)o->beta1, (double)o->step);
  const double bc2 = 1.0 - pow((double)o->beta2, (double)o->step);
  *step_size = (float)((double)o->lr / bc1);
  *rbc2 = (float)(1.0 / sqrt(bc2));
}

/* One element of AdamW with decoupled weight decay, fp32 in this order:
 *   m' = fmaf(beta1, m, (1 - beta1) g)
 *   v' = fmaf(beta2, v, (1 - beta2) (g g))
 *   d  = fmaf(sqrtf(v'), 1/sqrt(1 - beta2^t), eps)
 *   w' = fmaf(-lr/(1 - beta1^t), m'/d, w (1 - lr wd))                        */
static float adamw_one(float w, float* m, float* v, float g, float beta1, float beta2, float omb1, float omb2,
                       float eps, float decay, float step_size, float rbc2) {
  const float mm = fmaf(beta1, *m, omb1 * g);
  const float t = g * g;
  const float vv = fmaf(beta2, *v, omb2 * t);
  const float den = fmaf(sqrtf(vv), rbc2, eps);
  const float upd = mm / den;
  *m = mm;
  *v = vv;
  return fmaf(-step_size, upd, w * decay);
}

int qor_adamw_reconstruct(const qor_desc* d, const qor_adamw* o, int64_t row0, int64_t row1, void* W,
                          float* m, float* v, const void* g, float tensor_amax, uint8_t* codes_packed,
                          uint8_t* codes_unpacked, float* scale, float* zero, uint8_t* e4m3, void* r,
                          uint8_t* best_clip, float* err, double* scores, double* diag) {
  if (o->step < 1 || !(o->eps > 0.0f) || !(o->beta1 >= 0.0f && o->beta1 < 1.0f) ||
      !(o->beta2 >= 0.5f && o->beta2 < 1.0f))
    return -1;
  float omb1, omb2, decay, step_size, rbc2;
  qor_adamw_constants(o, &omb1, &omb2, &decay, &step_size, &rbc2);
  for (int64_t idx = row0 * d->cols; idx < row1 * d->cols; idx++) {
    const float gi = d->g_bf16 ? bf16_bits_to_f32(((const uint16_t*)g)[idx]) : ((const float*)g)[idx];
    const float wn = adamw_one(load_w(W, d->w_bf16, idx), &m[idx], &v[idx], gi, o->beta1, o->beta2, omb1,
                               omb2, o->eps, decay, step_size, rbc2);
    if (d->w_bf16)
      ((uint16_t*)W)[idx] = f32_to_bf16_bits(wn);
    else
      ((float*)W)[idx] = wn;
  }
  /* the updated second moment is the saliency; no further EMA */
  return qor_reconstruct(d, row0, row1, W, v, NULL, tensor_amax, NULL, codes_packed, codes_unpacked, scale,
                         zero, e4m3, r, best_clip, err, scores, diag);
}

/* ------------------------------------------------------------------------ */
/* Rubin INT3 LUT (App. B, Eq. rubin-fit)                                    */
/* ------------------------------------------------------------------------ */

/* Nearest E4M3 value to any x (sign-symmetric RNE, saturating at 448); zero
 * and NaN give the +0 code. */
static int e4m3_code_signed(double x) {
  if (!(x == x) || x == 0.0) return 0;
  const int c = e4m3_code_nonneg(fabs(x));
  return (x < 0.0 && c != 0) ? (c | 0x80) : c;
}

int qor_e4m3_code_signed(double x) { return e4m3_code_signed(x); }

/* One block of n = 512 weights (8 rows x 64 columns, element i = row * 64 +
 * col).  For each clip f: the INT3 codes of the range [c - f rho, c + f rho]
 * (the same fp32 recipe as the affine INT groups, qmax = 7), then for every
 * code k the entry C_k = E4M3(sum_{q=k} h w / sum_{q=k} h) (fp64 sums in
 * element order; a code with no saliency mass keeps the E4M3 value of its grid
 * level fmaf(k, s_f, lo_f)), and the score sum h (C_q - w)^2 (fp64).  The
 * lowest score wins, ties to the lowest index.  A constant block has every
 * code 0 and C = E4M3(w) for all entries. */
static void rubin_block(const float* w, const float* h, int n, const float* clips, int K, uint8_t* codes,
                        uint8_t* lut, float* r32, int* best_out, double* err_out, double* scores) {
  float mn = w[0], mx = w[0];
  for (int i = 1; i < n; i++) {
    if (w[i] < mn) mn = w[i];
    if (w[i] > mx) mx = w[i];
  }
  const float qmaxf = 7.0f;
  if (mx == mn) {
    const int e = e4m3_code_signed((double)mn);
    const double cv = e4m3_value(e);
    double s = 0.0;
    for (int i = 0; i < n; i++) {
      codes[i] = 0;
      r32[i] = (float)cv;
      const double d = cv - (double)w[i];
      s += (double)h[i] * d * d;
    }
    for (int k = 0; k < 8; k++) lut[k] = (uint8_t)e;
    *best_out = 0;
    *err_out = s;
    if (scores)
      for (int k = 0; k < K; k++) scores[k] = s;
    return;
  }
  const float c = 0.5f * (mx + mn);
  const float rho = 0.5f * (mx - mn);
  const float rrho = 1.0f / rho;
  const float nc = -(c * rrho);
  static const int kMaxN = 512;
  float u[512], q[512];
  uint8_t qbest[512];
  for (int i = 0; i < n && i < kMaxN; i++) u[i] = fmaf(w[i], rrho, nc);
  double sbest = 0.0;
  int best = 0;
  uint8_t lbest[8] = {0};
  for (int k = 0; k < K; k++) {
    const float f = clips[k];
    int_codes(u, n, qmaxf / (2.0f * f), 0.5f * qmaxf, qmaxf, q);
    const float fr = f * rho;
    const float s_rtn = (2.0f * fr) / qmaxf;
    const float lo = c - fr;
    double sh[8] = {0}, shw[8] = {0};
    for (int i = 0; i < n; i++) {
      const int b = (int)q[i];
      sh[b] += (double)h[i];
      shw[b] += (double)h[i] * (double)w[i];
    }
    uint8_t l[8];
    double cv[8];
    for (int b = 0; b < 8; b++) {
      /* Eq. rubin-fit: the loss-aware mean of the code's weights, in E4M3 */
      const double mean = sh[b] > 0.0 ? shw[b] / sh[b] : (double)fmaf((float)b, s_rtn, lo);
      l[b] = (uint8_t)e4m3_code_signed(mean);
      cv[b] = e4m3_value(l[b]);
    }
    double sc = 0.0;
    for (int i = 0; i < n; i++) {
      const double d = cv[(int)q[i]] - (double)w[i];
      sc += (double)h[i] * d * d;
    }
    if (scores) scores[k] = sc;
    if (k == 0 || sc < sbest) {
      sbest = sc;
      best = k;
      memcpy(lbest, l, 8);
      for (int i = 0; i < n; i++) qbest[i] = (uint8_t)q[i];
    }
  }
  for (int i = 0; i < n; i++) {
    codes[i] = qbest[i];
    r32[i] = (float)e4m3_value(lbest[qbest[i]]);
  }
  memcpy(lut, lbest, 8);
  *best_out = best;
  *err_out = sbest;
}

int qor_rubin_reconstruct(const qor_desc* d, int64_t rb0, int64_t rb1, const void* W, const float* v,
                          const void* g, float* v_out, uint8_t* codes_packed, uint8_t* codes_unpacked,
                          uint8_t* lut, void* r, uint8_t* best_clip, float* err, double* scores) {
  if (d->rows % 8 != 0 || d->cols % 64 != 0 || d->rows < 8 || d->cols < 64) return -2;
  if (d->n_clips < 1 || d->n_clips > QOR_MAX_CLIPS) return -1;
  if (d->weighting < 0 || d->weighting > 2) return -1;
  const int64_t bpr = d->cols / 64; /* blocks per block-row */
  const int K = d->n_clips;
  float w[512], h[512], r32[512];
  uint8_t codes[512];
  for (int64_t rb = rb0; rb < rb1; rb++) {   /* block rows: rows 8 rb .. 8 rb + 7 */
    for (int64_t cb = 0; cb < bpr; cb++) {
      const int64_t bid = rb * bpr + cb;
      for (int i = 0; i < 512; i++) {
        const int64_t idx = (rb * 8 + i / 64) * d->cols + cb * 64 + i % 64;
        w[i] = load_w(W, d->w_bf16, idx);
        float vi = v[idx];
        if (g) {
          const float gi = d->g_bf16 ? bf16_bits_to_f32(((const uint16_t*)g)[idx]) : ((const float*)g)[idx];
          vi = ema_one(vi, gi, d->beta2);
          if (v_out) v_out[idx] = vi;
        }
        h[i] = d->weighting == 1 ? vi * vi : d->weighting == 2 ? 1.0f : vi;
      }
      int best = 0;
      double e = 0.0;
      rubin_block(w, h, 512, d->clips, K, codes, lut ? lut + bid * 8 : (uint8_t[8]){0}, r32, &best, &e,
                  scores ? scores + bid * K : NULL);
      if (codes_packed) qor_pack_group(codes, 512, 3, codes_packed + bid * 192);
      for (int i = 0; i < 512; i++) {
        const int64_t idx = (rb * 8 + i / 64) * d->cols + cb * 64 + i % 64;
        if (codes_unpacked) codes_unpacked[idx] = codes[i];
        if (r) {
          if (d->w_bf16)
            ((uint16_t*)r)[idx] = f32_to_bf16_bits(r32[i]);
          else
            ((float*)r)[idx] = r32[i];
        }
      }
      if (best_clip) best_clip[bid] = (uint8_t)best;
      if (err) err[bid] = (float)e;
    }
  }
  return 0;
}
