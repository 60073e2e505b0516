// int_common.h -- the parts of Algorithm 1 (Sec. 4.1.2) that both INT-b
// reconstruction kernels share: the tile's matrix, the load with the optional
// fused EMA / AdamW step, the group range, the closed-form fit and score of
// one candidate, and the argmin + emit.  The kernels differ only in how they
// obtain the per-candidate weighted moments (int_kernel.hip: direct sums per
// clip; int_cells_kernel.hip: one binning by code threshold per weight).
//
// Work decomposition (both kernels): a group of G weights is owned by
// L = G/16 consecutive lanes, each holding 16 consecutive weights in
// registers; a wavefront processes 64/L groups.
#pragma once

#include "device_common.h"
#include "quasar_internal.h"

namespace quasar {

constexpr int kIntN = 16;  // weights per lane

// The L lanes that hold one group, and reductions over them.  Consecutive:
// lanes L s .. L s + L - 1 (DPP inside a row of 16).  Spread: member j of
// group s sits at lane s + 8 j (L = 8, s < 8) or (s & 7) + 8 j + 32 (s >> 3)
// (L = 4, s < 16), so that no two members share an 8-lane block; LDS atomics
// from members of one group that hit the same address then do not serialise.
// Every pairing is symmetric and the operations commute, so all members end
// with bit-identical results.
template <int L, bool SPREAD>
struct Members;

template <int L>
struct Members<L, false> {
  static __device__ __forceinline__ int member(int lane) { return lane % L; }
  static __device__ __forceinline__ int slot(int lane) { return lane / L; }
  static __device__ __forceinline__ float min(float x) { return run_min<L>(x); }
  static __device__ __forceinline__ float max(float x) { return run_max<L>(x); }
  static __device__ __forceinline__ double sum(double x) { return run_sum<L>(x); }
  static __device__ __forceinline__ double min_f64(double x) { return run_min_f64<L>(x); }
};

constexpr int kDppRor8 = 0x128;  // row_ror:8 -- lane i <-> i ^ 8 inside each 16

template <int L>
struct Members<L, true> {
  static_assert(L == 4 || L == 8, "spread groups of 4 or 8 lanes");
  static __device__ __forceinline__ int member(int lane) { return L == 8 ? lane >> 3 : (lane >> 3) & 3; }
  static __device__ __forceinline__ int slot(int lane) { return L == 8 ? lane & 7 : (lane & 7) | ((lane >> 5) << 3); }
  template <typename T, typename Op>
  static __device__ __forceinline__ T reduce(T x, Op op) {
    if constexpr (sizeof(T) == 8)
      x = op(x, dpp_f64<kDppRor8>(x));
    else
      x = op(x, dpp_f32<kDppRor8>(x));
    x = pair_rows<16>(x, op);
    if constexpr (L == 8) x = pair_rows<32>(x, op);
    return x;
  }
  static __device__ __forceinline__ float min(float x) { return reduce(x, [](float a, float b) { return min_f32(a, b); }); }
  static __device__ __forceinline__ float max(float x) { return reduce(x, [](float a, float b) { return max_f32(a, b); }); }
  static __device__ __forceinline__ double sum(double x) { return reduce(x, [](double a, double b) { return a + b; }); }
  static __device__ __forceinline__ double min_f64(double x) {  // of keys
    return reduce(x, [](double a, double b) { return min_key(a, b); });
  }
};

// The buffers of the matrix a workgroup works on: the call's own, or in a
// batched launch the slot the workgroup falls in (uniform per workgroup).
struct IntMatrix {
  const void* W;
  float* v;
  const void* g;
  uint8_t* codes;
  float* scales;
  float* zeros;
  void* r;
  uint8_t* best_clip;
  float* err;
  int64_t n_groups;
  float* m;  // the fused AdamW step: first moment and where the updated W goes
  void* Wu;
};

__device__ __forceinline__ IntMatrix int_matrix(const IntParams& p, int64_t& blk) {
  IntMatrix m = {p.W, p.v, p.g, p.codes, p.scales, p.zeros, p.r, p.best_clip, p.err, p.n_groups, p.m, p.Wu};
  if (p.batch.n > 1) {
    const MatrixSlot& ms = batch_slot<IntParams>(blk);
    m = {ms.W, ms.v, ms.g, ms.codes, static_cast<float*>(ms.scales), ms.zeros, ms.r, ms.best_clip, ms.err,
         ms.n_units, ms.m, ms.Wu};
  }
  return m;
}

// Pads of the store stage (wave_store) for the INT kernels' layouts: a group
// is G ESZ / 16 chunks of 16 bytes, a lane of a consecutive layout ESZ.
template <bool SPREAD, int G, int ESZ>
__host__ __device__ constexpr int int_stage_per() { return SPREAD ? G * ESZ / 16 : ESZ; }
// LDS of one wavefront's store stage (fp32 stretches, the larger)
template <bool SPREAD, int G>
__host__ __device__ constexpr int int_stage_bytes() { return 16 * wave_stage_chunks<4, int_stage_per<SPREAD, G, 4>()>(); }

// The wavefront's stretch of the matrix: groups wave_g0 .. wave_g0 + 64 / L - 1.
template <int L>
__device__ __forceinline__ WaveImage int_image(void* stage, int64_t wave_g0, int64_t n_groups, int slot, int j,
                                               int lane) {
  constexpr int G = L * kIntN;
  const int64_t left = (n_groups - wave_g0) * G;
  return WaveImage{reinterpret_cast<uint4*>(stage), wave_g0 * G, left < 1024 ? left : 1024, slot * L + j, lane};
}

// Load the lane's 16 weights and saliencies (each byte of W, v, g once, with
// 128-bit loads), run the fused EMA (EMA 1/2) or AdamW step (EMA 3/4) and
// store their results (coalesced through the wavefront's stage), then apply
// the saliency weighting: h = v, v*v (App. A.3) or 1 (Table 5).  W stays in
// its storage format in registers.
template <bool W_BF16, int EMA, bool SPREAD, int G>
__device__ __forceinline__ void int_load(const IntParams& p, const IntMatrix& mtx, const WaveImage& im, int64_t e0,
                                         WRegs<W_BF16>& wr, float (&v)[kIntN]) {
  constexpr int P4 = int_stage_per<SPREAD, G, 4>(), P2 = int_stage_per<SPREAD, G, 2>();
  wr.load(mtx.W, e0);
  load16<false>(mtx.v, e0, v);
  if constexpr (EMA == 1 || EMA == 2) {
    float g[kIntN];
    load16<EMA == 1>(mtx.g, e0, g);
#pragma unroll
    for (int i = 0; i < kIntN; i++) {
      // v' = beta2 v + (1 - beta2) g^2 in the oracle's fp32 order
      float t = g[i] * g[i];
      float u = p.omb2 * t;
      v[i] = __builtin_fmaf(p.beta2, v[i], u);
    }
    wave_store_f32<P4>(im, mtx.v, v);
  } else if constexpr (EMA >= 3) {
    // one AdamW step first; the updated W is reconstructed and the updated
    // second moment is the saliency
    float g[kIntN], m[kIntN], w[kIntN];
    load16<EMA == 3>(mtx.g, e0, g);
    load16<false>(mtx.m, e0, m);
#pragma unroll
    for (int i = 0; i < kIntN; i++) w[i] = wr.get(i);
    adamw16(w, m, v, g, p.adam, p.beta2, p.omb2);
    wr.set(w);  // bf16 W: rounded here, and the rounded value is reconstructed
    wave_store_f32<P4>(im, mtx.v, v);
    wave_store_f32<P4>(im, mtx.m, m);
    if constexpr (W_BF16)
      wave_store<2, P2>(im, mtx.Wu, wr.d);
    else
      wave_store_f32<P4>(im, static_cast<float*>(mtx.Wu), wr.f);
  }
  if (p.weighting != 0) {
#pragma unroll
    for (int i = 0; i < kIntN; i++) v[i] = weight_of(v[i], p.weighting);
  }
}

// The group's range (Alg. 1, first line).  Asymmetric: c = (mx + mn)/2,
// rho = (mx - mn)/2, normalised position u = fmaf(w, 1/rho, -c/rho) in
// [-1, 1].  Symmetric: m = max |w| (held in mx), u = w * (1/m).
struct IntRange {
  float mn, mx, c, rho, rrho, nc;
  bool constant;  // asymmetric: mx == mn; symmetric: an all-zero group
};

template <int L, bool SYM, bool W_BF16, bool SPREAD = false>
__device__ __forceinline__ IntRange int_range(const WRegs<W_BF16>& wr) {
  using M = Members<L, SPREAD>;
  IntRange g;
  if constexpr (SYM) {
    float mx = 0.0f;
#pragma unroll
    for (int i = 0; i < kIntN; i++) mx = fmaxf(mx, fabsf(wr.get(i)));
    mx = M::max(mx);
    g.mn = 0.0f;
    g.mx = mx;
    g.constant = (mx == 0.0f);
    g.c = 0.0f;
    g.rho = mx;
    g.rrho = 1.0f / mx;
    g.nc = 0.0f;
  } else {
    float mn = wr.get(0), mx = wr.get(0);
#pragma unroll
    for (int i = 1; i < kIntN; i++) {
      mn = fminf(mn, wr.get(i));
      mx = fmaxf(mx, wr.get(i));
    }
    mn = M::min(mn);
    mx = M::max(mx);
    g.mn = mn;
    g.mx = mx;
    g.constant = (mx == mn);
    g.c = 0.5f * (mx + mn);
    g.rho = 0.5f * (mx - mn);
    g.rrho = 1.0f / g.rho;
    g.nc = -(g.c * g.rrho);
  }
  return g;
}

// The normalised position of w (the codes of clip k are then
// clamp(rint(fmaf(u, alpha_k, qmax/2)), 0, qmax), symmetric
// clamp(rint(u * alpha_k), -Q, Q)).
template <bool SYM>
__device__ __forceinline__ float int_u(float w, const IntRange& g) {
  return SYM ? w * g.rrho : __builtin_fmaf(w, g.rrho, g.nc);
}

// Clip-independent moments of the group: sum h, sum h w, sum h w^2 (fp64),
// and what bounds the error of the moments the fit is formed from: each
// term of sum h may be off by qh / G in absolute value and each term of
// sum h w by qhw / G (so qh and qhw bound the sums over the group: the
// binned kernel's fixed-point rounding; 0 where the terms are exact), and
// every fp64 sum, product and difference by rel times the magnitude of its
// terms (wabs = max |w| over the group bounds those of sum h w, sum h q w).
struct IntMoments {
  double Sv, Svw, Svww;
  double thr;  // rank-deficiency threshold 1e-12 (sum h)^2 qmax^2
  double rSv;  // 1 / sum h
  double qh, qhw, rel, wabs;
  // per-group parts of the error bounds of int_fit_ill (int_fit_bounds)
  double eD0, eN0, eN1;
};

// Best candidate so far of one lane: the key (score with the clip index in
// its low bits), the emitted (s, z) and the score as fp32; `ill` marks a
// candidate whose fit the moments cannot fix to the required accuracy.
struct IntBest {
  double key;
  float a, b, err;
  bool ill;
};

__device__ __forceinline__ IntBest int_best_init() {
  IntBest b;
  b.key = __longlong_as_double(0x7ff0000000000000ll);  // +inf
  b.a = b.b = b.err = 0.0f;
  b.ill = false;
  return b;
}

// Relative accuracy the fast forms must guarantee for the two quantities the
// fit of Eq. ridgefit divides (the determinant and the slope's numerator);
// the fitted (s, z) then agree with an exact evaluation far inside fp32.
constexpr double kFitTol = 1e-8;
// ... and for the score of the emitted dequantiser (expanded from the
// moments), relative to itself, or, for a score below 1e-13 sum h w^2 (a fit
// that is exact to that level), to that floor.
constexpr double kScoreTol = 1e-8;
constexpr double kScoreFloor = 1e-13;

// Whether the score of the emitted (s, z), expanded from the moments, may be
// off by more than kScoreTol of itself.  It differs from sum h (s q + z - w)^2
// of the exact moments by sum_i [dh_i r_i^2 - 2 d(hw)_i r_i] with
// r_i = s q_i + z, |r_i| <= |s| qmax + |z|, and by the fp64 roundings of its
// six terms.
__device__ __forceinline__ bool int_score_ill(const IntMoments& mo, double s, double z, double qmax, double A0,
                                              double A1, double A2, double score) {
  const double R = fabs(s) * qmax + fabs(z);
  const double e = mo.qh * R * R + 2.0 * mo.qhw * R +
                   mo.rel * (mo.Svww + s * s * A1 + z * z * mo.Sv + 2.0 * fabs(s * z) * A0 + 2.0 * fabs(s * A2) +
                             2.0 * fabs(z * mo.Svw));
  return e > fmax(kScoreTol * score, kScoreFloor * mo.Svww);
}

// Whether the fit of one candidate from moments A0 = sum h q, A1 = sum h q^2,
// A2 = sum h q w is ill-conditioned: the error bounds of the determinant
// D = Sv A1 - A0^2 or of the numerator Sv A2 - A0 Svw exceed kFitTol of their
// values, or D lies so close to the rank-deficiency threshold that its side
// is not certain (symmetric: sum h q^2 and sum h q w against their bounds).
// Perturbing h_i moves D by Sv ((q_i - qbar)^2 + var) <= 2 qmax^2 Sv per unit
// of h_i, and the numerator by A2 - q_i Svw (|.| <= wabs (A0 + qmax Sv)) per
// unit of h_i and by Sv q_j - A0 (|.| <= qmax Sv) per unit of h_j w_j; the
// fp64 roundings add rel times the magnitudes of the products.  The parts
// that do not depend on the clip are formed once per group:
//   eD = eD0 + rel (Sv A1 + A0^2),   eN = eN0 + eN1 A0.
template <int QMAX>
__device__ __forceinline__ void int_fit_bounds(IntMoments& mo) {
  constexpr double Q = (double)QMAX;
  mo.eD0 = 2.0 * Q * Q * mo.qh * mo.Sv;
  mo.eN0 = (mo.wabs * mo.qh + mo.qhw) * Q * mo.Sv;
  mo.eN1 = mo.wabs * (mo.qh + 4.0 * mo.rel * mo.Sv);
}

template <bool SYM, int QMAX>
__device__ __forceinline__ bool int_fit_ill(const IntMoments& mo, double A0, double A1, double A2) {
  constexpr double Q = (double)QMAX;
  // every test is evaluated and combined bitwise: short-circuit forms
  // compile to a branch per test and clip
  if constexpr (SYM) {
    const double e1 = mo.qh * Q * Q + mo.rel * A1, e2 = mo.qhw * Q + mo.rel * mo.wabs * Q * mo.Sv;
    return (A1 > 0.0) & ((e1 > kFitTol * A1) | (e2 > kFitTol * fabs(A2)));
  } else {
    const double Sv = mo.Sv;
    const double p1 = Sv * A1, p2 = A0 * A0;
    const double D = p1 - p2;
    const double eD = __builtin_fma(mo.rel, p1 + p2, mo.eD0);
    const double num = Sv * A2 - A0 * mo.Svw;
    const double eN = __builtin_fma(mo.eN1, A0, mo.eN0);
    // Sv = 0: every candidate keeps its RTN dequantiser and scores 0.  D + eD
    // <= thr: certainly rank-deficient.  D - eD <= thr: either side of the
    // threshold.  Otherwise the bounds against their values.
    const bool deficient = D + eD <= mo.thr, straddles = D - eD <= mo.thr;
    const bool loose = (eD > kFitTol * D) | (eN > kFitTol * fabs(num));
    return (Sv != 0.0) & !deficient & (straddles | loose);
  }
}

// Every clip of a group evaluated the way Eq. ridgefit and Eq. fisher-obj
// read, in fp64 straight from the group's weights: the codes, the weighted
// means qbar and wbar, the centred sums sum h (q - qbar)^2 and
// sum h (q - qbar)(w - wbar) (symmetric: sum h q^2, sum h q w), the fit,
// its rank-deficiency decision, and the score as a sum of weighted squared
// residuals of the emitted dequantiser.  The path for the rare groups whose
// moments from the fast forms cannot fix the fit to the required accuracy
// (nearly all saliency on one code) or that the binned form cannot bin.
//
// The whole wavefront takes the flagged groups (`flagged`, uniform per
// group) one at a time: the group's members stage its G weights and
// saliencies in LDS (`stage`, 2 G floats the wavefront no longer needs;
// load_h(hv) gives a member lane's 16 saliencies), and lane l evaluates clip
// k0 + l / P (P = G / 16) over part l % P of the group, its sums combined
// over the clip's P lanes with DPP, then an argmin over the clips across the
// wavefront.  The group's members receive the winner in `best` (the key in
// member 0 only).
template <int L, bool SYM, int QMAX, bool SPREAD, bool W_BF16, typename LoadH>
__device__ __forceinline__ void int_exact_wave(const IntParams& p, const WRegs<W_BF16>& wr, LoadH load_h,
                                               const IntRange& g, const float* s_alpha, const float* s_clip,
                                               int lane, bool flagged, float* stage, IntBest& best) {
  using M = Members<L, SPREAD>;
  constexpr int G = L * kIntN;
  constexpr int P = L;               // parts of 16 weights per group
  constexpr int CPW = 64 / P;        // clips per pass of the wavefront
  constexpr float kQmax = (float)QMAX;
  constexpr float kQmin = SYM ? -(float)QMAX : 0.0f;
  constexpr float kBeta = 0.5f * (float)QMAX;
  const int j = M::member(lane), slot = M::slot(lane);
  const int K = p.n_clips;
  uint64_t todo = __ballot(flagged && j == 0);  // member 0 of every flagged group
#pragma unroll 1
  while (todo != 0) {
    const int s_lane = __ffsll((unsigned long long)todo) - 1;
    todo &= todo - 1;
    const bool mine = slot == M::slot(s_lane);
    wave_lds_fence();  // earlier use of the stage by this wavefront is done
    if (mine) {
      float hv[kIntN];
      load_h(hv);
#pragma unroll
      for (int c = 0; c < kIntN / 4; c++) {
        *reinterpret_cast<float4*>(stage + j * kIntN + 4 * c) =
            make_float4(wr.get(4 * c), wr.get(4 * c + 1), wr.get(4 * c + 2), wr.get(4 * c + 3));
        *reinterpret_cast<float4*>(stage + G + j * kIntN + 4 * c) =
            make_float4(hv[4 * c], hv[4 * c + 1], hv[4 * c + 2], hv[4 * c + 3]);
      }
    }
    wave_lds_fence();
    // the group's range, from its member 0 (uniform from here on)
    IntRange gg;
    gg.mn = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, g.mn), s_lane));
    gg.mx = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, g.mx), s_lane));
    gg.c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, g.c), s_lane));
    gg.rho = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, g.rho), s_lane));
    gg.rrho = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, g.rrho), s_lane));
    gg.nc = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, g.nc), s_lane));
    gg.constant = false;
    // this lane's part of the group
    const int part = lane % P;
    float w[kIntN], h[kIntN];
#pragma unroll
    for (int c = 0; c < kIntN / 4; c++) {
      const float4 a = *reinterpret_cast<const float4*>(stage + part * kIntN + 4 * c);
      const float4 b = *reinterpret_cast<const float4*>(stage + G + part * kIntN + 4 * c);
      w[4 * c] = a.x; w[4 * c + 1] = a.y; w[4 * c + 2] = a.z; w[4 * c + 3] = a.w;
      h[4 * c] = b.x; h[4 * c + 1] = b.y; h[4 * c + 2] = b.z; h[4 * c + 3] = b.w;
    }
    double sh = 0.0, shw = 0.0;
#pragma unroll
    for (int i = 0; i < kIntN; i++) {
      sh += (double)h[i];
      shw += (double)h[i] * (double)w[i];
    }
    sh = run_sum<P>(sh);
    shw = run_sum<P>(shw);
    IntBest lb = int_best_init();
#pragma unroll 1
    for (int k0 = 0; k0 < K; k0 += CPW) {
      const int k = k0 + lane / P;
      const int kc = k < K ? k : K - 1;  // lanes past the last clip repeat it; never kept
      const float al = s_alpha[kc], f = s_clip[kc];
      // the codes and the fp64 forms are formed again in every pass (the
      // values are made opaque between passes), one weight at a time, so
      // that few registers are live
      auto fresh = [&]() {
#pragma unroll
        for (int i = 0; i < kIntN; i++) asm volatile("" : "+v"(w[i]), "+v"(h[i]));
      };
      auto code = [&](int i) {
        const float u = int_u<SYM>(w[i], gg);
        const float x = SYM ? u * al : __builtin_fmaf(u, al, kBeta);
        return (double)__builtin_amdgcn_fmed3f(__builtin_rintf(x), kQmin, kQmax);
      };
      double a, b = 0.0;
      if constexpr (SYM) {
        double sqq = 0.0, sqw = 0.0;
        fresh();
#pragma unroll
        for (int i = 0; i < kIntN; i++) {
          const double Q = code(i), H = (double)h[i];
          sqq += H * Q * Q;
          sqw += H * Q * (double)w[i];
          __builtin_amdgcn_sched_barrier(0);
        }
        sqq = run_sum<P>(sqq);
        sqw = run_sum<P>(sqw);
        a = (sqq == 0.0) ? (double)((f * gg.mx) / kQmax) : sqw / sqq;
      } else {
        const float fr = f * gg.rho;
        const float s_rtn = (2.0f * fr) / kQmax;
        if (sh == 0.0) {
          a = (double)s_rtn;
          b = (double)(gg.c - fr);
        } else {
          double shq = 0.0;
          fresh();
#pragma unroll
          for (int i = 0; i < kIntN; i++) {
            shq += (double)h[i] * code(i);
            __builtin_amdgcn_sched_barrier(0);
          }
          shq = run_sum<P>(shq);
          const double qbar = shq / sh, wbar = shw / sh;
          double sqq = 0.0, sqw = 0.0;
          fresh();
#pragma unroll
          for (int i = 0; i < kIntN; i++) {
            const double dq = code(i) - qbar, dw = (double)w[i] - wbar, H = (double)h[i];
            sqq += H * dq * dq;
            sqw += H * dq * dw;
            __builtin_amdgcn_sched_barrier(0);
          }
          sqq = run_sum<P>(sqq);
          sqw = run_sum<P>(sqw);
          a = (sqq <= 1e-12 * sh * (double)QMAX * (double)QMAX) ? (double)s_rtn : sqw / sqq;
          b = wbar - a * qbar;
        }
      }
      const float af = round_param((float)a, p.param_dtype);
      const float bf = SYM ? 0.0f : round_param((float)b, p.param_dtype);
      double sc = 0.0;
      fresh();
#pragma unroll
      for (int i = 0; i < kIntN; i++) {
        const double e = (double)af * code(i) + (double)bf - (double)w[i];
        sc += (double)h[i] * e * e;
        __builtin_amdgcn_sched_barrier(0);
      }
      sc = run_sum<P>(sc);
      const double key = make_key(sc, k);
      if (k < K && part == 0 && key < lb.key) {
        lb.key = key;
        lb.a = af;
        lb.b = bf;
        lb.err = (float)sc;
      }
    }
    // argmin over the clips (keys order by score, then by clip index)
    const double kmin = rows_min_f64(run_min_f64<16>(lb.key));
    const int win = __ffsll((unsigned long long)__ballot(lb.key == kmin)) - 1;
    const float wa = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lb.a), win));
    const float wb = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lb.b), win));
    const float we = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lb.err), win));
    if (mine) {
      best.key = j == 0 ? kmin : __longlong_as_double(0x7ff0000000000000ll);
      best.a = wa;
      best.b = wb;
      best.err = we;
    }
  }
}

// Fit (Eq. ridgefit) and score (Eq. fisher-obj) of clip k from its
// clip-dependent moments A0 = sum h q, A1 = sum h q^2, A2 = sum h q w
// (symmetric: A0 unused, scale-only fit); keeps the better candidate.
template <bool SYM, int QMAX>
__device__ __forceinline__ void int_fit_score(const IntParams& p, int k, float f, const IntRange& g,
                                              const IntMoments& mo, double A0, double A1, double A2,
                                              IntBest& best) {
  constexpr float kQmax = (float)QMAX;
  best.ill |= int_fit_ill<SYM, QMAX>(mo, A0, A1, A2);
  if constexpr (SYM) {
    // scale-only fit: s* = sum h q w / sum h q^2 (the RTN scale f m / Q
    // when sum h q^2 = 0); the score of r = s q is Svww + s (s A1 - 2 A2)
    const double a = (A1 == 0.0) ? (double)((f * g.mx) / kQmax) : div_f64(A2, A1, rcp_f64(A1));
    const float af = round_param((float)a, p.param_dtype);
    const double ad = (double)af;
    const double score = mo.Svww + ad * (ad * A1 - 2.0 * A2);
    best.ill |= int_score_ill(mo, ad, 0.0, (double)QMAX, 0.0, A1, A2, score);
    const double key = make_key(score, k);
    if (key < best.key) {
      best.key = key;
      best.a = af;
      best.b = 0.0f;
      best.err = (float)fmax(score, 0.0);
    }
  } else {
    const double Sv = mo.Sv, Svw = mo.Svw;
    const double D = Sv * A1 - A0 * A0;
    double a, b;
    if (Sv == 0.0 || D <= mo.thr) {
      // no saliency, or all of it on one code: the slope is undetermined
      // and the RTN step of this range is kept
      const float fr = f * g.rho;
      const float s_rtn = (2.0f * fr) / kQmax;
      a = (double)s_rtn;
      b = (Sv == 0.0) ? (double)(g.c - fr) : div_f64(Svw - a * A0, Sv, mo.rSv);
    } else {
      // quotients from v_rcp_f64 + Newton: within a few ulp of the IEEE
      // quotient, far below the fp32 rounding of (s, z) that follows
      a = div_f64(Sv * A2 - A0 * Svw, D, rcp_f64(D));
      b = div_f64(Svw - a * A0, Sv, mo.rSv);
    }
    // fp32, then the deployed precision: the candidate is scored with the
    // dequantiser that is emitted
    const float af = round_param((float)a, p.param_dtype), bf = round_param((float)b, p.param_dtype);
    const double ad = (double)af, bd = (double)bf;
    // Eq. fisher-obj of the emitted dequantiser, expanded in fp64
    const double score = mo.Svww + ad * (ad * A1 + 2.0 * bd * A0 - 2.0 * A2) + bd * (bd * Sv - 2.0 * Svw);
    best.ill |= int_score_ill(mo, ad, bd, (double)QMAX, A0, A1, A2, score);
    const double key = make_key(score, k);
    if (key < best.key) {
      best.key = key;
      best.a = af;
      best.b = bf;
      best.err = (float)fmax(score, 0.0);
    }
  }
}

// Argmin over the group's L lanes (ties to the lowest clip index), winner
// broadcast through `win` (this group's 4 floats of LDS), then the emit:
// codes of f*, r = fmaf(s, q, z) in W's dtype (or fp32 r), (s, z) and the
// optional diagnostics.
template <bool W_BF16, int BITS, int G, bool SYM, bool SPREAD = false>
__device__ __forceinline__ void int_finish(const IntParams& p, const IntMatrix& mtx, const WRegs<W_BF16>& wr,
                                           const IntRange& g, double Sv, const IntBest& best, const float* s_alpha,
                                           float* win, int j, int64_t gid, const WaveImage& im, bool active) {
  constexpr int L = G / kIntN;
  constexpr int P4 = int_stage_per<SPREAD, G, 4>(), P2 = int_stage_per<SPREAD, G, 2>();
  constexpr int QMAX = SYM ? (1 << (BITS - 1)) - 1 : (1 << BITS) - 1;
  constexpr float kQmax = (float)QMAX;
  constexpr float kQmin = SYM ? -(float)QMAX : 0.0f;
  constexpr float kBeta = 0.5f * (float)QMAX;

  const double gkey = Members<L, SPREAD>::min_f64(best.key);
  const int kstar = key_index(gkey);
  if (best.key == gkey) {  // exactly one lane of the group owns clip kstar
    win[0] = best.a;
    win[1] = best.b;
    win[2] = best.err;
  }
  wave_lds_fence();
  float a = win[0], b = win[1], errv = win[2];
  const float alpha = s_alpha[kstar];
  int kout = kstar;
  if (g.constant) {  // every code 0, z = w in the deployed precision (exact at fp32)
    a = 0.0f;
    b = SYM ? 0.0f : round_param(g.mn, p.param_dtype);  // symmetric: an all-zero group
    const double d = (double)b - (double)g.mn;
    errv = (float)(Sv * d * d);
    kout = 0;
  }

  // two chunks of 8 weights: codes and r of a chunk are formed and its r
  // staged before the next chunk, which keeps few values live at once.  The
  // positions u are formed again here from opaque copies of the range: the
  // same expression earlier in the kernel would otherwise be kept, 16 values
  // held in registers through everything in between.
  float rrho = g.rrho, nc = g.nc;
  asm volatile("" : "+v"(rrho), "+v"(nc));
  const bool r_bf16 = W_BF16 || p.r_bf16;
  if (mtx.r) wave_lds_fence();  // the stage's earlier use is done
  uint64_t bits = 0;  // this lane's 16 codes, code i at bits [BITS i, BITS i + BITS)
#pragma unroll
  for (int h = 0; h < 2; h++) {
    float r[8];
#pragma unroll
    for (int t = 0; t < 8; t++) {
      const int i = 8 * h + t;
      uint32_t qi;
      if constexpr (SYM) {
        const float ui = wr.get(i) * rrho;
        // + 0.0f turns a rounded -0 into +0, so a zero code gives r = s * (+0)
        float q = __builtin_amdgcn_fmed3f(__builtin_rintf(ui * alpha), kQmin, kQmax) + 0.0f;
        if (g.constant) q = 0.0f;
        qi = (uint32_t)(int)q & ((1u << BITS) - 1u);  // two's complement in BITS bits
        r[t] = a * q;
      } else {
        const float ui = __builtin_fmaf(wr.get(i), rrho, nc);
        float x = __builtin_fmaf(ui, alpha, kBeta);
        float q = __builtin_amdgcn_fmed3f(__builtin_rintf(x), 0.0f, kQmax);
        if (g.constant) q = 0.0f;
        qi = (uint32_t)q;
        r[t] = __builtin_fmaf(a, q, b);
      }
      bits |= (uint64_t)qi << (BITS * i);
    }
    if (mtx.r) {
      if (r_bf16) {
        wave_put<2, P2>(im, h, make_uint4(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]), pack_bf16x2(r[4], r[5]),
                                          pack_bf16x2(r[6], r[7])));
      } else {
        wave_put<4, P4>(im, 2 * h, make_uint4(as_u32(r[0]), as_u32(r[1]), as_u32(r[2]), as_u32(r[3])));
        wave_put<4, P4>(im, 2 * h + 1, make_uint4(as_u32(r[4]), as_u32(r[5]), as_u32(r[6]), as_u32(r[7])));
      }
    }
  }
  if (mtx.r) {
    if (r_bf16)
      wave_flush<2, P2>(im, mtx.r);
    else
      wave_flush<4, P4>(im, mtx.r);
  }
  // INT3: members 2i and 2i + 1 hold bits [96 i, 96 i + 96) of the group's
  // stream, three whole dwords; the even member needs the odd one's low bits
  uint32_t partner_lo = 0;
  if constexpr (BITS == 3) {
    partner_lo = SPREAD ? dpp_u32<kDppRor8>((uint32_t)bits) : dpp_u32<kDppXor1>((uint32_t)bits);
  }
  if (!active) return;
  if constexpr (BITS == 4) {
    *reinterpret_cast<uint2*>(mtx.codes + gid * (G / 2) + j * 8) = make_uint2((uint32_t)bits, (uint32_t)(bits >> 32));
  } else if constexpr (BITS == 2) {
    *reinterpret_cast<uint32_t*>(mtx.codes + gid * (G / 4) + j * 4) = (uint32_t)bits;
  } else {  // BITS == 3: lane j's 48 bits start at bit 48 j of the group's stream
    uint32_t* dst = reinterpret_cast<uint32_t*>(mtx.codes + gid * (3 * G / 8) + (j >> 1) * 12);
    if ((j & 1) == 0) {
      dst[0] = (uint32_t)bits;
      dst[1] = ((uint32_t)(bits >> 32) & 0xffffu) | (partner_lo << 16);
    } else {
      dst[2] = (uint32_t)(bits >> 16);
    }
  }
  if (j == 0) {
    mtx.scales[gid] = a;
    if (mtx.zeros) mtx.zeros[gid] = b;
    if (mtx.best_clip) mtx.best_clip[gid] = (uint8_t)kout;
    if (mtx.err) mtx.err[gid] = errv;
  }
}

}  // namespace quasar
