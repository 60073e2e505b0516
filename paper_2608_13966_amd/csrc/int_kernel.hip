// int_kernel.hip -- QUASAR reconstruction for asymmetric INT-b groups on gfx950.
//
// Algorithm 1 (Sec. 4.1.2) for every group of G weights along a row:
//   c, rho from the group's min/max; for each clip factor f: codes on
//   [c - f rho, c + f rho] (Eq. rtn), weighted least-squares (s, z) (Eq. ridgefit),
//   score sum h (s q + z - w)^2 (Eq. fisher-obj); emit the argmin.
//
// Work decomposition: a group is owned by L = G/16 consecutive lanes of one
// wavefront, each holding 16 consecutive weights in registers (G = 128: 8 lanes,
// G = 64: 4 lanes); a wavefront processes 64/L groups.  W, v (and g) are read
// from HBM exactly once with 128-bit loads; codes, r, v' are written once.
//
// Per weight and clip: fp32 code (fma, rint, clamp -- the same fp32 recipe as
// the oracle, so codes are bit-identical) and three fp64 moments
// (sum v q, sum v q^2, sum v q w).  fp64 keeps the 2x2 normal equations and the
// expanded score exact enough to reproduce the argmin under heavy-tailed
// saliency (the weighted code variance can be 1e-4 of its mean square).
// Moments are combined across the L lanes through LDS (a transpose: each lane
// sums the partials of the clips it owns), the owner solves its clips, and an
// argmin over keys (score with the clip index in the low bits) picks the winner
// with DPP.  No atomics; every result has a single owner, so runs are
// deterministic.
#include <type_traits>

#include "device_common.h"
#include "quasar_internal.h"

namespace quasar {
namespace {

constexpr int N = 16;  // weights per lane

// SYM: symmetric groups (r = s q, q in [-Q, Q], Q = 2^(BITS-1) - 1, range
// [-f m, f m] with m = max |w|, scale-only fit); otherwise asymmetric groups
// (r = s q + z, q in [0, 2^BITS - 1], range [c - f rho, c + f rho]).
template <bool W_BF16, int EMA, int BITS, int G, int KC, bool MULTI, bool SYM>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu((KC > 8 || MULTI) ? 3 : 4)))
void int_reconstruct_kernel(IntParams p) {
  constexpr int L = G / N;          // lanes per group
  constexpr int GPW = 64 / L;       // groups per wavefront
  constexpr int QMAX = SYM ? (1 << (BITS - 1)) - 1 : (1 << BITS) - 1;
  constexpr int OWN = (KC + L - 1) / L;  // clips owned per lane per chunk
  constexpr int NM = SYM ? 2 : 3;        // clip-dependent moments
  constexpr float kQmax = (float)QMAX;
  constexpr float kQmin = SYM ? -(float)QMAX : 0.0f;
  constexpr float kBeta = 0.5f * (float)QMAX;

  __shared__ double s_red[kThreads / 64][64 * KC];
  __shared__ float s_alpha[kMaxClips], s_clip[kMaxClips];
  __shared__ float s_win[kThreads / 64][GPW][4];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int j = lane % L, slot = lane / L;
  const int K = p.n_clips;

  if (tid < kMaxClips) {  // the host pads both tables to kMaxClips entries
    s_alpha[tid] = p.alpha[tid];
    s_clip[tid] = p.clip[tid];
  }
  __syncthreads();

  // this workgroup's matrix: the call's own, or in a batched launch the slot
  // it falls in (uniform); the parameter block itself is only read
  int64_t blk = blockIdx.x;
  struct {
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
  } mtx = {p.W, p.v, p.g, p.codes, p.scales, p.zeros, p.r, p.best_clip, p.err, p.n_groups};
  if (p.batch.n > 1) {
    const MatrixSlot& ms = batch_slot<IntParams>(blk);
    mtx = {ms.W, ms.v, ms.g, ms.codes, static_cast<float*>(ms.scales), ms.zeros, ms.r, ms.best_clip, ms.err,
         ms.n_units};
  }
  int64_t gid = (blk * (kThreads / 64) + wave) * GPW + slot;
  const bool active = gid < mtx.n_groups;
  if (!active) gid = mtx.n_groups - 1;  // recompute the last group; nothing is stored
  const int64_t e0 = gid * G + (int64_t)j * N;

  // ---- load (each byte of W, v, g once) ------------------------------------
  // W stays in its storage format in registers (bf16: 8 dwords) and is widened
  // on use, which keeps the kernel inside 128 VGPRs (4 waves per SIMD).
  WRegs<W_BF16> wr;
  wr.load(mtx.W, e0);
  float v[N];
  load16<false>(mtx.v, e0, v);
  if constexpr (EMA == 1 || EMA == 2) {
    float g[N];
    load16<EMA == 1>(mtx.g, e0, g);
#pragma unroll
    for (int i = 0; i < N; i++) {
      // v' = beta2 v + (1 - beta2) g^2 in the oracle's fp32 order
      float t = g[i] * g[i];
      float u = p.omb2 * t;
      v[i] = __builtin_fmaf(p.beta2, v[i], u);
    }
    if (active) store16<false>(mtx.v, e0, v);
  } else if constexpr (EMA >= 3) {
    // one AdamW step first; the updated W is reconstructed and the updated
    // second moment is the saliency
    float g[N], m[N], w[N];
    load16<EMA == 3>(mtx.g, e0, g);
    load16<false>(p.m, e0, m);
#pragma unroll
    for (int i = 0; i < N; i++) w[i] = wr.get(i);
    adamw16(w, m, v, g, p.adam, p.beta2, p.omb2);
    wr.set(w);  // bf16 W: rounded here, and the rounded value is reconstructed
    if (active) {
      store16<false>(mtx.v, e0, v);
      store16<false>(p.m, e0, m);
      wr.store(p.Wu, e0);
    }
  }
  // saliency weighting (uniform branch): h = v, v*v (App. A.3) or 1 (Table 5)
  if (p.weighting != 0) {
#pragma unroll
    for (int i = 0; i < N; i++) v[i] = weight_of(v[i], p.weighting);
  }

  // ---- group range (Alg. 1, first line) ------------------------------------
  float mn, mx, c, rho, rrho, nc;
  bool constant;
  if constexpr (SYM) {  // m = max |w|
    mx = 0.0f;
#pragma unroll
    for (int i = 0; i < N; i++) mx = fmaxf(mx, fabsf(wr.get(i)));
    mx = run_max<L>(mx);
    mn = 0.0f;
    constant = (mx == 0.0f);  // an all-zero group
    c = 0.0f;
    rho = mx;
    rrho = 1.0f / mx;
    nc = 0.0f;
  } else {
    mn = wr.get(0);
    mx = wr.get(0);
#pragma unroll
    for (int i = 1; i < N; i++) {
      mn = fminf(mn, wr.get(i));
      mx = fmaxf(mx, wr.get(i));
    }
    mn = run_min<L>(mn);
    mx = run_max<L>(mx);
    constant = (mx == mn);
    c = 0.5f * (mx + mn);
    rho = 0.5f * (mx - mn);
    rrho = 1.0f / rho;
    nc = -(c * rrho);
  }
  // normalised position, recomputed where used: u = fmaf(w, 1/rho, -c/rho)
  // and x = fmaf(u, alpha_f, qmax/2) (symmetric: u = w * (1/m), x = u * alpha_f),
  // then q = clamp(rint(x))

  // ---- clip-independent moments (fp64), accumulated in the first pass --------
  double Sv = 0.0, Svw = 0.0, Svww = 0.0;
  double best_key = __longlong_as_double(0x7ff0000000000000ll);  // +inf
  float best_a = 0.f, best_b = 0.f, best_err = 0.f;
  double thr = 0.0, rSv = 0.0;
  double* red = s_red[wave];

  // One pass over the lane's 16 weights for clips k0 .. k0+KC-1 (entries past
  // the last clip repeat it and are never selected).
  auto pass = [&](const int k0, auto first_tag) {
    constexpr bool FIRST = decltype(first_tag)::value;
    float al[KC];
#pragma unroll
    for (int kk = 0; kk < KC; kk++)
      al[kk] = uniform_f32(s_alpha[(k0 + kk) < kMaxClips ? (k0 + kk) : kMaxClips - 1]);

    double acc[KC][3];
#pragma unroll
    for (int kk = 0; kk < KC; kk++) acc[kk][0] = acc[kk][1] = acc[kk][2] = 0.0;

#pragma unroll
    for (int i = 0; i < N; i++) {
      float vi = v[i], wi = wr.get(i);
      if constexpr (!FIRST) {
        // keep the per-weight fp64 values inside this pass (not hoisted and
        // held across passes)
        asm volatile("" : "+v"(vi), "+v"(wi));
      }
      const float ui = SYM ? wi * rrho : __builtin_fmaf(wi, rrho, nc);
      const double V = (double)vi, Wd = (double)wi;
      const double VW = V * Wd;
      if constexpr (FIRST) {
        Sv += V;
        Svw += VW;
        Svww = __builtin_fma(VW, Wd, Svww);
      }
#pragma unroll
      for (int kk = 0; kk < KC; kk++) {
        float x = SYM ? ui * al[kk] : __builtin_fmaf(ui, al[kk], kBeta);
        float q = __builtin_rintf(x);
        q = __builtin_amdgcn_fmed3f(q, kQmin, kQmax);
        const double Q = (double)q;
        const double VQ = V * Q;
        if constexpr (!SYM) acc[kk][0] += VQ;
        acc[kk][1] = __builtin_fma(VQ, Q, acc[kk][1]);
        acc[kk][2] = __builtin_fma(VW, Q, acc[kk][2]);
      }
      // one weight at a time: interleaving weights buys no latency hiding that
      // the other wavefronts on the SIMD do not already give, and costs VGPRs
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (FIRST) {
      Sv = run_sum<L>(Sv);
      Svw = run_sum<L>(Svw);
      Svww = run_sum<L>(Svww);
      thr = 1e-12 * Sv * Sv * (double)QMAX * (double)QMAX;
      rSv = rcp_f64(Sv);
    }

    // ---- combine the L partials: lane j sums the clips kk = j + L t ---------
    double own[OWN][3];
    if constexpr (SYM) {
#pragma unroll
      for (int t = 0; t < OWN; t++) own[t][0] = 0.0;
    }
#pragma unroll
    for (int m = 3 - NM; m < 3; m++) {
#pragma unroll
      for (int kk = 0; kk < KC; kk++) red[(slot * KC + kk) * L + j] = acc[kk][m];
      wave_lds_fence();
#pragma unroll
      for (int t = 0; t < OWN; t++) {
        const int kk = j + L * t;
        const int kr = kk < KC ? kk : KC - 1;
        double s = 0.0;
#pragma unroll
        for (int jj = 0; jj < L; jj++) s += red[(slot * KC + kr) * L + jj];
        own[t][m] = s;
      }
      wave_lds_fence();
    }

    // ---- solve the owned clips (Eq. ridgefit) and score them ----------------
#pragma unroll
    for (int t = 0; t < OWN; t++) {
      const int kk = j + L * t;
      const int k = k0 + kk;
      if (SYM && kk < KC && k < K) {
        // scale-only fit: s* = sum h q w / sum h q^2 (the RTN scale f m / Q
        // when sum h q^2 = 0); the score of r = s q is Svww + s (s A1 - 2 A2)
        const double A1 = own[t][1], A2 = own[t][2];
        const double a = (A1 == 0.0) ? (double)((s_clip[k] * mx) / kQmax) : div_f64(A2, A1, rcp_f64(A1));
        const float af = round_param((float)a, p.param_dtype);
        const double ad = (double)af;
        const double score = Svww + ad * (ad * A1 - 2.0 * A2);
        const double key = make_key(score, k);
        if (key < best_key) {
          best_key = key;
          best_a = af;
          best_b = 0.0f;
          best_err = (float)fmax(score, 0.0);
        }
      } else if (kk < KC && k < K) {
        const double A0 = own[t][0], A1 = own[t][1], A2 = own[t][2];
        const double D = Sv * A1 - A0 * A0;
        double a, b;
        if (Sv == 0.0 || D <= thr) {
          // no saliency, or all of it on one code: the slope is undetermined
          // and the RTN step of this range is kept
          const float f = s_clip[k];
          const float fr = f * rho;
          const float s_rtn = (2.0f * fr) / kQmax;
          a = (double)s_rtn;
          b = (Sv == 0.0) ? (double)(c - fr) : div_f64(Svw - a * A0, Sv, rSv);
        } else {
          // quotients from v_rcp_f64 + Newton: within a few ulp of the IEEE
          // quotient, far below the fp32 rounding of (s, z) that follows
          a = div_f64(Sv * A2 - A0 * Svw, D, rcp_f64(D));
          b = div_f64(Svw - a * A0, Sv, rSv);
        }
        // fp32, then the deployed precision: the candidate is scored with
        // the dequantiser that is emitted
        const float af = round_param((float)a, p.param_dtype), bf = round_param((float)b, p.param_dtype);
        const double ad = (double)af, bd = (double)bf;
        // Eq. fisher-obj of the emitted dequantiser, expanded in fp64
        const double score =
            Svww + ad * (ad * A1 + 2.0 * bd * A0 - 2.0 * A2) + bd * (bd * Sv - 2.0 * Svw);
        const double key = make_key(score, k);
        if (key < best_key) {
          best_key = key;
          best_a = af;
          best_b = bf;
          best_err = (float)fmax(score, 0.0);
        }
      }
    }
  };
  pass(0, std::true_type{});
  if constexpr (MULTI) {
#pragma unroll 1
    for (int k0 = KC; k0 < K; k0 += KC) pass(k0, std::false_type{});
  }

  // ---- argmin over the group's lanes, winner broadcast -----------------------
  const double gkey = run_min_f64<L>(best_key);
  const int kstar = key_index(gkey);
  float* win = s_win[wave][slot];
  if (best_key == gkey) {  // exactly one lane of the group owns clip kstar
    win[0] = best_a;
    win[1] = best_b;
    win[2] = best_err;
  }
  wave_lds_fence();
  float a = win[0], b = win[1], errv = win[2];
  const float alpha = s_alpha[kstar];
  int kout = kstar;
  if (constant) {  // every code 0, z = w in the deployed precision (exact at fp32)
    a = 0.0f;
    b = SYM ? 0.0f : round_param(mn, p.param_dtype);  // symmetric: an all-zero group
    const double d = (double)b - (double)mn;
    errv = (float)(Sv * d * d);
    kout = 0;
  }

  // ---- emit: codes of f*, r = fmaf(s, q, z) ---------------------------------
  uint32_t qi[N];
  float r[N];
#pragma unroll
  for (int i = 0; i < N; i++) {
    if constexpr (SYM) {
      const float ui = wr.get(i) * rrho;
      // + 0.0f turns a rounded -0 into +0, so a zero code gives r = s * (+0)
      float q = __builtin_amdgcn_fmed3f(__builtin_rintf(ui * alpha), kQmin, kQmax) + 0.0f;
      if (constant) q = 0.0f;
      qi[i] = (uint32_t)(int)q & ((1u << BITS) - 1u);  // two's complement in BITS bits
      r[i] = a * q;
    } else {
      const float ui = __builtin_fmaf(wr.get(i), rrho, nc);
      float x = __builtin_fmaf(ui, alpha, kBeta);
      float q = __builtin_amdgcn_fmed3f(__builtin_rintf(x), 0.0f, kQmax);
      if (constant) q = 0.0f;
      qi[i] = (uint32_t)q;
      r[i] = __builtin_fmaf(a, q, b);
    }
  }
  if (!active) return;
  if (mtx.r) {
    if (W_BF16 || p.r_bf16)
      store16<true>(mtx.r, e0, r);
    else
      store16<false>(mtx.r, e0, r);
  }
  if constexpr (BITS == 4) {
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int i = 0; i < 8; i++) {
      lo |= qi[i] << (4 * i);
      hi |= qi[8 + i] << (4 * i);
    }
    *reinterpret_cast<uint2*>(mtx.codes + gid * (G / 2) + j * 8) = make_uint2(lo, hi);
  } else if constexpr (BITS == 2) {
    uint32_t x = 0;
#pragma unroll
    for (int i = 0; i < N; i++) x |= qi[i] << (2 * i);
    *reinterpret_cast<uint32_t*>(mtx.codes + gid * (G / 4) + j * 4) = x;
  } else {  // BITS == 3: 48 bits per lane at byte offset 6 j of the group's stream
    uint64_t x = 0;
#pragma unroll
    for (int i = 0; i < N; i++) x |= (uint64_t)qi[i] << (3 * i);
    uint16_t* dst = reinterpret_cast<uint16_t*>(mtx.codes + gid * (3 * G / 8) + j * 6);
    dst[0] = (uint16_t)x;
    dst[1] = (uint16_t)(x >> 16);
    dst[2] = (uint16_t)(x >> 32);
  }
  if (j == 0) {
    mtx.scales[gid] = a;
    if (mtx.zeros) mtx.zeros[gid] = b;
    if (mtx.best_clip) mtx.best_clip[gid] = (uint8_t)kout;
    if (mtx.err) mtx.err[gid] = errv;
  }
}

template <bool W_BF16, int EMA, int BITS, int G>
hipError_t launch_kc(const IntParams& p, hipStream_t s) {
  constexpr int64_t groups_per_block = int_units_per_block(G);
  const int64_t blocks =
      p.batch.n > 1 ? p.batch.total_blocks : (p.n_groups + groups_per_block - 1) / groups_per_block;
  // clips per pass: one pass of 4, 8 or 12 clips when K <= 12 (entries past K
  // repeat the last clip and are never selected); passes of 8 beyond that
  const int K = p.n_clips;
  const dim3 grid((unsigned)blocks), block(kThreads);
  if (p.symmetric) {  // symmetric groups: passes of 8 or 12; not fused with the optimiser step
    if constexpr (EMA <= 2) {
      if (K <= 8)
        hipLaunchKernelGGL((int_reconstruct_kernel<W_BF16, EMA, BITS, G, 8, false, true>), grid, block, 0, s, p);
      else if (K <= 12)
        hipLaunchKernelGGL((int_reconstruct_kernel<W_BF16, EMA, BITS, G, 12, false, true>), grid, block, 0, s, p);
      else
        hipLaunchKernelGGL((int_reconstruct_kernel<W_BF16, EMA, BITS, G, 8, true, true>), grid, block, 0, s, p);
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  if (K <= 4)
    hipLaunchKernelGGL((int_reconstruct_kernel<W_BF16, EMA, BITS, G, 4, false, false>), grid, block, 0, s, p);
  else if (K <= 8)
    hipLaunchKernelGGL((int_reconstruct_kernel<W_BF16, EMA, BITS, G, 8, false, false>), grid, block, 0, s, p);
  else if (K <= 12)
    hipLaunchKernelGGL((int_reconstruct_kernel<W_BF16, EMA, BITS, G, 12, false, false>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((int_reconstruct_kernel<W_BF16, EMA, BITS, G, 8, true, false>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <bool W_BF16, int EMA, int BITS>
hipError_t launch_g(const IntParams& p, int group, hipStream_t s) {
  return group == 64 ? launch_kc<W_BF16, EMA, BITS, 64>(p, s) : launch_kc<W_BF16, EMA, BITS, 128>(p, s);
}

template <bool W_BF16, int EMA>
hipError_t launch_b(const IntParams& p, int bits, int group, hipStream_t s) {
  switch (bits) {
    case 2: return launch_g<W_BF16, EMA, 2>(p, group, s);
    case 3: return launch_g<W_BF16, EMA, 3>(p, group, s);
    default: return launch_g<W_BF16, EMA, 4>(p, group, s);
  }
}

template <bool W_BF16>
hipError_t launch_e(const IntParams& p, int bits, int group, int ema_mode, hipStream_t s) {
  switch (ema_mode) {
    case 1: return launch_b<W_BF16, 1>(p, bits, group, s);
    case 2: return launch_b<W_BF16, 2>(p, bits, group, s);
    case 3: return launch_b<W_BF16, 3>(p, bits, group, s);
    case 4: return launch_b<W_BF16, 4>(p, bits, group, s);
    default: return launch_b<W_BF16, 0>(p, bits, group, s);
  }
}

}  // namespace

hipError_t launch_int(const IntParams& p, int bits, int group, bool w_bf16, int ema_mode, hipStream_t s) {
  return w_bf16 ? launch_e<true>(p, bits, group, ema_mode, s) : launch_e<false>(p, bits, group, ema_mode, s);
}

}  // namespace quasar
