// int_kernel.hip -- QUASAR reconstruction for INT-b groups on gfx950, the
// direct form: every candidate's moments are summed weight by weight.
//
// Algorithm 1 (Sec. 4.1.2) for every group of G weights along a row:
//   c, rho from the group's min/max; for each clip factor f: codes on
//   [c - f rho, c + f rho] (Eq. rtn), weighted least-squares (s, z) (Eq. ridgefit),
//   score sum h (s q + z - w)^2 (Eq. fisher-obj); emit the argmin.
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
// deterministic.  This form serves every shape and clip count; the binned form
// (int_cells_kernel.hip) replaces it where its tables fit.
#include <type_traits>

#include "device_common.h"
#include "int_common.h"
#include "quasar_internal.h"

namespace quasar {
namespace {

constexpr int N = kIntN;  // weights per lane

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

  // per wavefront: the moment transpose, the exact path's stage, the stage of
  // the coalesced stores.  The transpose holds group slot s, clip kk, member j
  // at s KC (L + 1) + kk (L + 1) + j: one pad word per clip row, so that the
  // reads (a lane's clip row, L + 1 words apart from its neighbours') and the
  // writes (a clip's row per slot) spread over all the banks
  constexpr int ROW = L + 1;
  constexpr int TRANS = GPW * KC * ROW;
  constexpr int RED = TRANS > int_stage_bytes<false, G>() / 8 ? TRANS : int_stage_bytes<false, G>() / 8;
  __shared__ __align__(16) double s_red[kThreads / 64][RED];
  __shared__ float s_alpha[kMaxClips], s_clip[kMaxClips];
  __shared__ float s_win[kThreads / 64][GPW][4];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_index();
  const int j = lane % L, slot = lane / L;
  const int K = p.n_clips;

  if (tid < kMaxClips) {  // the host pads both tables to kMaxClips entries
    s_alpha[tid] = p.alpha[tid];
    s_clip[tid] = p.clip[tid];
  }
  __syncthreads();

  int64_t blk = blockIdx.x;
  const IntMatrix mtx = int_matrix(p, blk);
  const int64_t wave_g0 = (blk * (kThreads / 64) + wave) * GPW;
  int64_t gid = wave_g0 + slot;
  const bool active = gid < mtx.n_groups;
  if (!active) gid = mtx.n_groups - 1;  // recompute the last group; nothing is stored
  const int64_t e0 = gid * G + (int64_t)j * N;
  double* red = s_red[wave];
  const WaveImage im = int_image<L>(red, wave_g0, mtx.n_groups, slot, j, lane);

  // W stays in its storage format in registers (bf16: 8 dwords) and is widened
  // on use, which keeps the kernel inside 128 VGPRs (4 waves per SIMD).
  WRegs<W_BF16> wr;
  float v[N];
  int_load<W_BF16, EMA, false, G>(p, mtx, im, e0, wr, v);
  const IntRange rg = int_range<L, SYM>(wr);

  // clip-independent moments (fp64), accumulated in the first pass
  // every moment is an fp64 sum of at most 20 exact products: no fixed-point
  // rounding, and fp64 rounding inside 2^-47 of the terms' magnitude
  IntMoments mo = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0x1p-47, (double)fmaxf(fabsf(rg.mn), fabsf(rg.mx)),
                   0.0, 0.0, 0.0};
  IntBest best = int_best_init();

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
      const float ui = int_u<SYM>(wi, rg);
      const double V = (double)vi, Wd = (double)wi;
      const double VW = V * Wd;
      if constexpr (FIRST) {
        mo.Sv += V;
        mo.Svw += VW;
        mo.Svww = __builtin_fma(VW, Wd, mo.Svww);
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
      mo.Sv = run_sum<L>(mo.Sv);
      mo.Svw = run_sum<L>(mo.Svw);
      mo.Svww = run_sum<L>(mo.Svww);
      mo.thr = 1e-12 * mo.Sv * mo.Sv * (double)QMAX * (double)QMAX;
      mo.rSv = rcp_f64(mo.Sv);
      int_fit_bounds<QMAX>(mo);
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
      for (int kk = 0; kk < KC; kk++) red[(slot * KC + kk) * ROW + j] = acc[kk][m];
      wave_lds_fence();
#pragma unroll
      for (int t = 0; t < OWN; t++) {
        const int kk = j + L * t;
        const int kr = kk < KC ? kk : KC - 1;
        double s = 0.0;
#pragma unroll
        for (int jj = 0; jj < L; jj++) s += red[(slot * KC + kr) * ROW + jj];
        own[t][m] = s;
      }
      wave_lds_fence();
    }

    // ---- solve the owned clips (Eq. ridgefit) and score them ----------------
#pragma unroll
    for (int t = 0; t < OWN; t++) {
      const int kk = j + L * t;
      const int k = k0 + kk;
      if (kk < KC && k < K) int_fit_score<SYM, QMAX>(p, k, s_clip[k], rg, mo, own[t][0], own[t][1], own[t][2], best);
    }
  };
  pass(0, std::true_type{});
  if constexpr (MULTI) {
#pragma unroll 1
    for (int k0 = KC; k0 < K; k0 += KC) pass(k0, std::false_type{});
  }

  // a group whose fit the moments cannot fix accurately enough: every clip
  // again, straight from the weights
  {
    auto load_h = [&](float (&hv)[N]) {
#pragma unroll
      for (int i = 0; i < N; i++) hv[i] = v[i];
    };
    const bool ill = run_max<L>(best.ill ? 1.0f : 0.0f) > 0.0f;
    int_exact_wave<L, SYM, QMAX, false, W_BF16>(p, wr, load_h, rg, s_alpha, s_clip, lane,
                                                ill && active && !rg.constant, reinterpret_cast<float*>(red), best);
  }

  int_finish<W_BF16, BITS, G, SYM>(p, mtx, wr, rg, mo.Sv, best, s_alpha, s_win[wave][slot], j, gid, im, active);
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
  if (p.cells.n_cells > 0) return launch_int_cells(p, bits, group, w_bf16, ema_mode, s);
  return w_bf16 ? launch_e<true>(p, bits, group, ema_mode, s) : launch_e<false>(p, bits, group, ema_mode, s);
}

}  // namespace quasar
