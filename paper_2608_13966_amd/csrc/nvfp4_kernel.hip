// nvfp4_kernel.hip -- QUASAR reconstruction for NVFP4 on gfx950 (Sec. 4.2).
//
// Tensor level: S_t = amax / (6 * 448) from the tensor absmax (not optimised).
// Per 16-element block: for every clip factor f the search scale f m / 6
// (m = block absmax) gives E2M1 codes; the block scale is fitted to the same
// saliency-weighted objective (scale only: s* = sum h q w / sum h q^2) and
// stored as the E4M3 value nearest to s*/S_t, which is the best E4M3 value
// because the objective is a parabola in the scale; the candidate with the
// lowest score is emitted.
//
// One lane owns one block: 16 weights in registers, no cross-lane reduction.
// Moments and score in fp64 (see int_kernel.hip for why).
#include "device_common.h"
#include "formats.h"
#include "quasar_internal.h"

namespace quasar {
namespace {

constexpr int N = 16;

template <bool W_BF16, int EMA, int KC>
__global__ __launch_bounds__(kThreads) void nvfp4_reconstruct_kernel(Nvfp4Params p) {
  __shared__ float s_c6[kMaxClips], s_clip[kMaxClips];
  const int tid = threadIdx.x;
  const int K = p.n_clips;
  if (tid < kMaxClips) {  // the host pads both tables to kMaxClips entries
    s_c6[tid] = p.c6[tid];
    s_clip[tid] = p.clip[tid];
  }
  __syncthreads();

  int64_t bid = (int64_t)blockIdx.x * kThreads + tid;
  const bool active = bid < p.n_blocks;
  if (!active) bid = p.n_blocks - 1;
  const int64_t e0 = bid * N;

  float w[N], v[N];
  load16<W_BF16>(p.W, e0, w);
  load16<false>(p.v, e0, v);
  if constexpr (EMA != 0) {
    float g[N];
    load16<EMA == 1>(p.g, e0, g);
#pragma unroll
    for (int i = 0; i < N; i++) {
      float t = g[i] * g[i];
      float u = p.omb2 * t;
      v[i] = __builtin_fmaf(p.beta2, v[i], u);
    }
    if (active) store16<false>(p.v, e0, v);
  }

  const float amax = __builtin_nontemporal_load(p.amax);
  const float st = amax / 2688.0f;  // 6 * 448
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < N; i++) m = fmaxf(m, fabsf(w[i]));
  const bool zero = (m == 0.0f) || (st == 0.0f);
  const float rm = 1.0f / m;
  float u[N];
#pragma unroll
  for (int i = 0; i < N; i++) u[i] = w[i] * rm;

  double Sww = 0.0;
#pragma unroll
  for (int i = 0; i < N; i++) {
    const double Wd = (double)w[i];
    Sww = __builtin_fma((double)v[i] * Wd, Wd, Sww);
  }
  const double st_d = (double)st;

  double best_key = __longlong_as_double(0x7ff0000000000000ll);
  float best_s = 0.0f;
  uint32_t best_e = 0;
  float best_err = 0.0f;

  for (int k0 = 0; k0 < K; k0 += KC) {
    float cs[KC];
#pragma unroll
    for (int kk = 0; kk < KC; kk++)
      cs[kk] = uniform_f32(s_c6[(k0 + kk) < kMaxClips ? (k0 + kk) : kMaxClips - 1]);
    double acc[KC][2];
#pragma unroll
    for (int kk = 0; kk < KC; kk++) acc[kk][0] = acc[kk][1] = 0.0;
#pragma unroll
    for (int i = 0; i < N; i++) {
      const double H = (double)v[i], Wd = (double)w[i];
#pragma unroll
      for (int kk = 0; kk < KC; kk++) {
        const double Q = (double)e2m1_round(u[i] * cs[kk]);
        const double HQ = H * Q;
        acc[kk][0] = __builtin_fma(HQ, Q, acc[kk][0]);
        acc[kk][1] = __builtin_fma(HQ, Wd, acc[kk][1]);
      }
    }
#pragma unroll
    for (int kk = 0; kk < KC; kk++) {
      const int k = k0 + kk;
      if (k < K) {
        const double Sqq = acc[kk][0], Sqw = acc[kk][1];
        const double sstar = (Sqq == 0.0) ? (double)s_clip[k] * (double)m / 6.0 : Sqw / Sqq;
        uint32_t ecode;
        const double ev = e4m3_round(sstar / st_d, &ecode);
        const float sblk = st * (float)ev;
        const double sb = (double)sblk;
        const double score = sb * (sb * Sqq - 2.0 * Sqw) + Sww;
        const double key = make_key(score, k);
        if (key < best_key) {
          best_key = key;
          best_s = sblk;
          best_e = ecode;
          best_err = (float)fmax(score, 0.0);
        }
      }
    }
  }

  int kstar = key_index(best_key);
  float cstar = s_c6[kstar];
  if (zero) {
    kstar = 0;
    best_s = 0.0f;
    best_e = 0;
    best_err = (float)Sww;
  }
  uint32_t lo = 0, hi = 0;
  float r[N];
#pragma unroll
  for (int i = 0; i < N; i++) {
    const float q = zero ? 0.0f : e2m1_round(u[i] * cstar);
    const uint32_t code = zero ? 0u : e2m1_code_of(q);
    if (i < 8)
      lo |= code << (4 * i);
    else
      hi |= code << (4 * (i - 8));
    // a zero code is +0 (the E2M1 rounding keeps the sign of y)
    r[i] = (code == 0u) ? 0.0f : best_s * q;
  }
  if (!active) return;
  if (p.r) store16<W_BF16>(p.r, e0, r);
  *reinterpret_cast<uint2*>(p.codes + bid * 8) = make_uint2(lo, hi);
  p.scales[bid] = (uint8_t)best_e;
  if (p.best_clip) p.best_clip[bid] = (uint8_t)kstar;
  if (p.err) p.err[bid] = best_err;
  if (bid == 0) p.tensor_scale[0] = st;
}

// ---- tensor absmax ----------------------------------------------------------
__global__ void absmax_clear_kernel(unsigned* ws) {
  if (threadIdx.x == 0 && blockIdx.x == 0) ws[0] = 0u;
}

template <bool W_BF16>
__global__ __launch_bounds__(kThreads) void absmax_kernel(const void* W, int64_t n16, unsigned* ws) {
  __shared__ float s_m[kThreads / 64];
  float m = 0.0f;
  for (int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x; c < n16; c += (int64_t)gridDim.x * kThreads) {
    float w[N];
    load16<W_BF16>(W, c * N, w);
#pragma unroll
    for (int i = 0; i < N; i++) m = fmaxf(m, fabsf(w[i]));
  }
  m = run_max<16>(m);
  m = fmaxf(m, __shfl_xor(m, 16, 64));
  m = fmaxf(m, __shfl_xor(m, 32, 64));
  if ((threadIdx.x & 63) == 0) s_m[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = s_m[0];
#pragma unroll
    for (int i = 1; i < kThreads / 64; i++) t = fmaxf(t, s_m[i]);
    // |w| >= 0: the fp32 bit patterns order like unsigned integers
    atomicMax(ws, __float_as_uint(t));
  }
}

template <bool W_BF16, int EMA>
hipError_t launch_kc(const Nvfp4Params& p, hipStream_t s) {
  const int64_t blocks = (p.n_blocks + kThreads - 1) / kThreads;
  if (p.n_clips > 8 && p.n_clips <= 12)
    hipLaunchKernelGGL((nvfp4_reconstruct_kernel<W_BF16, EMA, 12>), dim3((unsigned)blocks), dim3(kThreads), 0,
                       s, p);
  else
    hipLaunchKernelGGL((nvfp4_reconstruct_kernel<W_BF16, EMA, 8>), dim3((unsigned)blocks), dim3(kThreads), 0,
                       s, p);
  return hipGetLastError();
}

template <bool W_BF16>
hipError_t launch_e(const Nvfp4Params& p, int ema_mode, hipStream_t s) {
  switch (ema_mode) {
    case 1: return launch_kc<W_BF16, 1>(p, s);
    case 2: return launch_kc<W_BF16, 2>(p, s);
    default: return launch_kc<W_BF16, 0>(p, s);
  }
}

}  // namespace

hipError_t launch_nvfp4(const Nvfp4Params& p, bool w_bf16, int ema_mode, hipStream_t s) {
  return w_bf16 ? launch_e<true>(p, ema_mode, s) : launch_e<false>(p, ema_mode, s);
}

hipError_t launch_absmax(const void* W, bool w_bf16, int64_t n, unsigned* ws, hipStream_t s) {
  const int64_t n16 = n / N;
  int64_t blocks = (n16 + kThreads - 1) / kThreads;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(absmax_clear_kernel, dim3(1), dim3(64), 0, s, ws);
  if (w_bf16)
    hipLaunchKernelGGL(absmax_kernel<true>, dim3((unsigned)blocks), dim3(kThreads), 0, s, W, n16, ws);
  else
    hipLaunchKernelGGL(absmax_kernel<false>, dim3((unsigned)blocks), dim3(kThreads), 0, s, W, n16, ws);
  return hipGetLastError();
}

}  // namespace quasar
