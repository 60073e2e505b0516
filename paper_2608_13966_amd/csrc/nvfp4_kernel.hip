// nvfp4_kernel.hip -- QUASAR reconstruction for NVFP4 on gfx950 (Sec. 4.2).
//
// Tensor level: S_t = amax / (6 * 448) from the tensor absmax (not optimised).
// E2M1 rounding uses the gfx950 FP4 conversion instructions (round to nearest
// even, saturating at 6); the block scale is rounded to E4M3 with the gfx950
// FP8 conversion (round to nearest even, the input clamped to 448 first,
// since the conversion returns NaN from 464 up).  The GPU tests drive both
// through this kernel at the formats' midpoints, subnormals and saturation.
// Per 16-element block: for every clip factor f the search scale f m / 6
// (m = block absmax) gives E2M1 codes; the block scale is fitted to the same
// saliency-weighted objective (scale only: s* = sum h q w / sum h q^2) and
// stored as the E4M3 value nearest to s*/S_t, which is the best E4M3 value
// because the objective is a parabola in the scale; the candidate with the
// lowest score is emitted.
//
// One lane owns one block: 16 weights in registers, no cross-lane reduction.
// Moments and score in fp64 (see int_kernel.hip for why).
#include <cstring>

#include "device_common.h"
#include "quasar_internal.h"

namespace quasar {
namespace {

constexpr int N = 16;
typedef float f32x2 __attribute__((ext_vector_type(2)));

// E2M1 codes of (a, b) into byte `sel` of `old` (the other bytes kept), and
// the two values of byte `sel` back; sel must fold to a constant
__device__ __forceinline__ uint32_t fp4_put(uint32_t old, float a, float b, int sel) {
  switch (sel) {
    case 0: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, 1.0f, 0);
    case 1: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, 1.0f, 1);
    case 2: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, 1.0f, 2);
    default: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, 1.0f, 3);
  }
}
__device__ __forceinline__ f32x2 fp4_get(uint32_t pk, int sel) {
  switch (sel) {
    case 0: return __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pk, 1.0f, 0);
    case 1: return __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pk, 1.0f, 1);
    case 2: return __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pk, 1.0f, 2);
    default: return __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pk, 1.0f, 3);
  }
}

// E4M3 bytes of (a, b) into word `hi` of `old` (the other word kept), and the
// value of byte `sel`; hi and sel must fold to constants
__device__ __forceinline__ uint32_t fp8_put(uint32_t old, float a, float b, int hi) {
  return (uint32_t)(hi ? __builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, true)
                       : __builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, false));
}
__device__ __forceinline__ float fp8_get(uint32_t d, int sel) {
  switch (sel) {
    case 0: return __builtin_amdgcn_cvt_f32_fp8((int)d, 0);
    case 1: return __builtin_amdgcn_cvt_f32_fp8((int)d, 1);
    case 2: return __builtin_amdgcn_cvt_f32_fp8((int)d, 2);
    default: return __builtin_amdgcn_cvt_f32_fp8((int)d, 3);
  }
}

template <bool W_BF16, int EMA, int KC, bool MULTI>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu((KC > 8 || MULTI) ? 3 : 4)))
void nvfp4_reconstruct_kernel(Nvfp4Params p) {
  static_assert(KC % 4 == 0, "clips are converted four at a time");
  __shared__ float s_c6[kMaxClips], s_clip[kMaxClips];
  const int tid = threadIdx.x;
  const int K = p.n_clips;
  if (tid < kMaxClips) {  // the host pads both tables to kMaxClips entries
    s_c6[tid] = p.c6[tid];
    s_clip[tid] = p.clip[tid];
  }
  __syncthreads();

  // this workgroup's matrix (see int_kernel.hip)
  int64_t blk = blockIdx.x;
  struct {
    const void* W;
    float* v;
    const void* g;
    uint8_t* codes;
    uint8_t* scales;
    void* r;
    uint8_t* best_clip;
    float* err;
    float* tensor_scale;
    const float* amax;
    int64_t n_blocks;
    float* m;  // the fused AdamW step
    void* Wu;
    unsigned* amax_out;
  } mtx = {p.W, p.v, p.g, p.codes, p.scales, p.r, p.best_clip, p.err, p.tensor_scale, p.amax, p.n_blocks,
           p.m, p.Wu, p.amax_out};
  if (p.batch.n > 1) {
    const MatrixSlot& ms = batch_slot<Nvfp4Params>(blk);
    mtx = {ms.W, ms.v, ms.g, ms.codes, static_cast<uint8_t*>(ms.scales), ms.r, ms.best_clip, ms.err,
         ms.tensor_scale, ms.amax, ms.n_units, ms.m, ms.Wu, ms.amax_out};
  }
  int64_t bid = blk * kThreads + tid;
  const bool active = bid < mtx.n_blocks;
  if (!active) bid = mtx.n_blocks - 1;
  const int64_t e0 = bid * N;

  WRegs<W_BF16> wr;
  wr.load(mtx.W, e0);
  float v[N];
  load16<false>(mtx.v, e0, v);
  if constexpr (EMA == 1 || EMA == 2) {
    float g[N];
    load16<EMA == 1>(mtx.g, e0, g);
#pragma unroll
    for (int i = 0; i < N; i++) {
      float t = g[i] * g[i];
      float u = p.omb2 * t;
      v[i] = __builtin_fmaf(p.beta2, v[i], u);
    }
    if (active) store16<false>(mtx.v, e0, v);
  } else if constexpr (EMA >= 3) {
    // one AdamW step first (see int_kernel.hip)
    float g[N], m[N], w[N];
    load16<EMA == 3>(mtx.g, e0, g);
    load16<false>(mtx.m, e0, m);
#pragma unroll
    for (int i = 0; i < N; i++) w[i] = wr.get(i);
    adamw16(w, m, v, g, p.adam, p.beta2, p.omb2);
    wr.set(w);
    if (active) {
      store16<false>(mtx.v, e0, v);
      store16<false>(mtx.m, e0, m);
      wr.store(mtx.Wu, e0);
    }
  }
  if (p.weighting != 0) {  // h = v, v*v or 1 (uniform branch)
#pragma unroll
    for (int i = 0; i < N; i++) v[i] = weight_of(v[i], p.weighting);
  }

  const float amax = __builtin_nontemporal_load(mtx.amax);
  const float st = amax / 2688.0f;  // 6 * 448
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < N; i++) m = fmaxf(m, fabsf(wr.get(i)));
  const bool zero = (m == 0.0f) || (st == 0.0f);
  const float rm = 1.0f / m;
  float u[N];
#pragma unroll
  for (int i = 0; i < N; i++) u[i] = wr.get(i) * rm;

  double Sww = 0.0;  // sum h w^2, accumulated in the first pass
  // x of the search scale, used when no weight with saliency gets a non-zero
  // code: f * (m / 6) / S_t (like every x, it only picks an E4M3 neighbour)
  const float mx = m * (1.0f / 6.0f) * __builtin_amdgcn_rcpf(st);

  double best_key = __longlong_as_double(0x7ff0000000000000ll);
  uint32_t best_e = 0;

  // one pass over the clips when K <= KC (the per-weight values then die as
  // they are consumed), otherwise passes of KC
#pragma unroll 1
  for (int k0 = 0; k0 < (MULTI ? K : 1); k0 += KC) {
    float cs[KC], fs[KC];
#pragma unroll
    for (int kk = 0; kk < KC; kk++) {
      const int kt = (k0 + kk) < kMaxClips ? (k0 + kk) : kMaxClips - 1;
      cs[kk] = uniform_f32(s_c6[kt]);
      fs[kk] = uniform_f32(s_clip[kt]);
    }
    double acc[KC][2];
#pragma unroll
    for (int kk = 0; kk < KC; kk++) acc[kk][0] = acc[kk][1] = 0.0;
    // Clips kk .. kk+3 put their two codes in bytes 0..3 of pk, and all four
    // are read back from the finished dword (no zeroing, one live copy).
    uint32_t pk = 0u;
#pragma unroll
    for (int i = 0; i < N; i += 2) {
      float v0 = v[i], v1 = v[i + 1], w0 = wr.get(i), w1 = wr.get(i + 1);
      if (MULTI) asm volatile("" : "+v"(v0), "+v"(v1), "+v"(w0), "+v"(w1));  // not hoisted across passes
      const double H0 = (double)v0, W0 = (double)w0;
      const double H1 = (double)v1, W1 = (double)w1;
      if (k0 == 0) {
        Sww = __builtin_fma(H0 * W0, W0, Sww);
        Sww = __builtin_fma(H1 * W1, W1, Sww);
      }
#pragma unroll
      for (int k4 = 0; k4 < KC; k4 += 4) {
        // E2M1 round-to-nearest-even with saturation at 6 for two weights
        // (v_cvt_scalef32_pk_fp4_f32) and back to fp32
#pragma unroll
        for (int kk = k4; kk < k4 + 4; kk++) pk = fp4_put(pk, u[i] * cs[kk], u[i + 1] * cs[kk], kk & 3);
#pragma unroll
        for (int kk = k4; kk < k4 + 4; kk++) {
          const f32x2 qq = fp4_get(pk, kk & 3);
          const double Q0 = (double)qq[0], Q1 = (double)qq[1];
          const double HQ0 = H0 * Q0, HQ1 = H1 * Q1;
          acc[kk][0] = __builtin_fma(HQ0, Q0, acc[kk][0]);
          acc[kk][1] = __builtin_fma(HQ0, W0, acc[kk][1]);
          acc[kk][0] = __builtin_fma(HQ1, Q1, acc[kk][0]);
          acc[kk][1] = __builtin_fma(HQ1, W1, acc[kk][1]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // Branch-free on purpose: a clip-dependent branch here would let the
    // compiler sink each clip's moment accumulation into its own block and
    // serialise the clips (one 16-deep fp64 chain at a time).
    // The E4M3 bytes of clips kk, kk+1 are converted together and kept, four
    // to a dword, in eb[kk / 4].
    uint32_t eb[KC / 4];
#pragma unroll
    for (int kk = 0; kk < KC; kk += 2) {
      float xc[2];
#pragma unroll
      for (int t = 0; t < 2; t++) {
        const double Sqq = acc[kk + t][0], Sqw = acc[kk + t][1];
        // x = s*/S_t with s* = Sqw / Sqq (the search scale f m / 6 when no
        // weight with saliency has a non-zero code).  fp32 is enough: x only
        // picks an E4M3 neighbour, and its error (a few 1e-7 relative) can
        // flip that choice only next to a rounding midpoint.  x >= 0 (q has
        // the sign of w); the clamp to 448, the saturated value, keeps it
        // below 464, above which the conversion returns NaN.
        // One residual step after the reciprocal: a quotient that is exactly
        // an fp32 value (an E4M3 midpoint among them) comes out exactly.
        const float xn = (float)Sqw, xd = (float)Sqq * st;
        const float xrd = __builtin_amdgcn_rcpf(xd);
        const float xq = xn * xrd;
        const float xr = __builtin_fmaf(__builtin_fmaf(-xd, xq, xn), xrd, xq);
        // xr is formed for every clip and the zero case picked by a select:
        // as a branch (the compiler's choice for the reciprocal) it cost
        // exec-mask work per clip and kept 27 more registers live
        float xv = xr;
        asm volatile("" : "+v"(xv));
        xc[t] = __builtin_amdgcn_fmed3f((Sqq == 0.0) ? fs[kk + t] * mx : xv, 0.0f, 448.0f);
      }
      // nearest E4M3FN (RNE) of both
      eb[kk / 4] = fp8_put(kk % 4 == 0 ? __float_as_uint(xc[0]) : eb[kk / 4], xc[0], xc[1], (kk / 2) & 1);
#pragma unroll
      for (int t = 0; t < 2; t++) {
        const int k = k0 + kk + t;
        const double Sqq = acc[kk + t][0], Sqw = acc[kk + t][1];
        const double sb = (double)(st * fp8_get(eb[kk / 4], (kk + t) & 3));
        // sum h (sb q - w)^2 expanded: Sww + sb (sb Sqq - 2 Sqw)
        const double score = __builtin_fma(sb, __builtin_fma(sb, Sqq, -2.0 * Sqw), Sww);
        // keys order like the scores and keep the lowest index among equal
        // ones; padding clips repeat clip K-1 with a larger index
        best_key = min_key(best_key, make_key(score, k));
      }
    }
    // the winner's E4M3 byte, if it is a clip of this pass
    const int kb = key_index(best_key) - k0;
    if (kb >= 0 && kb < KC) {
      uint32_t d = eb[0];
#pragma unroll
      for (int t = 1; t < KC / 4; t++) d = (kb >= 4 * t) ? eb[t] : d;
      best_e = (d >> (8 * (kb & 3))) & 0xffu;
    }
  }

  int kstar = key_index(best_key);
  const float cstar = s_c6[kstar];
  float best_s = st * __builtin_amdgcn_cvt_f32_fp8((int)best_e, 0);
  float best_err = (float)__longlong_as_double(__double_as_longlong(best_key) & ~15ll);
  if (zero) {
    kstar = 0;
    best_s = 0.0f;
    best_e = 0;
    best_err = (float)Sww;
  }
  // codes of the winning clip: four pairs per dword, then zero magnitudes
  // get a clear sign bit (a zero code is +0)
  uint32_t cw[2] = {0u, 0u};
#define QUASAR_PUT(D, SEL)                                                                           \
  cw[D] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(cw[D], u[8 * D + 2 * SEL] * cstar,                \
                                                   u[8 * D + 2 * SEL + 1] * cstar, 1.0f, SEL)
  QUASAR_PUT(0, 0); QUASAR_PUT(0, 1); QUASAR_PUT(0, 2); QUASAR_PUT(0, 3);
  QUASAR_PUT(1, 0); QUASAR_PUT(1, 1); QUASAR_PUT(1, 2); QUASAR_PUT(1, 3);
#undef QUASAR_PUT
  float r[N];
#pragma unroll
  for (int d = 0; d < 2; d++) {
    const uint32_t mag = cw[d] & 0x77777777u;
    const uint32_t nz = (mag | (mag >> 1) | (mag >> 2)) & 0x11111111u;
    cw[d] = zero ? 0u : (mag | (cw[d] & (nz << 3)));
  }
#define QUASAR_GET(D, SEL)                                                            \
  {                                                                                   \
    const auto qq = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(cw[D], 1.0f, SEL);       \
    r[8 * D + 2 * SEL] = best_s * qq[0];                                              \
    r[8 * D + 2 * SEL + 1] = best_s * qq[1];                                          \
  }
  QUASAR_GET(0, 0) QUASAR_GET(0, 1) QUASAR_GET(0, 2) QUASAR_GET(0, 3)
  QUASAR_GET(1, 0) QUASAR_GET(1, 1) QUASAR_GET(1, 2) QUASAR_GET(1, 3)
#undef QUASAR_GET
  if constexpr (EMA >= 3) {
    // by-product of the fused step: max |W'| for the next step's tensor scale.
    // One atomic per wavefront, skipped when the stored maximum is already
    // larger (|w| >= 0, so fp32 bit patterns order like unsigned integers).
    // Lanes past the last block re-ran the step on a copy of the last block,
    // whose W its owner may already have updated in place: they contribute
    // nothing (|w| >= 0, so 0 is the identity of the maximum).
    if (mtx.amax_out) {
      float mw = run_max<16>(active ? m : 0.0f);
      mw = fmaxf(mw, __shfl_xor(mw, 16, 64));
      mw = fmaxf(mw, __shfl_xor(mw, 32, 64));
      if ((tid & 63) == 0 && __float_as_uint(mw) > __builtin_nontemporal_load(mtx.amax_out))
        atomicMax(mtx.amax_out, __float_as_uint(mw));
    }
  }
  if (!active) return;
  if (mtx.r) {
    if (W_BF16 || p.r_bf16)
      store16<true>(mtx.r, e0, r);
    else
      store16<false>(mtx.r, e0, r);
  }
  *reinterpret_cast<uint2*>(mtx.codes + bid * 8) = make_uint2(cw[0], cw[1]);
  mtx.scales[bid] = (uint8_t)best_e;
  if (mtx.best_clip) mtx.best_clip[bid] = (uint8_t)kstar;
  if (mtx.err) mtx.err[bid] = best_err;
  if (bid == 0) mtx.tensor_scale[0] = st;
}

// ---- tensor absmax ----------------------------------------------------------
__global__ void absmax_clear_kernel(unsigned* ws) {
  if (threadIdx.x == 0 && blockIdx.x == 0) ws[0] = 0u;
}

// every output of an absmax launch to 0 (a kernel, so that it may be captured)
__global__ void absmax_clear_all_kernel(AbsmaxTable t) {
#pragma unroll
  for (int i = 0; i < kMaxBatch; i++)
    if (i < t.n && threadIdx.x == 0) t.out[i][0] = 0u;
}

// max |x| over the 16-byte chunk t (8 bf16 or 4 fp32 values); NaNs are
// ignored, as by fmaxf
template <bool W_BF16>
__device__ __forceinline__ float chunk_absmax(uint4 t) {
  const uint32_t d[4] = {t.x, t.y, t.z, t.w};
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; k++) {
    if constexpr (W_BF16) {
      m = fmaxf(m, fmaxf(fabsf(as_f32(d[k] << 16)), fabsf(as_f32(d[k] & 0xffff0000u))));
    } else {
      m = fmaxf(m, fabsf(as_f32(d[k])));
    }
  }
  return m;
}

// One workgroup per span of kAbsChunks 16-byte chunks of one matrix: lane t
// loads chunks t, t + 256, ... (each load instruction reads 1 KB contiguous per
// wavefront), kAbsBatch loads in flight at a time; then a DPP / LDS maximum
// and at most one atomicMax on the fp32 bit pattern per workgroup.
constexpr int64_t kAbsChunks = (int64_t)kThreads * kAbsSpan;

template <bool W_BF16>
__global__ __launch_bounds__(kThreads) void absmax_kernel(AbsmaxTable t) {
  __shared__ float s_m[kThreads / 64];
  // the table is read from the kernel-argument segment (see batch_slot)
#if defined(__HIP_DEVICE_COMPILE__)
  const AbsmaxTable* kt = reinterpret_cast<const AbsmaxTable*>(__builtin_amdgcn_kernarg_segment_ptr());
#else
  const AbsmaxTable* kt = nullptr;
#endif
  int64_t blk = blockIdx.x;
  int mi = 0;
#pragma unroll 1
  while (mi + 1 < kt->n && blk >= kt->block0[mi + 1]) mi++;
  blk -= kt->block0[mi];
  const uint4* src = reinterpret_cast<const uint4*>(kt->W[mi]);
  const int64_t n_chunks = kt->n_chunks[mi];
  const int64_t c0 = blk * kAbsChunks + threadIdx.x;
  // batches of kAbsBatch loads in flight at a time
  float m = 0.0f;
#pragma unroll 1
  for (int b0 = 0; b0 < kAbsSpan; b0 += kAbsBatch) {
    uint4 buf[kAbsBatch];
#pragma unroll
    for (int u = 0; u < kAbsBatch; u++) {
      const int64_t c = c0 + (int64_t)(b0 + u) * kThreads;
      buf[u] = c < n_chunks ? src[c] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < kAbsBatch; u++) m = fmaxf(m, chunk_absmax<W_BF16>(buf[u]));
  }
  m = rows_max(run_max<16>(m));
  if ((threadIdx.x & 63) == 0) s_m[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    float x = s_m[0];
#pragma unroll
    for (int i = 1; i < kThreads / 64; i++) x = fmaxf(x, s_m[i]);
    // |w| >= 0: the fp32 bit patterns order like unsigned integers.  The
    // stored maximum only grows, so a workgroup whose maximum does not exceed
    // the value it reads skips its atomic (most do: the atomics on one
    // address otherwise serialise)
    if (__float_as_uint(x) > __builtin_nontemporal_load(kt->out[mi])) atomicMax(kt->out[mi], __float_as_uint(x));
  }
}

template <bool W_BF16, int EMA>
hipError_t launch_kc(const Nvfp4Params& p, hipStream_t s) {
  const int64_t blocks = p.batch.n > 1 ? p.batch.total_blocks : (p.n_blocks + kThreads - 1) / kThreads;
  const dim3 grid((unsigned)blocks), block(kThreads);
  const int K = p.n_clips;
  if (K <= 4)
    hipLaunchKernelGGL((nvfp4_reconstruct_kernel<W_BF16, EMA, 4, false>), grid, block, 0, s, p);
  else if (K <= 8)
    hipLaunchKernelGGL((nvfp4_reconstruct_kernel<W_BF16, EMA, 8, false>), grid, block, 0, s, p);
  else if (K <= 12)
    hipLaunchKernelGGL((nvfp4_reconstruct_kernel<W_BF16, EMA, 12, false>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((nvfp4_reconstruct_kernel<W_BF16, EMA, 8, true>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <bool W_BF16>
hipError_t launch_e(const Nvfp4Params& p, int ema_mode, hipStream_t s) {
  switch (ema_mode) {
    case 1: return launch_kc<W_BF16, 1>(p, s);
    case 2: return launch_kc<W_BF16, 2>(p, s);
    case 3: return launch_kc<W_BF16, 3>(p, s);
    case 4: return launch_kc<W_BF16, 4>(p, s);
    default: return launch_kc<W_BF16, 0>(p, s);
  }
}

}  // namespace

hipError_t launch_nvfp4(const Nvfp4Params& p, bool w_bf16, int ema_mode, hipStream_t s) {
  return w_bf16 ? launch_e<true>(p, ema_mode, s) : launch_e<false>(p, ema_mode, s);
}

hipError_t launch_clear(unsigned* ws, hipStream_t s) {
  hipLaunchKernelGGL(absmax_clear_kernel, dim3(1), dim3(64), 0, s, ws);
  return hipGetLastError();
}

hipError_t launch_clear_all(const AbsmaxTable& t, hipStream_t s) {
  hipLaunchKernelGGL(absmax_clear_all_kernel, dim3(1), dim3(64), 0, s, t);
  return hipGetLastError();
}

hipError_t launch_absmax(const AbsmaxTable& t, bool w_bf16, hipStream_t s) {
  hipLaunchKernelGGL(absmax_clear_all_kernel, dim3(1), dim3(64), 0, s, t);
  const dim3 grid((unsigned)t.block0[t.n]), block(kThreads);
  if (w_bf16)
    hipLaunchKernelGGL(absmax_kernel<true>, grid, block, 0, s, t);
  else
    hipLaunchKernelGGL(absmax_kernel<false>, grid, block, 0, s, t);
  return hipGetLastError();
}

hipError_t launch_absmax(const void* W, bool w_bf16, int64_t n, unsigned* ws, hipStream_t s) {
  AbsmaxTable t;
  memset(&t, 0, sizeof(t));
  t.n = 1;
  t.W[0] = W;
  t.out[0] = ws;
  // n is a multiple of 16 (whole NVFP4 blocks), so W is a whole number of
  // 16-byte chunks in either dtype
  t.n_chunks[0] = n / (w_bf16 ? 8 : 4);
  t.block0[1] = absmax_blocks(t.n_chunks[0]);
  return launch_absmax(t, w_bf16, s);
}

}  // namespace quasar
