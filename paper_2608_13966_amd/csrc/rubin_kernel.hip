// rubin_kernel.hip -- QUASAR for the Rubin INT3 lookup-table format on gfx950
// (App. B, Eq. rubin-fit).
//
// A block is 8 rows x 64 columns (512 weights) with 3-bit indices and an
// 8-entry E4M3 codebook.  For every clip factor f the indices are the INT3
// codes of the range [c - f rho, c + f rho] (the same fp32 recipe as the
// affine kernel), each codebook entry is the saliency-weighted mean of the
// weights with that index rounded to E4M3, and the candidate is scored with
// Eq. fisher-obj; the lowest score is emitted.
//
// Work decomposition: one wavefront per block, lane l holding row l/8 of the
// block and its 8 consecutive columns 8 (l % 8) .. 8 (l % 8) + 7.  The
// per-index sums (sum h, sum h w) cannot be kept in registers (an element's
// index selects one of 8 accumulators), so every lane accumulates into its own
// 8 bins in LDS -- laid out [index][lane] so that a wavefront access touches
// consecutive 16-byte slots -- and the wavefront then reduces the 64 lanes'
// bins in two LDS stages.  No atomics: results are deterministic.
#include "device_common.h"
#include "quasar_internal.h"

namespace quasar {
namespace {

constexpr int NE = 8;          // weights per lane
constexpr int kWaves = kThreads / 64;

struct alignas(16) Bin {  // one 128-bit LDS access
  double h, hw;
};

// E4M3 byte of x (nearest even, |x| clamped to 448 first: the conversion
// gives NaN above 464), +0 for a zero result.
__device__ __forceinline__ uint32_t e4m3_byte(float x) {
  x = fminf(fmaxf(x, -448.0f), 448.0f);
  uint32_t e = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x, 0.0f, 0, false) & 0xffu;
  return e == 0x80u ? 0u : e;
}
__device__ __forceinline__ float e4m3_value(uint32_t e) { return __builtin_amdgcn_cvt_f32_fp8((int)e, 0); }

template <bool W_BF16, int EMA>
__global__ __launch_bounds__(kThreads) void rubin_reconstruct_kernel(RubinParams p) {
  __shared__ Bin s_bins[kWaves][8][64];      // [wave][index][lane]
  __shared__ Bin s_part[kWaves][8][8];       // [wave][lane group][index]
  __shared__ float s_lut[kWaves][8];
  __shared__ float s_alpha[kMaxClips], s_clip[kMaxClips];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int K = p.n_clips;
  if (tid < kMaxClips) {
    s_alpha[tid] = p.alpha[tid];
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
    uint8_t* lut;
    void* r;
    uint8_t* best_clip;
    float* err;
    int64_t n_blocks, cols, blocks_per_row;
  } mtx = {p.W, p.v, p.g, p.codes, p.lut, p.r, p.best_clip, p.err, p.n_blocks, p.cols, p.blocks_per_row};
  if (p.batch.n > 1) {
    const MatrixSlot& ms = batch_slot<RubinParams>(blk);
    mtx = {ms.W, ms.v, ms.g, ms.codes, static_cast<uint8_t*>(ms.scales), ms.r, ms.best_clip, ms.err, ms.n_units,
         ms.cols, ms.blocks_per_row};
  }
  int64_t bid = blk * kWaves + wave;
  const bool active = bid < mtx.n_blocks;  // uniform per wavefront
  if (!active) return;                   // no block-wide barrier follows
  const int64_t rb = bid / mtx.blocks_per_row, cb = bid - rb * mtx.blocks_per_row;
  const int64_t e0 = (rb * 8 + (lane >> 3)) * mtx.cols + cb * 64 + (lane & 7) * NE;

  // ---- load (each byte once), optional fused EMA, weighting ------------------
  float w[NE], v[NE];
  if constexpr (W_BF16) {
    const uint4 t = ld128(reinterpret_cast<const uint16_t*>(mtx.W) + e0);
    const uint32_t d[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
    for (int k = 0; k < 4; k++) {
      w[2 * k] = as_f32(d[k] << 16);
      w[2 * k + 1] = as_f32(d[k] & 0xffff0000u);
    }
  } else {
    const float* wp = reinterpret_cast<const float*>(mtx.W) + e0;
    const uint4 a = ld128(wp), b = ld128(wp + 4);
    w[0] = as_f32(a.x); w[1] = as_f32(a.y); w[2] = as_f32(a.z); w[3] = as_f32(a.w);
    w[4] = as_f32(b.x); w[5] = as_f32(b.y); w[6] = as_f32(b.z); w[7] = as_f32(b.w);
  }
  {
    const uint4 a = ld128(mtx.v + e0), b = ld128(mtx.v + e0 + 4);
    v[0] = as_f32(a.x); v[1] = as_f32(a.y); v[2] = as_f32(a.z); v[3] = as_f32(a.w);
    v[4] = as_f32(b.x); v[5] = as_f32(b.y); v[6] = as_f32(b.z); v[7] = as_f32(b.w);
  }
  if constexpr (EMA != 0) {
    float g[NE];
    if constexpr (EMA == 1) {
      const uint4 t = ld128(reinterpret_cast<const uint16_t*>(mtx.g) + e0);
      const uint32_t d[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
      for (int k = 0; k < 4; k++) {
        g[2 * k] = as_f32(d[k] << 16);
        g[2 * k + 1] = as_f32(d[k] & 0xffff0000u);
      }
    } else {
      const float* gp = reinterpret_cast<const float*>(mtx.g) + e0;
      const uint4 a = ld128(gp), b = ld128(gp + 4);
      g[0] = as_f32(a.x); g[1] = as_f32(a.y); g[2] = as_f32(a.z); g[3] = as_f32(a.w);
      g[4] = as_f32(b.x); g[5] = as_f32(b.y); g[6] = as_f32(b.z); g[7] = as_f32(b.w);
    }
#pragma unroll
    for (int i = 0; i < NE; i++) {
      const float t = g[i] * g[i];
      const float u = p.omb2 * t;
      v[i] = __builtin_fmaf(p.beta2, v[i], u);
    }
    st128(mtx.v + e0, make_uint4(as_u32(v[0]), as_u32(v[1]), as_u32(v[2]), as_u32(v[3])));
    st128(mtx.v + e0 + 4, make_uint4(as_u32(v[4]), as_u32(v[5]), as_u32(v[6]), as_u32(v[7])));
  }
  if (p.weighting != 0) {
#pragma unroll
    for (int i = 0; i < NE; i++) v[i] = weight_of(v[i], p.weighting);
  }

  // ---- block range and clip-independent moments ------------------------------
  float mn = w[0], mx = w[0];
#pragma unroll
  for (int i = 1; i < NE; i++) {
    mn = fminf(mn, w[i]);
    mx = fmaxf(mx, w[i]);
  }
  mn = run_min<16>(mn);
  mn = fminf(mn, __shfl_xor(mn, 16, 64));
  mn = fminf(mn, __shfl_xor(mn, 32, 64));
  mx = run_max<16>(mx);
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  double H[NE], HW[NE];
  double sww = 0.0, sh = 0.0;
#pragma unroll
  for (int i = 0; i < NE; i++) {
    H[i] = (double)v[i];
    HW[i] = H[i] * (double)w[i];
    sww = __builtin_fma(HW[i], (double)w[i], sww);
    sh += H[i];
  }
  sww = run_sum<16>(sww);
  sww += __shfl_xor(sww, 16, 64);
  sww += __shfl_xor(sww, 32, 64);
  sh = run_sum<16>(sh);
  sh += __shfl_xor(sh, 16, 64);
  sh += __shfl_xor(sh, 32, 64);

  const bool constant = (mx == mn);
  const float c = 0.5f * (mx + mn);
  const float rho = 0.5f * (mx - mn);
  const float rrho = 1.0f / rho;
  const float nc = -(c * rrho);
  float u[NE];
#pragma unroll
  for (int i = 0; i < NE; i++) u[i] = __builtin_fmaf(w[i], rrho, nc);

  Bin(*bins)[64] = s_bins[wave];
  Bin(*part)[8] = s_part[wave];
  const int b8 = lane & 7;  // the index this lane reduces / owns in the codebook stage
  double best_key = __longlong_as_double(0x7ff0000000000000ll);
  uint32_t best_e = 0;  // lane b8's codebook byte of the best clip (lanes 0..7)

  for (int k = 0; k < (constant ? 0 : K); k++) {
    const float al = uniform_f32(s_alpha[k]);
    // ---- this lane's per-index sums, in its private LDS bins -----------------
#pragma unroll
    for (int b = 0; b < 8; b++) bins[b][lane] = Bin{0.0, 0.0};
#pragma unroll
    for (int i = 0; i < NE; i++) {
      const float x = __builtin_fmaf(u[i], al, 3.5f);
      const int q = (int)__builtin_amdgcn_fmed3f(__builtin_rintf(x), 0.0f, 7.0f);
      Bin t = bins[q][lane];
      t.h += H[i];
      t.hw += HW[i];
      bins[q][lane] = t;
    }
    wave_lds_fence();
    // ---- reduce over lanes: lane j sums index j/8 over the lanes congruent
    // to j mod 8 (each group of 8 lanes reads 8 consecutive 16-byte slots:
    // no bank conflicts) ----------------------------------------------------
    {
      const int bi = lane >> 3, r0 = lane & 7;
      double a = 0.0, bsum = 0.0;
#pragma unroll
      for (int t = 0; t < 8; t++) {
        const Bin x = bins[bi][r0 + 8 * t];
        a += x.h;
        bsum += x.hw;
      }
      part[r0][bi] = Bin{a, bsum};
    }
    wave_lds_fence();
    // ---- lanes b = 0..7 (replicated in every group of 8): index b's totals ---
    double hb = 0.0, hwb = 0.0;
#pragma unroll
    for (int t = 0; t < 8; t++) {
      const Bin x = part[t][b8];
      hb += x.h;
      hwb += x.hw;
    }
    wave_lds_fence();  // every lane has read part before the next clip writes it
    // Eq. rubin-fit: the loss-aware mean, in E4M3; an index with no saliency
    // mass keeps the E4M3 value of its grid level
    float meanf;
    if (hb > 0.0) {
      meanf = (float)div_f64(hwb, hb, rcp_f64(hb));
    } else {
      const float f = uniform_f32(s_clip[k]);
      const float fr = f * rho;
      meanf = __builtin_fmaf((float)b8, (2.0f * fr) / 7.0f, c - fr);
    }
    const uint32_t e = e4m3_byte(meanf);
    const double cv = (double)e4m3_value(e);
    // score: sum_b (C_b^2 H_b - 2 C_b HW_b) + sum h w^2, summed over b = lane % 8
    double term = cv * (cv * hb - 2.0 * hwb);
    term = run_sum<8>(term);
    const double score = sww + term;
    const double key = make_key(score, k);
    if (key < best_key) {  // uniform: every lane holds the same score
      best_key = key;
      best_e = e;
    }
  }

  // ---- emit ------------------------------------------------------------------
  const int kstar = key_index(best_key);
  float* lut = s_lut[wave];
  uint32_t lut_byte;
  float err;
  if (constant) {
    lut_byte = e4m3_byte(mn);
    const double d = (double)e4m3_value(lut_byte) - (double)mn;
    err = (float)(sh * d * d);
  } else {
    lut_byte = best_e;
    err = (float)__longlong_as_double(__double_as_longlong(best_key) & ~15ll);
  }
  if (lane < 8) lut[lane] = e4m3_value(lut_byte);
  wave_lds_fence();
  const float alpha = s_alpha[constant ? 0 : kstar];
  uint32_t bits = 0;
  float r[NE];
#pragma unroll
  for (int i = 0; i < NE; i++) {
    const float x = __builtin_fmaf(u[i], alpha, 3.5f);
    uint32_t q = (uint32_t)__builtin_amdgcn_fmed3f(__builtin_rintf(x), 0.0f, 7.0f);
    if (constant) q = 0;
    bits |= q << (3 * i);
    r[i] = lut[q];
  }
  // 24 bits per lane at byte offset 3 lane of the block's 192-byte stream
  uint8_t* cp = mtx.codes + bid * 192 + lane * 3;
  cp[0] = (uint8_t)bits;
  cp[1] = (uint8_t)(bits >> 8);
  cp[2] = (uint8_t)(bits >> 16);
  if (mtx.r) {
    if constexpr (W_BF16) {
      st128(reinterpret_cast<uint16_t*>(mtx.r) + e0,
            make_uint4(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]), pack_bf16x2(r[4], r[5]),
                       pack_bf16x2(r[6], r[7])));
    } else {
      float* rp = reinterpret_cast<float*>(mtx.r) + e0;
      st128(rp, make_uint4(as_u32(r[0]), as_u32(r[1]), as_u32(r[2]), as_u32(r[3])));
      st128(rp + 4, make_uint4(as_u32(r[4]), as_u32(r[5]), as_u32(r[6]), as_u32(r[7])));
    }
  }
  if (lane < 8) mtx.lut[bid * 8 + lane] = (uint8_t)lut_byte;
  if (lane == 0) {
    if (mtx.best_clip) mtx.best_clip[bid] = (uint8_t)(constant ? 0 : kstar);
    if (mtx.err) mtx.err[bid] = err;
  }
}

template <bool W_BF16>
hipError_t launch_e(const RubinParams& p, int ema_mode, hipStream_t s) {
  const int64_t blocks = p.batch.n > 1 ? p.batch.total_blocks : (p.n_blocks + kWaves - 1) / kWaves;
  const dim3 grid((unsigned)blocks), block(kThreads);
  switch (ema_mode) {
    case 1: hipLaunchKernelGGL((rubin_reconstruct_kernel<W_BF16, 1>), grid, block, 0, s, p); break;
    case 2: hipLaunchKernelGGL((rubin_reconstruct_kernel<W_BF16, 2>), grid, block, 0, s, p); break;
    default: hipLaunchKernelGGL((rubin_reconstruct_kernel<W_BF16, 0>), grid, block, 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rubin(const RubinParams& p, bool w_bf16, int ema_mode, hipStream_t s) {
  return w_bf16 ? launch_e<true>(p, ema_mode, s) : launch_e<false>(p, ema_mode, s);
}

}  // namespace quasar
