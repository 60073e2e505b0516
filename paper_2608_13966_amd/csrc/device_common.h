// device_common.h -- device helpers for the CDNA4 (gfx950) kernels:
// 128-bit loads/stores, bf16 <-> fp32, DPP lane exchanges inside a row of 16.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace quasar {

// ---- bit casts -------------------------------------------------------------
__device__ __forceinline__ float as_f32(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t as_u32(float f) { return __float_as_uint(f); }

// A value known to be the same in every lane, moved to a scalar register
// (bit copy: the builtin's operand is an int).
__device__ __forceinline__ float uniform_f32(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

// The wavefront's index in its workgroup, in a scalar register: the compiler
// does not see that threadIdx.x / 64 is the same in every lane, and would
// otherwise do the arithmetic derived from it (addresses, a block index
// division) per lane.
__device__ __forceinline__ int wave_index() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// The bucket of u among 256 equal slices of [-1, 1]: clamp(floor(u * 128),
// -128, 127) + 128 (u * 128 is exact, so a boundary falls exactly at u = 0);
// any u, NaN included, gives an index in [0, 256).
__device__ __forceinline__ int cell_bucket(float u) {
  int f;
  asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(f) : "v"(u * 128.0f));
  return min(max(f, -128), 127) + 128;
}

// ---- bf16 ------------------------------------------------------------------
// Two fp32 values -> packed bf16 (round to nearest even) in one gfx950
// instruction (v_cvt_pk_bf16_f32); the low half holds `a`.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  f32x2 v = {a, b};
  bf16x2 h = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// ---- deployed precision of a dequantiser parameter ---------------------------
// fp32 -> fp16 or bf16 (round to nearest even; fp16 overflows to infinity as
// the IEEE conversion does) and back.  mode: 0 fp32 (unchanged), 1 bf16, 2 fp16.
__device__ __forceinline__ float round_param(float x, int mode) {
  if (mode == 2) return (float)(_Float16)x;
  if (mode == 1) return as_f32(pack_bf16x2(x, 0.0f) << 16);
  return x;
}

// Saliency weight of one element: h = v, v*v (fp32) or 1.
__device__ __forceinline__ float weight_of(float v, int weighting) {
  return weighting == 1 ? v * v : weighting == 2 ? 1.0f : v;
}

// ---- reciprocal and quotient in fp64 without the IEEE division sequence ------
// v_rcp_f64 plus Newton steps: within a few ulp of 1/d (d normal, not huge).
__device__ __forceinline__ double rcp_f64(double d) {
  double r = __builtin_amdgcn_rcp(d);
  double e = __builtin_fma(-d, r, 1.0);
  r = __builtin_fma(r, e, r);
  e = __builtin_fma(-d, r, 1.0);
  return __builtin_fma(r, e, r);
}
// n / d from a reciprocal, with one residual correction.
__device__ __forceinline__ double div_f64(double n, double d, double rd) {
  double q = n * rd;
  double res = __builtin_fma(-d, q, n);
  return __builtin_fma(res, rd, q);
}

// ---- 128-bit global memory access ------------------------------------------
__device__ __forceinline__ uint4 ld128(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st128(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

// Load N = 16 consecutive elements of a fp32 or bf16 tensor as fp32.
template <bool BF16>
__device__ __forceinline__ void load16(const void* base, int64_t e0, float (&x)[16]) {
  if constexpr (BF16) {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(base) + e0;
#pragma unroll
    for (int c = 0; c < 2; c++) {
      uint4 t = ld128(p + 8 * c);
      uint32_t w4[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
      for (int k = 0; k < 4; k++) {
        x[8 * c + 2 * k] = as_f32(w4[k] << 16);
        x[8 * c + 2 * k + 1] = as_f32(w4[k] & 0xffff0000u);
      }
    }
  } else {
    const float* p = reinterpret_cast<const float*>(base) + e0;
#pragma unroll
    for (int c = 0; c < 4; c++) {
      uint4 t = ld128(p + 4 * c);
      x[4 * c] = as_f32(t.x);
      x[4 * c + 1] = as_f32(t.y);
      x[4 * c + 2] = as_f32(t.z);
      x[4 * c + 3] = as_f32(t.w);
    }
  }
}

template <bool BF16>
__device__ __forceinline__ void store16(void* base, int64_t e0, const float (&x)[16]) {
  if constexpr (BF16) {
    uint16_t* p = reinterpret_cast<uint16_t*>(base) + e0;
#pragma unroll
    for (int c = 0; c < 2; c++) {
      uint32_t w4[4];
#pragma unroll
      for (int k = 0; k < 4; k++) w4[k] = pack_bf16x2(x[8 * c + 2 * k], x[8 * c + 2 * k + 1]);
      st128(p + 8 * c, make_uint4(w4[0], w4[1], w4[2], w4[3]));
    }
  } else {
    float* p = reinterpret_cast<float*>(base) + e0;
#pragma unroll
    for (int c = 0; c < 4; c++)
      st128(p + 4 * c, make_uint4(as_u32(x[4 * c]), as_u32(x[4 * c + 1]), as_u32(x[4 * c + 2]),
                                  as_u32(x[4 * c + 3])));
  }
}

// 16 consecutive W elements held in their storage format (bf16: 8 packed
// dwords) and widened to fp32 on use.
template <bool BF16>
struct WRegs;
template <>
struct WRegs<true> {
  uint32_t d[8];
  __device__ __forceinline__ void load(const void* base, int64_t e0) {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(base) + e0;
    uint4 a = ld128(p), b = ld128(p + 8);
    d[0] = a.x; d[1] = a.y; d[2] = a.z; d[3] = a.w;
    d[4] = b.x; d[5] = b.y; d[6] = b.z; d[7] = b.w;
  }
  __device__ __forceinline__ float get(int i) const {
    return (i & 1) ? as_f32(d[i >> 1] & 0xffff0000u) : as_f32(d[i >> 1] << 16);
  }
  // replace the weights by w rounded to bf16 (nearest even)
  __device__ __forceinline__ void set(const float (&w)[16]) {
#pragma unroll
    for (int k = 0; k < 8; k++) d[k] = pack_bf16x2(w[2 * k], w[2 * k + 1]);
  }
  __device__ __forceinline__ void store(void* base, int64_t e0) const {
    uint16_t* p = reinterpret_cast<uint16_t*>(base) + e0;
    st128(p, make_uint4(d[0], d[1], d[2], d[3]));
    st128(p + 8, make_uint4(d[4], d[5], d[6], d[7]));
  }
};
template <>
struct WRegs<false> {
  float f[16];
  __device__ __forceinline__ void load(const void* base, int64_t e0) { load16<false>(base, e0, f); }
  __device__ __forceinline__ float get(int i) const { return f[i]; }
  __device__ __forceinline__ void set(const float (&w)[16]) {
#pragma unroll
    for (int i = 0; i < 16; i++) f[i] = w[i];
  }
  __device__ __forceinline__ void store(void* base, int64_t e0) const { store16<false>(base, e0, f); }
};

// Constants of one AdamW step, computed on the host.
struct AdamWConsts {
  float beta1, omb1;     // beta1 and 1 - beta1 (fp32)
  float eps;
  float decay;           // 1 - lr * weight_decay
  float step_size;       // lr / (1 - beta1^t)
  float rbc2;            // 1 / sqrt(1 - beta2^t)
};

// One AdamW step (decoupled weight decay, bias-corrected) on 16 weights, in
// place, fp32 in a fixed order:
//   m' = fmaf(beta1, m, (1 - beta1) g)        v' = fmaf(beta2, v, (1 - beta2) (g g))
//   w' = fmaf(-step_size, m' / fmaf(sqrtf(v'), rbc2, eps), w * decay)
// sqrtf and the quotient are the correctly rounded ones.
__device__ __forceinline__ void adamw16(float (&w)[16], float (&m)[16], float (&v)[16], const float (&g)[16],
                                        const AdamWConsts& a, float beta2, float omb2) {
#pragma unroll
  for (int i = 0; i < 16; i++) {
    const float mm = __builtin_fmaf(a.beta1, m[i], a.omb1 * g[i]);
    const float t = g[i] * g[i];
    const float vv = __builtin_fmaf(beta2, v[i], omb2 * t);
    const float den = __builtin_fmaf(__builtin_sqrtf(vv), a.rbc2, a.eps);
    const float upd = mm / den;
    m[i] = mm;
    v[i] = vv;
    w[i] = __builtin_fmaf(-a.step_size, upd, w[i] * a.decay);
  }
}

// ---- DPP exchanges (GFX9 encodings; all stay inside a row of 16 lanes) ------
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i inside each 8
constexpr int kDppMirror = 0x140;     // lane i <-> 15 - i inside each 16

// x of the lane that DPP control CTRL names, 0 where it names none (bound_ctrl:
// no old value to set up first)
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) { return as_f32(dpp_u32<CTRL>(as_u32(x))); }
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  uint64_t u = __double_as_longlong(x);
  uint32_t lo = dpp_u32<CTRL>((uint32_t)u), hi = dpp_u32<CTRL>((uint32_t)(u >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// min / max of two floats as one v_min_f32 / v_max_f32: fminf and fmaxf
// first quiet their inputs (one more instruction for each value that comes
// from another lane).  Equal for non-NaN inputs; NaN inputs give unspecified
// results, as everywhere in the library.
__device__ __forceinline__ float min_f32(float a, float b) {
  float r;
  asm("v_min_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ float max_f32(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// All-reduce over aligned runs of L consecutive lanes (L in 1, 2, 4, 8, 16).
// The patterns pair lanes symmetrically, and IEEE addition / min / max are
// commutative, so every lane of a run ends with a bit-identical result.
template <int L>
__device__ __forceinline__ float run_min(float x) {
  if constexpr (L >= 2) x = min_f32(x, dpp_f32<kDppXor1>(x));
  if constexpr (L >= 4) x = min_f32(x, dpp_f32<kDppXor2>(x));
  if constexpr (L >= 8) x = min_f32(x, dpp_f32<kDppHalfMirror>(x));
  if constexpr (L >= 16) x = min_f32(x, dpp_f32<kDppMirror>(x));
  return x;
}
template <int L>
__device__ __forceinline__ float run_max(float x) {
  if constexpr (L >= 2) x = max_f32(x, dpp_f32<kDppXor1>(x));
  if constexpr (L >= 4) x = max_f32(x, dpp_f32<kDppXor2>(x));
  if constexpr (L >= 8) x = max_f32(x, dpp_f32<kDppHalfMirror>(x));
  if constexpr (L >= 16) x = max_f32(x, dpp_f32<kDppMirror>(x));
  return x;
}
template <int L>
__device__ __forceinline__ double run_sum(double x) {
  if constexpr (L >= 2) x = x + dpp_f64<kDppXor1>(x);
  if constexpr (L >= 4) x = x + dpp_f64<kDppXor2>(x);
  if constexpr (L >= 8) x = x + dpp_f64<kDppHalfMirror>(x);
  if constexpr (L >= 16) x = x + dpp_f64<kDppMirror>(x);
  return x;
}
// minimum of two keys (non-negative, never NaN: see make_key): v_min_f64
// without the quieting of its inputs that fmin() adds
__device__ __forceinline__ double min_key(double a, double b) {
  double r;
  asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
template <int L>
__device__ __forceinline__ double run_min_f64(double x) {
  if constexpr (L >= 2) x = min_key(x, dpp_f64<kDppXor1>(x));
  if constexpr (L >= 4) x = min_key(x, dpp_f64<kDppXor2>(x));
  if constexpr (L >= 8) x = min_key(x, dpp_f64<kDppHalfMirror>(x));
  if constexpr (L >= 16) x = min_key(x, dpp_f64<kDppMirror>(x));
  return x;
}

// op(x, x of lane l ^ 16) (ROWS = 16) or op(x, x of lane l ^ 32) (ROWS = 32)
// without LDS: v_permlane16_swap / v_permlane32_swap of x with itself leave
// the two rows (halves) of each pair in two registers, at the same positions
// in both, so op of the two is the same value in every lane of the pair (for
// a commutative op).
template <int ROWS>
__device__ __forceinline__ void swap_rows(uint32_t x, uint32_t& a, uint32_t& b) {
  if constexpr (ROWS == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    a = r[0];
    b = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    a = r[0];
    b = r[1];
  }
}
template <int ROWS, typename Op>
__device__ __forceinline__ float pair_rows(float x, Op op) {
  uint32_t a, b;
  swap_rows<ROWS>(as_u32(x), a, b);
  return op(as_f32(a), as_f32(b));
}
template <int ROWS, typename Op>
__device__ __forceinline__ double pair_rows(double x, Op op) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  uint32_t alo, blo, ahi, bhi;
  swap_rows<ROWS>((uint32_t)u, alo, blo);
  swap_rows<ROWS>((uint32_t)(u >> 32), ahi, bhi);
  return op(__longlong_as_double((long long)(((uint64_t)ahi << 32) | alo)),
            __longlong_as_double((long long)(((uint64_t)bhi << 32) | blo)));
}

// Combine values that are uniform within each row of 16 over the wavefront's
// four rows, without LDS: row_bcast:15 brings row 0's value into row 1 and
// row 2's into row 3, row_bcast:31 brings lane 31's into rows 2 and 3 (rows
// outside the mask take `id`, the operation's identity), and lane 63, which
// then holds op(op(r3, r2), op(r1, r0)), is read into every lane.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_rows(uint32_t id, uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)x, CTRL, ROW_MASK, 0xF, false);
}
__device__ __forceinline__ float rows_min(float x) {
  x = min_f32(x, as_f32(dpp_rows<0x142, 0xA>(as_u32(INFINITY), as_u32(x))));
  x = min_f32(x, as_f32(dpp_rows<0x143, 0xC>(as_u32(INFINITY), as_u32(x))));
  return as_f32((uint32_t)__builtin_amdgcn_readlane((int)as_u32(x), 63));
}
__device__ __forceinline__ float rows_max(float x) {
  x = max_f32(x, as_f32(dpp_rows<0x142, 0xA>(as_u32(-INFINITY), as_u32(x))));
  x = max_f32(x, as_f32(dpp_rows<0x143, 0xC>(as_u32(-INFINITY), as_u32(x))));
  return as_f32((uint32_t)__builtin_amdgcn_readlane((int)as_u32(x), 63));
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_rows_f64(double id, double x) {
  const uint64_t i = (uint64_t)__double_as_longlong(id), u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = dpp_rows<CTRL, ROW_MASK>((uint32_t)i, (uint32_t)u);
  const uint32_t hi = dpp_rows<CTRL, ROW_MASK>((uint32_t)(i >> 32), (uint32_t)(u >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ double lane63_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 63);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ double rows_sum(double x) {
  x = x + dpp_rows_f64<0x142, 0xA>(0.0, x);
  x = x + dpp_rows_f64<0x143, 0xC>(0.0, x);
  return lane63_f64(x);
}
__device__ __forceinline__ double rows_min_f64(double x) {  // of keys
  x = min_key(x, dpp_rows_f64<0x142, 0xA>(INFINITY, x));
  x = min_key(x, dpp_rows_f64<0x143, 0xC>(INFINITY, x));
  return lane63_f64(x);
}

// A non-negative score with the candidate index in its 4 low mantissa bits:
// ordering keys as doubles orders by score (to 2^-48 relative) and then by
// index, so a min over keys is the argmin with ties to the lowest index.
__device__ __forceinline__ double make_key(double score, int k) {
  score = fmax(score, 0.0);
  uint64_t u = (uint64_t)__double_as_longlong(score);
  u = (u & ~(uint64_t)15) | (uint64_t)(k & 15);
  return __longlong_as_double((long long)u);
}
__device__ __forceinline__ int key_index(double key) {
  return (int)((uint64_t)__double_as_longlong(key) & 15);
}

// Orders this wave's LDS accesses across lanes: writes issued before the
// fence are visible to reads issued after it (a wavefront executes its LDS
// instructions in order; the fence stops the compiler from reordering them).
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---- coalesced stores of a wavefront's stretch of a tensor -------------------
// A wavefront whose lanes hold 16 consecutive elements each covers one
// contiguous stretch of 1024 elements: lane l's 16 start at element
// 16 idx(l) of it, idx a permutation of the lanes.  Stored straight from the
// registers, every store instruction writes a 16-byte piece of each of 64
// different cache lines, and the lines are completed by later instructions.
// Written into LDS in stretch order and read back 16 bytes per lane in memory
// order, each store instruction writes 1 KB of whole lines instead.  One
// 16-byte pad after every PER chunks of 16 bytes keeps the LDS writes free of
// bank conflicts: PER is the chunks of one group (spread layouts, where lanes
// 0..7 hold the first chunks of eight groups) or of one lane (consecutive
// layouts).
struct WaveImage {
  uint4* stage;  // this wavefront's LDS area: wave_stage_chunks() chunks of 16 bytes
  int64_t e0;    // the stretch's first element
  int64_t n;     // how many of its 1024 elements exist (<= 0: none)
  int idx;       // this lane's 16 elements start at element 16 idx of the stretch
  int lane;
};

template <int ESZ, int PER>
__host__ __device__ constexpr int wave_stage_chunks() {
  return 64 * ESZ + 64 * ESZ / PER;  // ESZ chunks per lane for 16 elements of ESZ bytes
}

// Every lane of the wavefront takes part; `base` is the tensor (16-byte
// aligned), and elements of the stretch at or past n are not written.
// wave_put writes the lane's chunk c (c < ESZ: its elements 16 c / ESZ
// onwards) into the stage, after a wave_lds_fence() that follows any earlier
// use of the stage; wave_flush then stores the whole stretch and leaves the
// stage free.  wave_store does both for the lane's 16 elements given as
// 4 ESZ dwords in element order.
template <int ESZ, int PER>
__device__ __forceinline__ void wave_put(const WaveImage& im, int c, uint4 x) {
  const int ch = im.idx * ESZ + c;
  im.stage[ch + ch / PER] = x;
}
template <int ESZ, int PER>
__device__ __forceinline__ void wave_flush(const WaveImage& im, void* base) {
  static_assert(ESZ == 2 || ESZ == 4, "bf16 or fp32 elements");
  wave_lds_fence();
  // one chunk in flight at a time: fewer live registers than reading all
  // chunks first, which the kernels around this cannot spare
  uint4* out = reinterpret_cast<uint4*>(base) + (im.e0 * ESZ) / 16;
#pragma unroll
  for (int t = 0; t < ESZ; t++) {
    const int ch = im.lane + 64 * t;
    const uint4 x = im.stage[ch + ch / PER];
    if ((int64_t)ch * (16 / ESZ) < im.n) out[ch] = x;
  }
  wave_lds_fence();
}
template <int ESZ, int PER>
__device__ __forceinline__ void wave_store(const WaveImage& im, void* base, const uint32_t (&d)[4 * ESZ]) {
  wave_lds_fence();  // earlier reads of the stage by this wavefront are done
#pragma unroll
  for (int c = 0; c < ESZ; c++) wave_put<ESZ, PER>(im, c, make_uint4(d[4 * c], d[4 * c + 1], d[4 * c + 2], d[4 * c + 3]));
  wave_flush<ESZ, PER>(im, base);
}

template <int PER>
__device__ __forceinline__ void wave_store_f32(const WaveImage& im, float* base, const float (&x)[16]) {
  uint32_t d[16];
#pragma unroll
  for (int i = 0; i < 16; i++) d[i] = as_u32(x[i]);
  wave_store<4, PER>(im, base, d);
}

}  // namespace quasar
