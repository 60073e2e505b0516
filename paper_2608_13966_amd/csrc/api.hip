// api.hip -- the C ABI of libquasar.so (declared in include/quasar.h):
// host-side argument validation, clip-table preparation and kernel dispatch.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>

#include "quasar.h"
#include "quasar_internal.h"

namespace {

bool aligned16(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int group_of(const quasar_desc* d) { return d->format == QUASAR_NVFP4 ? 16 : d->group; }
int bits_of(const quasar_desc* d) { return d->format == QUASAR_NVFP4 ? 4 : d->bits; }
bool is_rubin(const quasar_desc* d) { return d->format == QUASAR_RUBIN_INT3; }

// Validation of the descriptor alone.
int check_desc(const quasar_desc* d) {
  if (d == nullptr) return QUASAR_ERR_ARG;
  if (d->w_dtype != QUASAR_F32 && d->w_dtype != QUASAR_BF16) return QUASAR_ERR_FORMAT;
  if (d->format == QUASAR_INT || d->format == QUASAR_INT_SYM) {
    if (d->bits < 2 || d->bits > 4) return QUASAR_ERR_FORMAT;
    if (d->group != 64 && d->group != 128) return QUASAR_ERR_FORMAT;
  } else if (d->format == QUASAR_NVFP4) {
    if (d->group != 16) return QUASAR_ERR_FORMAT;
  } else if (d->format == QUASAR_RUBIN_INT3) {
    if (d->bits != 3 || d->group != 512) return QUASAR_ERR_FORMAT;
  } else {
    return QUASAR_ERR_FORMAT;
  }
  if (d->rows < 1 || d->cols < 1) return QUASAR_ERR_SHAPE;
  if (is_rubin(d)) {
    if (d->rows % 8 != 0 || d->cols % 64 != 0) return QUASAR_ERR_SHAPE;
  } else if (d->cols % group_of(d) != 0) {
    return QUASAR_ERR_SHAPE;
  }
  // group ids and grid sizes stay far inside int64 / launch limits
  if (d->rows > ((int64_t)1 << 40) / d->cols) return QUASAR_ERR_SHAPE;
  if (d->n_clips < 1 || d->n_clips > QUASAR_MAX_CLIPS) return QUASAR_ERR_ARG;
  if (d->weighting < QUASAR_WEIGHT_H || d->weighting > QUASAR_WEIGHT_NONE) return QUASAR_ERR_ARG;
  if (d->param_dtype != QUASAR_F32 && d->param_dtype != QUASAR_F16 && d->param_dtype != QUASAR_BF16)
    return QUASAR_ERR_FORMAT;
  if (d->format != QUASAR_INT && d->format != QUASAR_INT_SYM && d->param_dtype != QUASAR_F32)
    return QUASAR_ERR_FORMAT;
  if (d->clip_ratios == nullptr) return QUASAR_ERR_ARG;
  for (int k = 0; k < d->n_clips; k++) {
    const float f = d->clip_ratios[k];
    // (0, 1] as in Alg. 1; factors below 2^-24 would overflow qmax / (2 f)
    if (!(f > 0.0f && f <= 1.0f) || f < 5.9604645e-08f) return QUASAR_ERR_ARG;
  }
  return QUASAR_OK;
}

}  // namespace

extern "C" {

const char* quasar_version(void) { return "0.1.0"; }

const char* quasar_status_string(int s) {
  switch (s) {
    case QUASAR_OK: return "ok";
    case QUASAR_ERR_ARG:
      return "invalid argument (NULL pointer, n_clips, clip ratio, beta2 or weighting out of range)";
    case QUASAR_ERR_SHAPE: return "invalid shape (rows/cols < 1, cols not a multiple of the group, too large)";
    case QUASAR_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case QUASAR_ERR_FORMAT: return "unsupported format, bits, group size, dtype or parameter precision";
    case QUASAR_ERR_WORKSPACE: return "workspace missing or too small";
    case QUASAR_ERR_DEVICE: return "HIP launch error";
    default: return "unknown status";
  }
}

int64_t quasar_num_groups(const quasar_desc* d) {
  if (check_desc(d) != QUASAR_OK) return 0;
  if (is_rubin(d)) return (d->rows / 8) * (d->cols / 64);
  return d->rows * (d->cols / group_of(d));
}

size_t quasar_codes_bytes(const quasar_desc* d) {
  if (check_desc(d) != QUASAR_OK) return 0;
  return (size_t)(d->rows * d->cols) * (size_t)bits_of(d) / 8u;
}

size_t quasar_workspace_bytes(const quasar_desc* d, int has_tensor_amax) {
  if (check_desc(d) != QUASAR_OK) return 0;
  return (d->format == QUASAR_NVFP4 && !has_tensor_amax) ? 256u : 0u;
}

int quasar_check(const quasar_desc* d, const void* W, const float* v, const void* g, const uint8_t* codes,
                 const void* scales, const float* zeros, const void* r, const uint8_t* best_clip,
                 const float* err, const float* tensor_scale, const float* tensor_amax, const void* workspace,
                 size_t workspace_bytes) {
  int s = check_desc(d);
  if (s != QUASAR_OK) return s;
  if (g != nullptr) {
    if (d->g_dtype != QUASAR_F32 && d->g_dtype != QUASAR_BF16) return QUASAR_ERR_FORMAT;  // no fp16 g
    if (!(d->beta2 >= 0.5f && d->beta2 < 1.0f)) return QUASAR_ERR_ARG;
  }
  if (W == nullptr || v == nullptr || codes == nullptr || scales == nullptr) return QUASAR_ERR_ARG;
  if (d->format == QUASAR_INT && zeros == nullptr) return QUASAR_ERR_ARG;
  if (d->format == QUASAR_NVFP4 && tensor_scale == nullptr) return QUASAR_ERR_ARG;
  if (d->format != QUASAR_NVFP4 && tensor_amax != nullptr) return QUASAR_ERR_ARG;
  const void* ptrs[] = {W, v, g, codes, scales, zeros, r, best_clip, err, tensor_scale, tensor_amax, workspace};
  for (const void* p : ptrs)
    if (!aligned16(p)) return QUASAR_ERR_ALIGN;
  const size_t need = quasar_workspace_bytes(d, tensor_amax != nullptr);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return QUASAR_ERR_WORKSPACE;
  return QUASAR_OK;
}

int quasar_absmax(const quasar_desc* d, const void* W, float* amax_out, void* stream) {
  int s = check_desc(d);
  if (s != QUASAR_OK) return s;
  if (d->format != QUASAR_NVFP4) return QUASAR_ERR_FORMAT;
  if (W == nullptr || amax_out == nullptr) return QUASAR_ERR_ARG;
  if (!aligned16(W) || !aligned16(amax_out)) return QUASAR_ERR_ALIGN;
  const hipError_t e = quasar::launch_absmax(W, d->w_dtype == QUASAR_BF16, d->rows * d->cols,
                                             reinterpret_cast<unsigned*>(amax_out),
                                             reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? QUASAR_OK : QUASAR_ERR_DEVICE;
}

int quasar_absmax_batch_check(const quasar_desc* d, const quasar_matrix* mats, int n_mats,
                              float* const* amax_out) {
  if (d == nullptr || mats == nullptr || amax_out == nullptr || n_mats < 1 || n_mats > QUASAR_MAX_BATCH)
    return QUASAR_ERR_ARG;
  int64_t total = 0;
  for (int i = 0; i < n_mats; i++) {
    quasar_desc dd = *d;
    dd.rows = mats[i].rows;
    dd.cols = mats[i].cols;
    const int s = check_desc(&dd);
    if (s != QUASAR_OK) return s;
    if (dd.format != QUASAR_NVFP4) return QUASAR_ERR_FORMAT;
    if (mats[i].W == nullptr || amax_out[i] == nullptr) return QUASAR_ERR_ARG;
    if (!aligned16(mats[i].W) || !aligned16(amax_out[i])) return QUASAR_ERR_ALIGN;
    // each output is cleared and then collects one matrix's maximum: two
    // matrices on one buffer would both get the larger of their maxima
    for (int k = 0; k < i; k++)
      if (amax_out[k] == amax_out[i]) return QUASAR_ERR_ARG;
    total += quasar::absmax_blocks(dd.rows * dd.cols / (dd.w_dtype == QUASAR_BF16 ? 8 : 4));
  }
  if (total >= ((int64_t)1 << 31)) return QUASAR_ERR_SHAPE;  // one grid
  return QUASAR_OK;
}

int quasar_absmax_batch(const quasar_desc* d, const quasar_matrix* mats, int n_mats, float* const* amax_out,
                        void* stream) {
  const int s = quasar_absmax_batch_check(d, mats, n_mats, amax_out);
  if (s != QUASAR_OK) return s;
  const bool w_bf16 = d->w_dtype == QUASAR_BF16;
  quasar::AbsmaxTable t;
  memset(&t, 0, sizeof(t));
  t.n = n_mats;
  for (int i = 0; i < n_mats; i++) {
    t.W[i] = mats[i].W;
    t.out[i] = reinterpret_cast<unsigned*>(amax_out[i]);
    // cols % 16 == 0: a whole number of 16-byte chunks in either dtype
    t.n_chunks[i] = mats[i].rows * mats[i].cols / (w_bf16 ? 8 : 4);
    t.block0[i + 1] = t.block0[i] + quasar::absmax_blocks(t.n_chunks[i]);
  }
  const hipError_t e = quasar::launch_absmax(t, w_bf16, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? QUASAR_OK : QUASAR_ERR_DEVICE;
}

}  // extern "C"

namespace {

// One AdamW step's host constants, fp64 then fp32 (the same expressions as
// the oracle's).
quasar::AdamWConsts adamw_consts(const quasar_adamw* opt) {
  quasar::AdamWConsts a;
  a.beta1 = opt->beta1;
  a.omb1 = 1.0f - opt->beta1;
  a.eps = opt->eps;
  a.decay = (float)(1.0 - (double)opt->lr * (double)opt->weight_decay);
  const double bc1 = 1.0 - pow((double)opt->beta1, (double)opt->step);
  const double bc2 = 1.0 - pow((double)opt->beta2, (double)opt->step);
  a.step_size = (float)((double)opt->lr / bc1);
  a.rbc2 = (float)(1.0 / sqrt(bc2));
  return a;
}

// The clip tables of the INT kernels: f_k and the code scale alpha_k
// (qmax / (2 f_k), symmetric Q / f_k, fp32 division); entries past K repeat
// the last clip.
void int_clip_tables(const quasar_desc* d, quasar::IntParams& p) {
  const bool sym = d->format == QUASAR_INT_SYM;
  const int K = d->n_clips;
  const float qmax = (float)((1 << d->bits) - 1);
  const float qsym = (float)((1 << (d->bits - 1)) - 1);
  for (int k = 0; k < quasar::kMaxClips; k++) {
    const float f = d->clip_ratios[k < K ? k : K - 1];
    p.clip[k] = f;
    p.alpha[k] = sym ? qsym / f : qmax / (2.0f * f);
  }
}

// The clip tables of the Rubin kernel: f_k and alpha_k = 7 / (2 f_k) (fp32
// division); entries past K repeat the last clip.
void rubin_clip_tables(const quasar_desc* d, quasar::RubinParams& p) {
  const int K = d->n_clips;
  for (int k = 0; k < quasar::kMaxClips; k++) {
    const float f = d->clip_ratios[k < K ? k : K - 1];
    p.clip[k] = f;
    p.alpha[k] = 7.0f / (2.0f * f);
  }
}

// The code of u under a clip with scale alpha, in the kernels' fp32 recipe:
// clamp(rint(fma(u, alpha, 3.5)), 0, 7) (correctly rounded fma, ties to even).
int rubin_code(float u, float alpha) {
  const float x = rintf(fmaf(u, alpha, 3.5f));
  return (int)fminf(fmaxf(x, 0.0f), 7.0f);
}

// fp32 values in increasing order <-> unsigned keys in increasing order
uint32_t f32_order_key(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
float f32_from_order_key(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

// Lay the sorted list out as an implicit binary search tree (node n's children
// at 2n and 2n + 1) by an in-order walk.
void eytzinger_fill(float* tree, const float* sorted, int& next, int node) {
  if (node >= quasar::kRubinThresholds) return;
  eytzinger_fill(tree, sorted, next, 2 * node);
  tree[node] = sorted[next++];
  eytzinger_fill(tree, sorted, next, 2 * node + 1);
}

int cell_bucket(float u);

// Extra cell boundaries for the Rubin kernel.  A boundary that is no clip's
// threshold leaves every code constant on both of its sides, so no result
// changes; what changes is how many of a block's weights share a cell, and
// the lanes of one 64-bit LDS atomic that land on one cell serialise.  Every
// clip's middle threshold lies at u = 0 and its next ones at +-f/3.5 or
// further, so on a grid of clips down to f = 0.3 the two cells beside 0 hold
// about a tenth of a bell-shaped block each.  Each cell is weighted by the
// share an N(0, 0.3^2) model of u puts in it (u = (w - c) / rho, with rho
// about three standard deviations for a bell-shaped block of 512), and the
// heaviest cell is halved until none holds more than 1.2% or the cells run
// out.  A split never falls inside [ulo, uhi] (the merged tie span); when
// `cnt` (thresholds per bucket, the bucket form) is given, it never takes a
// bucket above `cmax` thresholds.  Inserts into the sorted s[0 .. m) and
// returns the new m (at most m_max).
int rubin_split_cells(float* s, int m, int m_max, int* cnt, int cmax, float ulo, float uhi) {
  constexpr double kSigma = 0.3, kTarget = 0.012;
  auto cdf = [&](double x) { return 0.5 * std::erfc(-x / (kSigma * std::sqrt(2.0))); };
  // cell i = [s[i - 1], s[i]), the ends taken at -1 and 1; its model mass, or
  // -1 for an empty cell and for one found not to split
  auto lo = [&](int i) { return i == 0 ? -1.0f : s[i - 1]; };
  auto hi = [&](int i, int n) { return i == n ? 1.0f : s[i]; };
  auto mass_of = [&](int i, int n) {
    const double a = lo(i), b = hi(i, n);
    return b > a ? cdf(b) - cdf(a) : -1.0;
  };
  double mass[quasar::kRubinThresholds + 1];
  for (int i = 0; i <= m; i++) mass[i] = mass_of(i, m);
  while (m < m_max) {
    int best = -1;
    double best_mass = kTarget;
    for (int i = 0; i <= m; i++) {
      if (mass[i] > best_mass) {
        best_mass = mass[i];
        best = i;
      }
    }
    if (best < 0) break;
    const float a = lo(best), b = hi(best, m);
    const float mid = 0.5f * (a + b);
    bool ok = mid > a && mid < b && !(mid >= ulo && mid <= uhi);
    if (ok && cnt != nullptr) ok = cnt[cell_bucket(mid)] < cmax;
    if (!ok) {
      mass[best] = -1.0;
      continue;
    }
    if (cnt != nullptr) cnt[cell_bucket(mid)]++;
    for (int j = m; j > best; j--) s[j] = s[j - 1];
    s[best] = mid;
    for (int j = m + 1; j > best + 1; j--) mass[j] = mass[j - 1];
    m++;
    mass[best] = mass_of(best, m);
    mass[best + 1] = mass_of(best + 1, m);
  }
  return m;
}

// The bucket form of the Rubin kernel's cells from the thresholds t[7 k + b]
// = T(k, b) (see RubinParams): the tie-cluster thresholds T(k, 3) are merged
// into one at their least value, and every other bucket may hold at most
// three thresholds.  Returns false (the tree form is used) when the grid does
// not allow it or QUASAR_RUBIN_PATH=tree is set.
bool rubin_buckets(quasar::RubinParams& p, const float* t, int K) {
  const char* force = getenv("QUASAR_RUBIN_PATH");
  if (force != nullptr && strcmp(force, "tree") == 0) return false;
  const int n = 7 * K;
  float ulo = INFINITY, uhi = -INFINITY;
  for (int k = 0; k < K; k++) {
    ulo = fminf(ulo, t[7 * k + 3]);
    uhi = fmaxf(uhi, t[7 * k + 3]);
  }
  if (!(ulo > -0x1p-20f && uhi < 0.0f)) return false;
  const bool merge = ulo < uhi;
  float srt[quasar::kRubinThresholds];
  int m = 0;
  for (int i = 0; i < n; i++) srt[m++] = (merge && t[i] >= ulo && t[i] <= uhi) ? ulo : t[i];
  std::sort(srt, srt + m);
  m = (int)(std::unique(srt, srt + m) - srt);
  if (merge) {  // no other threshold may fall inside the merged span
    for (int i = 0; i < m; i++)
      if (srt[i] > ulo && srt[i] <= uhi) return false;
  }
  int cnt[quasar::kCellBuckets] = {0};
  int cmax = 1, below = 0;
  for (int i = 0; i < m; i++) cnt[cell_bucket(srt[i])]++;
  for (int b = 0; b < quasar::kCellBuckets; b++) cmax = std::max(cmax, cnt[b]);
  if (cmax > 3) return false;
  cmax = std::max(cmax, 2);
  // a bucket whose first cell is c reads thr[c .. c + 2], so the list keeps
  // two NaN entries of padding after its last threshold (c <= m)
  m = rubin_split_cells(srt, m, quasar::kRubinThresholds - 3, cnt, cmax, merge ? ulo : INFINITY,
                        merge ? uhi : INFINITY);
  cmax = 1;
  uint8_t base[quasar::kCellBuckets];
  for (int b = 0; b < quasar::kCellBuckets; b++) {
    cmax = std::max(cmax, cnt[b]);
    base[b] = (uint8_t)below;
    below += cnt[b];
  }
  for (int k = 0; k < quasar::kMaxClips; k++) {
    for (int b = 0; b < 9; b++) {
      int c = 0;
      if (k < K && b >= 1 && b <= 7) {
        float tb = t[7 * k + b - 1];
        if (merge && tb >= ulo && tb <= uhi) tb = ulo;
        c = (int)(std::lower_bound(srt, srt + m, tb) - srt) + 1;
      } else if (k < K && b == 8) {
        c = m + 1;
      }
      p.tpos[k][b] = (uint8_t)c;
    }
  }
  for (int i = 0; i < quasar::kRubinThresholds; i++) p.thr[i] = i < m ? srt[i] : NAN;
  memcpy(p.base, base, sizeof(base));
  p.buckets = 1;
  p.cmax = cmax;
  p.unsafe_lo = merge ? ulo : INFINITY;
  p.unsafe_hi = merge ? uhi : INFINITY;
  return true;
}

// The Rubin kernel's code thresholds: the code is non-decreasing in u, so
// T(k, b) = min{u : code_k(u) >= b + 1} is found by bisection over the
// ordered fp32 values between -inf (code 0) and +inf (code 7).
void rubin_thresholds(quasar::RubinParams& p, int K) {
  float t[quasar::kRubinThresholds];
  int n = 0;
  for (int k = 0; k < K; k++) {
    for (int b = 0; b < 7; b++) {
      // bracket: around the threshold of exact arithmetic, (b - 3) / alpha,
      // widened until it holds (else the whole range)
      const double center = (b - 3.0) / (double)p.alpha[k];
      uint32_t lo = f32_order_key(-INFINITY), hi = f32_order_key(INFINITY);
      for (double half = 1e-6; half < 4.0; half *= 16.0) {
        const uint32_t a = f32_order_key((float)(center - half)), z = f32_order_key((float)(center + half));
        if (rubin_code(f32_from_order_key(a), p.alpha[k]) < b + 1 &&
            rubin_code(f32_from_order_key(z), p.alpha[k]) >= b + 1) {
          lo = a;
          hi = z;
          break;
        }
      }
      while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (rubin_code(f32_from_order_key(mid), p.alpha[k]) >= b + 1)
          hi = mid;
        else
          lo = mid;
      }
      t[n++] = f32_from_order_key(hi);
    }
  }
  if (rubin_buckets(p, t, K)) return;
  // the tree form: every threshold (repeats included) plus the extra
  // boundaries; a weight's cell is the number of them at or below u
  float all[quasar::kRubinThresholds];
  std::copy(t, t + n, all);
  std::sort(all, all + n);
  const int na = rubin_split_cells(all, n, quasar::kRubinThresholds - 1, nullptr, 0, INFINITY, INFINITY);
  for (int k = 0; k < quasar::kMaxClips; k++) {
    for (int b = 0; b < 9; b++) {
      int cnt = 0;
      if (k < K && b >= 1 && b <= 7) {
        const float tb = t[7 * k + b - 1];
        for (int i = 0; i < na; i++) cnt += all[i] <= tb;
      } else if (k < K && b == 8) {
        cnt = na + 1;
      }
      p.tpos[k][b] = (uint8_t)cnt;
    }
  }
  // in-order walk of the complete tree with nodes 1 .. 127 = the sorted list
  float sorted[quasar::kRubinThresholds - 1];
  for (int i = 0; i < quasar::kRubinThresholds - 1; i++) sorted[i] = i < na ? all[i] : INFINITY;
  int next = 0;
  eytzinger_fill(p.thr, sorted, next, 1);
  p.thr[0] = INFINITY;
}

// The code of u under clip k of an INT-b group, in the kernels' fp32 recipe:
// asymmetric clamp(rint(fma(u, alpha, qmax/2)), 0, qmax), symmetric
// clamp(rint(u * alpha), -Q, Q) (correctly rounded fma and product, ties to
// even).
int int_code(float u, float alpha, int qmax, bool sym) {
  if (sym) {
    const float x = rintf(u * alpha);
    return (int)fminf(fmaxf(x, -(float)qmax), (float)qmax);
  }
  const float x = rintf(fmaf(u, alpha, 0.5f * (float)qmax));
  return (int)fminf(fmaxf(x, 0.0f), (float)qmax);
}

// The bucket of a finite u in the binned kernel, in its fp32 recipe:
// clamp(floor(u * 128), -128, 127) + 128 (u * 128 is exact), so a bucket
// boundary falls exactly at u = 0.
int cell_bucket(float u) {
  const float h = 0.5f * (float)quasar::kCellBuckets;
  return (int)fminf(fmaxf(floorf(u * h), -h), h - 1.0f) + quasar::kCellBuckets / 2;
}

// The binned INT kernel's tables for this clip grid (int_cells_kernel.hip):
// every threshold T(k, b) = the least fp32 u with code_k(u) >= q0 + b, found
// by bisection over the ordered fp32 values between -inf (the lowest code)
// and +inf (the highest).  Leaves n_cells = 0 -- the direct kernel runs --
// when the cells do not fit the kernel's LDS budget, when a lane would scan
// more than kCellsPerLaneAuto cells (the binned kernel's per-cell LDS work
// then outweighs the per-clip work it saves: INT4 grids), when a bucket
// needs more than three compares, or when QUASAR_INT_PATH=direct is set.
// QUASAR_INT_PATH=binned takes the binned kernel wherever its tables fit.
//
// With odd qmax every clip has a threshold just below u = 0, where the fp32
// code rounding ties at qmax/2: T(k, (qmax+1)/2) lies in (-2^-20, 0).  These
// tie thresholds are merged into one cell boundary at their least value, and
// the float after the greatest of them is one more boundary: the cell between
// the two (the unsafe cell) holds the u for which the cell does not fix every
// clip's code (a few weights in ten million), and a group with saliency there
// has its moments summed directly.
void int_cells(quasar::IntParams& p, int K, int bits, bool sym, int group) {
  memset(&p.cells, 0, sizeof(p.cells));
  const char* force = getenv("QUASAR_INT_PATH");
  if (force != nullptr && strcmp(force, "direct") == 0) return;
  const bool any_fit = force != nullptr && strcmp(force, "binned") == 0;
  const int qmax = sym ? (1 << (bits - 1)) - 1 : (1 << bits) - 1;
  const int q0 = sym ? -qmax : 0;
  const int nb = sym ? 2 * qmax : qmax;
  const int tie = sym ? 0 : (qmax + 1) / 2;  // step b whose thresholds are the tie cluster
  const int L = group / 16;
  {
    // at most K nb thresholds (the tie ones count once): when even that many
    // fit, or when they cannot fit at all, this is decided before any search
    const int m_upper = K * nb - (tie > 0 ? K - 2 : 0);
    const int limit = any_fit ? quasar::kCellsPerLane : quasar::kCellsPerLaneAuto;
    if ((m_upper + 1 + L - 1) / L > limit) return;
  }
  float t[quasar::kMaxClips * quasar::kCellSteps];
  int n = 0;
  float ulo = INFINITY, uhi = -INFINITY;
  for (int k = 0; k < K; k++) {
    for (int b = 1; b <= nb; b++) {
      // bracket: around the threshold of exact arithmetic, (b - q0 - qmax/2 - 1/2) / alpha
      // (symmetric: (b - Q - 1/2) / alpha), widened until it holds
      const double center = sym ? (b - qmax - 0.5) / (double)p.alpha[k]
                                : (b - 0.5 * qmax - 0.5) / (double)p.alpha[k];
      uint32_t lo = f32_order_key(-INFINITY), hi = f32_order_key(INFINITY);
      for (double half = 1e-6; half < 4.0; half *= 16.0) {
        const uint32_t a = f32_order_key((float)(center - half)), z = f32_order_key((float)(center + half));
        if (int_code(f32_from_order_key(a), p.alpha[k], qmax, sym) < q0 + b &&
            int_code(f32_from_order_key(z), p.alpha[k], qmax, sym) >= q0 + b) {
          lo = a;
          hi = z;
          break;
        }
      }
      while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (int_code(f32_from_order_key(mid), p.alpha[k], qmax, sym) >= q0 + b)
          hi = mid;
        else
          lo = mid;
      }
      t[n++] = f32_from_order_key(hi);
      if (b == tie) {
        ulo = fminf(ulo, t[n - 1]);
        uhi = fmaxf(uhi, t[n - 1]);
      }
    }
  }
  const bool merge = tie > 0 && ulo < uhi;  // more than one distinct tie threshold
  if (tie > 0 && !(ulo > -0x1p-20f && uhi < 0.0f)) return;
  float srt[quasar::kMaxClips * quasar::kCellSteps];
  int m = 0;
  for (int i = 0; i < n; i++) srt[m++] = (merge && t[i] >= ulo && t[i] <= uhi) ? ulo : t[i];
  if (merge) srt[m++] = nextafterf(uhi, INFINITY);  // the unsafe cell's upper end
  std::sort(srt, srt + m);
  m = (int)(std::unique(srt, srt + m) - srt);
  if (merge) {
    // no other threshold may fall inside the merged span
    for (int i = 0; i < m; i++)
      if (srt[i] > ulo && srt[i] <= uhi) return;
  }
  const int cpl = (m + 1 + L - 1) / L;
  if (cpl > quasar::kCellsPerLane || m + 3 > quasar::kCellThr || m > 127) return;
  if (!any_fit && cpl > quasar::kCellsPerLaneAuto) return;
  int cnt[quasar::kCellBuckets] = {0};
  int cmax = 1, below = 0;
  for (int i = 0; i < m; i++) cnt[cell_bucket(srt[i])]++;
  for (int b = 0; b < quasar::kCellBuckets; b++) {
    cmax = std::max(cmax, cnt[b]);
    p.cells.base[b] = (uint8_t)below;
    below += cnt[b];
  }
  if (cmax > 3) return;
  for (int k = 0; k < K; k++)
    for (int b = 1; b <= nb; b++) {
      float tb = t[k * nb + b - 1];
      if (merge && tb >= ulo && tb <= uhi) tb = ulo;
      p.cells.tp[k][b - 1] = (uint8_t)((std::lower_bound(srt, srt + m, tb) - srt) + 1);
    }
  for (int i = 0; i < quasar::kCellThr; i++) p.cells.thr[i] = i < m ? srt[i] : NAN;
  p.cells.cpl = cpl;
  p.cells.cmax = cmax;
  // cells count the thresholds at or below u: the unsafe cell is the one
  // just above ulo
  p.cells.unsafe_cell = merge ? (int)(std::lower_bound(srt, srt + m, ulo) - srt) + 1 : -1;
  p.cells.n_cells = m + 1;
}

// Launch the reconstruction (ema_mode 0-2) or the fused AdamW step plus
// reconstruction (ema_mode 3-4) after the arguments were validated.
int launch_path(const quasar_desc* d, const void* W, void* Wu, float* m, float* v, const void* g, int ema_mode,
                const quasar::AdamWConsts* adam, uint8_t* codes, void* scales, float* zeros, void* r, int r_bf16,
                uint8_t* best_clip, float* err, float* tensor_scale, const float* tensor_amax, float* amax_out,
                void* workspace, hipStream_t st, const quasar::BatchTable* batch = nullptr) {
  const bool w_bf16 = d->w_dtype == QUASAR_BF16;
  const int K = d->n_clips;
  const float beta2 = ema_mode >= 3 ? d->beta2 : (g ? d->beta2 : 0.0f);
  const float omb2 = 1.0f - beta2;
  hipError_t e;
  if (d->format == QUASAR_INT || d->format == QUASAR_INT_SYM) {
    const bool sym = d->format == QUASAR_INT_SYM;
    quasar::IntParams p;
    memset(&p, 0, sizeof(p));
    p.W = W;
    p.v = v;
    p.g = g;
    p.codes = codes;
    p.scales = static_cast<float*>(scales);
    p.zeros = zeros;
    p.r = r;
    p.best_clip = best_clip;
    p.err = err;
    p.n_groups = d->rows * (d->cols / d->group);
    p.beta2 = beta2;
    p.omb2 = omb2;
    p.n_clips = K;
    p.weighting = d->weighting;
    p.param_dtype = d->param_dtype;
    p.symmetric = sym;
    int_clip_tables(d, p);
    p.Wu = Wu;
    p.m = m;
    if (adam) p.adam = *adam;
    p.r_bf16 = r_bf16;
    if (batch) p.batch = *batch;
    int_cells(p, K, d->bits, sym, d->group);
    e = quasar::launch_int(p, d->bits, d->group, w_bf16, ema_mode, st);
  } else if (is_rubin(d)) {
    quasar::RubinParams p;
    memset(&p, 0, sizeof(p));
    p.W = W;
    p.v = v;
    p.g = g;
    p.codes = codes;
    p.lut = static_cast<uint8_t*>(scales);
    p.r = r;
    p.best_clip = best_clip;
    p.err = err;
    p.blocks_per_row = d->cols / 64;
    p.n_blocks = (d->rows / 8) * p.blocks_per_row;
    p.cols = d->cols;
    p.beta2 = beta2;
    p.omb2 = omb2;
    p.n_clips = K;
    p.weighting = d->weighting;
    rubin_clip_tables(d, p);
    rubin_thresholds(p, K);
    if (batch) p.batch = *batch;
    e = quasar::launch_rubin(p, w_bf16, ema_mode, st);
  } else {
    quasar::Nvfp4Params p;
    memset(&p, 0, sizeof(p));
    p.W = W;
    p.v = v;
    p.g = g;
    p.codes = codes;
    p.scales = static_cast<uint8_t*>(scales);
    p.r = r;
    p.best_clip = best_clip;
    p.err = err;
    p.tensor_scale = tensor_scale;
    p.n_blocks = d->rows * (d->cols / 16);
    p.beta2 = beta2;
    p.omb2 = omb2;
    p.n_clips = K;
    p.weighting = d->weighting;
    for (int k = 0; k < quasar::kMaxClips; k++) {
      const float f = d->clip_ratios[k < K ? k : K - 1];
      p.clip[k] = f;
      p.c6[k] = 6.0f / f;
    }
    p.Wu = Wu;
    p.m = m;
    if (adam) p.adam = *adam;
    p.r_bf16 = r_bf16;
    p.amax_out = reinterpret_cast<unsigned*>(amax_out);
    if (batch) p.batch = *batch;
    if (amax_out != nullptr) {
      e = quasar::launch_clear(p.amax_out, st);
      if (e != hipSuccess) return QUASAR_ERR_DEVICE;
    }
    if (tensor_amax != nullptr) {
      p.amax = tensor_amax;
    } else {
      unsigned* ws = static_cast<unsigned*>(workspace);
      e = quasar::launch_absmax(W, w_bf16, d->rows * d->cols, ws, st);
      if (e != hipSuccess) return QUASAR_ERR_DEVICE;
      p.amax = reinterpret_cast<const float*>(ws);
    }
    e = quasar::launch_nvfp4(p, w_bf16, ema_mode, st);
  }
  return e == hipSuccess ? QUASAR_OK : QUASAR_ERR_DEVICE;
}

}  // namespace

extern "C" {

int quasar_reconstruct(const quasar_desc* d, const void* W, float* v, const void* g, uint8_t* codes,
                       void* scales, float* zeros, void* r, uint8_t* best_clip, float* err, float* tensor_scale,
                       const float* tensor_amax, void* workspace, size_t workspace_bytes, void* stream) {
  const int s = quasar_check(d, W, v, g, codes, scales, zeros, r, best_clip, err, tensor_scale, tensor_amax,
                             workspace, workspace_bytes);
  if (s != QUASAR_OK) return s;
  const int ema_mode = g == nullptr ? 0 : (d->g_dtype == QUASAR_BF16 ? 1 : 2);
  return launch_path(d, W, nullptr, nullptr, v, g, ema_mode, nullptr, codes, scales, zeros, r,
                     d->w_dtype == QUASAR_BF16, best_clip, err, tensor_scale, tensor_amax, nullptr, workspace,
                     reinterpret_cast<hipStream_t>(stream));
}

}  // extern "C"

// ---- the entry point that allocates nothing --------------------------------
// Its scratch memory (the NVFP4 tensor absmax of a call without tensor_amax)
// is this file-scope device array, one copy per GPU, held until the process
// ends.  In host code its name is not a device address: the address is taken
// once per device with hipGetSymbolAddress and kept here.
namespace {

constexpr size_t kScratchBytes = 256;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch` (NULL on a HIP error).
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int quasar_reconstruct_noalloc(const quasar_desc* d, const void* W, float* v, const void* g, uint8_t* codes,
                               void* scales, float* zeros, void* r, uint8_t* best_clip, float* err,
                               float* tensor_scale, const float* tensor_amax, void* stream) {
  const size_t need = quasar_workspace_bytes(d, tensor_amax != nullptr);
  if (need > kScratchBytes) return QUASAR_ERR_WORKSPACE;  // more scratch than the static array holds
  void* ws = nullptr;
  if (need > 0) {
    ws = scratch_ptr();
    if (ws == nullptr) return QUASAR_ERR_DEVICE;
  }
  // the same validation and launches as quasar_reconstruct, with the static
  // array as its workspace (the absmax pass clears it with a kernel first)
  const int s = quasar_check(d, W, v, g, codes, scales, zeros, r, best_clip, err, tensor_scale, tensor_amax, ws,
                             need);
  if (s != QUASAR_OK) return s;
  const int ema_mode = g == nullptr ? 0 : (d->g_dtype == QUASAR_BF16 ? 1 : 2);
  return launch_path(d, W, nullptr, nullptr, v, g, ema_mode, nullptr, codes, scales, zeros, r,
                     d->w_dtype == QUASAR_BF16, best_clip, err, tensor_scale, tensor_amax, nullptr, ws,
                     reinterpret_cast<hipStream_t>(stream));
}

int quasar_batch_check(const quasar_desc* d, const quasar_matrix* mats, int n_mats) {
  if (d == nullptr || mats == nullptr || n_mats < 1 || n_mats > QUASAR_MAX_BATCH) return QUASAR_ERR_ARG;
  const bool ema = mats[0].g != nullptr;
  int64_t total = 0;
  for (int i = 0; i < n_mats; i++) {
    const quasar_matrix& x = mats[i];
    if ((x.g != nullptr) != ema) return QUASAR_ERR_ARG;  // one EMA mode per launch
    if (d->format == QUASAR_NVFP4 && x.tensor_amax == nullptr) return QUASAR_ERR_ARG;
    quasar_desc dd = *d;
    dd.rows = x.rows;
    dd.cols = x.cols;
    const int s = quasar_check(&dd, x.W, x.v, x.g, x.codes, x.scales, x.zeros, x.r, x.best_clip, x.err,
                               x.tensor_scale, x.tensor_amax, nullptr, 0);
    if (s != QUASAR_OK) return s;
    const int64_t upb = d->format == QUASAR_NVFP4 ? quasar::nvfp4_units_per_block()
                        : is_rubin(d)              ? quasar::rubin_units_per_block()
                                                   : quasar::int_units_per_block(d->group);
    total += (quasar_num_groups(&dd) + upb - 1) / upb;
  }
  if (total >= ((int64_t)1 << 31)) return QUASAR_ERR_SHAPE;  // one grid
  return QUASAR_OK;
}

int quasar_reconstruct_batch(const quasar_desc* d, const quasar_matrix* mats, int n_mats, void* stream) {
  const int s = quasar_batch_check(d, mats, n_mats);
  if (s != QUASAR_OK) return s;
  quasar::BatchTable bt;
  memset(&bt, 0, sizeof(bt));
  bt.n = n_mats;
  const int64_t upb = d->format == QUASAR_NVFP4 ? quasar::nvfp4_units_per_block()
                      : is_rubin(d)              ? quasar::rubin_units_per_block()
                                                 : quasar::int_units_per_block(d->group);
  for (int i = 0; i < n_mats; i++) {
    const quasar_matrix& x = mats[i];
    quasar_desc dd = *d;
    dd.rows = x.rows;
    dd.cols = x.cols;
    quasar::MatrixSlot& ms = bt.s[i];
    ms.W = x.W;
    ms.v = x.v;
    ms.g = x.g;
    ms.codes = x.codes;
    ms.scales = x.scales;
    ms.zeros = x.zeros;
    ms.r = x.r;
    ms.best_clip = x.best_clip;
    ms.err = x.err;
    ms.tensor_scale = x.tensor_scale;
    ms.amax = x.tensor_amax;
    ms.n_units = quasar_num_groups(&dd);
    ms.block0 = bt.total_blocks;
    ms.cols = x.cols;
    ms.blocks_per_row = x.cols / 64;
    bt.total_blocks += (ms.n_units + upb - 1) / upb;
  }
  // the shared fields come from the descriptor; slot 0 also fills the
  // single-matrix fields
  quasar_desc d0 = *d;
  d0.rows = mats[0].rows;
  d0.cols = mats[0].cols;
  const quasar_matrix& x = mats[0];
  const int ema_mode = x.g == nullptr ? 0 : (d->g_dtype == QUASAR_BF16 ? 1 : 2);
  return launch_path(&d0, x.W, nullptr, nullptr, x.v, x.g, ema_mode, nullptr, x.codes, x.scales, x.zeros, x.r,
                     d->w_dtype == QUASAR_BF16, x.best_clip, x.err, x.tensor_scale, x.tensor_amax, nullptr, nullptr,
                     reinterpret_cast<hipStream_t>(stream), n_mats > 1 ? &bt : nullptr);
}

int quasar_adamw_check(const quasar_desc* d, const quasar_adamw* opt, const void* W, const float* m,
                       const float* v, const void* g, const uint8_t* codes, const void* scales, const float* zeros,
                       const void* r, int r_dtype, const uint8_t* best_clip, const float* err,
                       const float* tensor_scale, const float* tensor_amax, const float* amax_out) {
  if (d == nullptr || opt == nullptr) return QUASAR_ERR_ARG;
  if (g == nullptr || m == nullptr) return QUASAR_ERR_ARG;
  // the reconstruction's own checks (pointers, alignment, the decay range,
  // here the optimiser's); the fused step always has its tensor amax, so no
  // workspace is needed
  if (d->format == QUASAR_RUBIN_INT3 || d->format == QUASAR_INT_SYM)
    return QUASAR_ERR_FORMAT;  // not fused with the optimiser step
  if (d->format == QUASAR_NVFP4 && tensor_amax == nullptr) return QUASAR_ERR_ARG;
  quasar_desc dd = *d;
  dd.beta2 = opt->beta2;
  int s = quasar_check(&dd, W, v, g, codes, scales, zeros, r, best_clip, err, tensor_scale,
                       d->format == QUASAR_NVFP4 ? tensor_amax : nullptr, nullptr, 0);
  if (s != QUASAR_OK) return s;
  if (d->format == QUASAR_INT && (tensor_amax != nullptr || amax_out != nullptr)) return QUASAR_ERR_ARG;
  // amax_out is cleared before the pass that reads tensor_amax
  if (amax_out != nullptr && amax_out == tensor_amax) return QUASAR_ERR_ARG;
  if (!aligned16(m) || !aligned16(amax_out)) return QUASAR_ERR_ALIGN;
  if (r_dtype != QUASAR_F32 && r_dtype != QUASAR_BF16) return QUASAR_ERR_FORMAT;
  if (d->w_dtype == QUASAR_BF16 && r_dtype != QUASAR_BF16) return QUASAR_ERR_FORMAT;
  if (opt->step < 1 || !(opt->eps > 0.0f) || !std::isfinite(opt->eps) || !(opt->beta1 >= 0.0f && opt->beta1 < 1.0f) ||
      !(opt->beta2 >= 0.5f && opt->beta2 < 1.0f) || !std::isfinite(opt->lr) || !(opt->lr >= 0.0f) ||
      !std::isfinite(opt->weight_decay))
    return QUASAR_ERR_ARG;
  return QUASAR_OK;
}

int quasar_adamw_reconstruct(const quasar_desc* d, const quasar_adamw* opt, void* W, float* m, float* v,
                             const void* g, uint8_t* codes, void* scales, float* zeros, void* r, int r_dtype,
                             uint8_t* best_clip, float* err, float* tensor_scale, const float* tensor_amax,
                             float* amax_out, void* stream) {
  const int s = quasar_adamw_check(d, opt, W, m, v, g, codes, scales, zeros, r, r_dtype, best_clip, err,
                                   tensor_scale, tensor_amax, amax_out);
  if (s != QUASAR_OK) return s;
  quasar_desc dd = *d;
  dd.beta2 = opt->beta2;  // the optimiser's decay updates v
  const quasar::AdamWConsts a = adamw_consts(opt);
  const int ema_mode = dd.g_dtype == QUASAR_BF16 ? 3 : 4;
  return launch_path(&dd, W, W, m, v, g, ema_mode, &a, codes, scales, zeros, r, r_dtype == QUASAR_BF16,
                     best_clip, err, tensor_scale, tensor_amax, amax_out, nullptr,
                     reinterpret_cast<hipStream_t>(stream));
}

int quasar_adamw_batch_check(const quasar_desc* d, const quasar_adamw* opt, const quasar_adamw_matrix* mats,
                             int n_mats, int r_dtype) {
  if (d == nullptr || opt == nullptr || mats == nullptr || n_mats < 1 || n_mats > QUASAR_MAX_BATCH)
    return QUASAR_ERR_ARG;
  int64_t total = 0;
  for (int i = 0; i < n_mats; i++) {
    const quasar_adamw_matrix& x = mats[i];
    quasar_desc dd = *d;
    dd.rows = x.rows;
    dd.cols = x.cols;
    const int s = quasar_adamw_check(&dd, opt, x.W, x.m, x.v, x.g, x.codes, x.scales, x.zeros, x.r, r_dtype,
                                     x.best_clip, x.err, x.tensor_scale, x.tensor_amax, x.amax_out);
    if (s != QUASAR_OK) return s;
    // every amax_out is cleared before the pass that reads the tensor_amax,
    // and each collects one matrix's maximum
    for (int k = 0; k < n_mats; k++) {
      if (x.amax_out != nullptr && x.amax_out == mats[k].tensor_amax) return QUASAR_ERR_ARG;
      if (k != i && x.amax_out != nullptr && x.amax_out == mats[k].amax_out) return QUASAR_ERR_ARG;
    }
    const int64_t upb = d->format == QUASAR_NVFP4 ? quasar::nvfp4_units_per_block()
                                                  : quasar::int_units_per_block(d->group);
    total += (quasar_num_groups(&dd) + upb - 1) / upb;
  }
  if (total >= ((int64_t)1 << 31)) return QUASAR_ERR_SHAPE;  // one grid
  return QUASAR_OK;
}

int quasar_adamw_reconstruct_batch(const quasar_desc* d, const quasar_adamw* opt,
                                   const quasar_adamw_matrix* mats, int n_mats, int r_dtype, void* stream) {
  const int s = quasar_adamw_batch_check(d, opt, mats, n_mats, r_dtype);
  if (s != QUASAR_OK) return s;
  const quasar_adamw_matrix& x0 = mats[0];
  if (n_mats == 1)
    return quasar_adamw_reconstruct(d, opt, x0.W, x0.m, x0.v, x0.g, x0.codes, x0.scales, x0.zeros, x0.r, r_dtype,
                                    x0.best_clip, x0.err, x0.tensor_scale, x0.tensor_amax, x0.amax_out, stream);
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  quasar::BatchTable bt;
  memset(&bt, 0, sizeof(bt));
  bt.n = n_mats;
  quasar::AbsmaxTable clear;  // the amax_out buffers given
  memset(&clear, 0, sizeof(clear));
  const int64_t upb =
      d->format == QUASAR_NVFP4 ? quasar::nvfp4_units_per_block() : quasar::int_units_per_block(d->group);
  for (int i = 0; i < n_mats; i++) {
    const quasar_adamw_matrix& x = mats[i];
    quasar_desc dd = *d;
    dd.rows = x.rows;
    dd.cols = x.cols;
    quasar::MatrixSlot& ms = bt.s[i];
    ms.W = x.W;
    ms.v = x.v;
    ms.g = x.g;
    ms.codes = x.codes;
    ms.scales = x.scales;
    ms.zeros = x.zeros;
    ms.r = x.r;
    ms.best_clip = x.best_clip;
    ms.err = x.err;
    ms.tensor_scale = x.tensor_scale;
    ms.amax = x.tensor_amax;
    ms.m = x.m;
    ms.Wu = x.W;
    ms.amax_out = reinterpret_cast<unsigned*>(x.amax_out);
    if (x.amax_out != nullptr) clear.out[clear.n++] = ms.amax_out;
    ms.n_units = quasar_num_groups(&dd);
    ms.block0 = bt.total_blocks;
    ms.cols = x.cols;
    ms.blocks_per_row = x.cols / 64;
    bt.total_blocks += (ms.n_units + upb - 1) / upb;
  }
  if (clear.n > 0 && quasar::launch_clear_all(clear, st) != hipSuccess) return QUASAR_ERR_DEVICE;
  // the shared fields come from the descriptor; slot 0 also fills the
  // single-matrix fields (the by-products are the slots')
  quasar_desc d0 = *d;
  d0.rows = x0.rows;
  d0.cols = x0.cols;
  d0.beta2 = opt->beta2;
  const quasar::AdamWConsts a = adamw_consts(opt);
  const int ema_mode = d0.g_dtype == QUASAR_BF16 ? 3 : 4;
  return launch_path(&d0, x0.W, x0.W, x0.m, x0.v, x0.g, ema_mode, &a, x0.codes, x0.scales, x0.zeros, x0.r,
                     r_dtype == QUASAR_BF16, x0.best_clip, x0.err, x0.tensor_scale, x0.tensor_amax, nullptr,
                     nullptr, st, &bt);
}

}  // extern "C"

extern "C" int quasar_int_path(const quasar_desc* d) {
  const int s = check_desc(d);
  if (s != QUASAR_OK) return s;
  if (is_rubin(d)) {
    quasar::RubinParams p;
    memset(&p, 0, sizeof(p));
    rubin_clip_tables(d, p);
    rubin_thresholds(p, d->n_clips);
    return p.buckets;
  }
  if (d->format != QUASAR_INT && d->format != QUASAR_INT_SYM) return QUASAR_ERR_FORMAT;
  quasar::IntParams p;
  memset(&p, 0, sizeof(p));
  int_clip_tables(d, p);
  int_cells(p, d->n_clips, d->bits, d->format == QUASAR_INT_SYM, d->group);
  return p.cells.n_cells > 0 ? 1 : 0;
}
