// int_cells_kernel.hip -- QUASAR reconstruction for INT-b groups on gfx950,
// the binned form: each weight is placed once among the code thresholds of
// all candidates, and every candidate's moments come from per-group cell sums.
//
// Algorithm 1 (Sec. 4.1.2) needs, for every clip factor f_k, the weighted
// moments sum h q, sum h q^2 and sum h q w of the RTN codes q = q_k(u)
// (Eq. rtn) of the group's normalised positions u.  Each q_k is a
// non-decreasing step function of u:
//   q_k(u) = q0 + #{b in 1..NB : u >= T(k, b)},
// with q0 = 0 and NB = qmax for asymmetric groups, q0 = -Q and NB = 2Q for
// symmetric ones, and T(k, b) the least fp32 u whose code under clip k is at
// least q0 + b.  The host finds every T(k, b) exactly, by bisection over the
// ordered fp32 values with the kernels' own fp32 code recipe, and sorts the
// distinct ones, t_0 < ... < t_{M-1}.  The cell of u is #{i : t_i <= u} in
// [0, M]; all K codes of a weight are fixed by its cell.  With
// P_b = sum of h over the weights with u >= T(k, b) (a suffix sum over cells)
// and PW_b the same sum of h w, and n = q - q0:
//   sum h n = sum_b P_b,   sum h n^2 = sum_b (2b - 1) P_b,   sum h n w = sum_b PW_b.
// So the per-weight work no longer grows with the number of clips: one
// bucket lookup and two LDS additions per weight replace K code evaluations
// and 3K moment updates.
//
// Per weight: u; its bucket among 256 equal slices of [-1, 1] (the host table
// gives the thresholds below the bucket and the next three thresholds), its
// cell, then h and h w added into the group's cell as exact int64 values
// (LDS atomics).  A group's lanes are spread over the wavefront (8 apart), so
// members of one group that hit the same cell do not serialise the atomic.
// Per group: suffix sums over the cells (each of the L lanes takes a chunk;
// the chunk totals are combined across lanes with DPP and permlane swaps),
// then each lane assembles the moments of the clips it owns from NB suffix
// sums each and solves and scores them exactly as the direct form does
// (int_common.h).
// The emitted codes are recomputed from u with the fp32 recipe, so they are
// bit-identical to the direct form's.
#include <type_traits>

#include "device_common.h"
#include "int_common.h"
#include "quasar_internal.h"

namespace quasar {
namespace {

constexpr int N = kIntN;

// Lanes of one group: spread over the wavefront (member j of a group 8 lanes
// from member j - 1), so that LDS atomics from members of one group that hit
// the same address do not serialise.
constexpr bool kSpread = true;
constexpr int kMemberStride = kSpread ? 8 : 1;

// The value x of the lane in the paired row (ROWS = 16: rows 0 <-> 1, 2 <-> 3)
// or half (ROWS = 32), at the same position, for a lane in an even row (the
// lower half) when `low` is set: the swap leaves the even rows' values in its
// first result and the odd rows' in its second.
template <int ROWS>
__device__ __forceinline__ double paired(double x, bool low) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  uint32_t alo, blo, ahi, bhi;
  swap_rows<ROWS>((uint32_t)u, alo, blo);
  swap_rows<ROWS>((uint32_t)(u >> 32), ahi, bhi);
  return low ? __longlong_as_double((long long)(((uint64_t)bhi << 32) | blo))
             : __longlong_as_double((long long)(((uint64_t)ahi << 32) | alo));
}

// Exclusive suffix sum over the members of a group: member j gets the sum of
// the values of members j+1 .. L-1.  Members 2i and 2i+1 share a row of 16
// (8 lanes apart), so member j's suffix is its row partner's value (j even)
// plus the totals of the later rows, exchanged between rows and halves
// without LDS.  The values are the chunk totals (integers rounded once to
// fp64), and the member order of the additions is fixed.
template <int L>
__device__ __forceinline__ double members_excl_suffix(double x, int j) {
  static_assert(kSpread, "members 8 lanes apart");
  const double nb = dpp_f64<kDppRor8>(x);  // member j ^ 1
  double e = (j & 1) ? 0.0 : nb;
  const double r = x + nb;                 // this row's two members
  const int row = j >> 1;                  // the group's rows in order
  const double t = paired<16>(r, (row & 1) == 0);
  if constexpr (L == 4) {
    if (row == 0) e += t;
  } else {
    const double o = paired<32>(r + t, row < 2);  // the other half's four members
    e += ((row & 1) ? 0.0 : t) + (row < 2 ? o : 0.0);
  }
  return e;
}

// x * scale rounded to an integer (ties to even), as int64, for
// |x * scale| < 2^51: x * scale + 1.5 2^52 (one fma, one rounding) lies in
// [2^52, 2^53), where its bit pattern is that of 1.5 2^52 plus the integer,
// and the low word of 1.5 2^52 is zero.
constexpr double kMagic = 6755399441055744.0;  // 1.5 * 2^52
constexpr uint32_t kMagicHi = 0x43380000u;
__device__ __forceinline__ uint64_t scaled_to_i64(double x, double scale) {
  const uint64_t b = (uint64_t)__double_as_longlong(__builtin_fma(x, scale, kMagic));
  return ((uint64_t)((uint32_t)(b >> 32) - kMagicHi) << 32) | (uint32_t)b;
}
// ... and back, correctly rounded: the high word exactly times 2^32 plus the
// low word, one rounding (sums of the cells reach 2^58)
__device__ __forceinline__ double i64_to_double(uint64_t n) {
  return __builtin_fma((double)(int32_t)(uint32_t)(n >> 32), 4294967296.0, (double)(uint32_t)n);
}

template <bool W_BF16, int EMA, int BITS, int G, bool SYM>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void int_cells_kernel(IntParams p) {
  constexpr int L = G / N;     // lanes per group
  constexpr int GPW = 64 / L;  // groups per wavefront
  constexpr int QMAX = SYM ? (1 << (BITS - 1)) - 1 : (1 << BITS) - 1;
  constexpr int NB = SYM ? 2 * QMAX : QMAX;  // code steps per clip
  constexpr int OWN = kMaxClips / L;         // clips a lane may own
  static_assert(kThreads == kCellBuckets && kThreads == kMaxClips * kCellSteps, "one table entry per thread");
  static_assert((size_t)int_stage_bytes<kSpread, G>() == int_cells_stage_bytes(G), "the launch sizes the stage");

  extern __shared__ __align__(16) double s_hist[];  // [wave][group slot][cell][h, h w], or the store stage
  __shared__ uint4 s_bucket[kCellBuckets];
  __shared__ uint8_t s_tp[kMaxClips * kCellSteps];
  __shared__ float s_alpha[kMaxClips], s_clip[kMaxClips];
  __shared__ float s_win[kThreads / 64][GPW][4];

  using M = Members<L, kSpread>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_index();
  const int j = M::member(lane), slot = M::slot(lane);
  const int K = p.n_clips;

  {  // the tables, read from the kernel-argument segment with per-lane indices
    const IntCells& cl = kernarg_params<IntParams>()->cells;
    const int c = cl.base[tid];
    s_bucket[tid] = make_uint4((uint32_t)c, as_u32(cl.thr[c]), as_u32(cl.thr[c + 1]), as_u32(cl.thr[c + 2]));
    s_tp[tid] = (&cl.tp[0][0])[tid];
  }
  if (tid < kMaxClips) {
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

  // this wavefront's LDS: its groups' cells, before that the stage of the
  // EMA's store, and after them the stage of the exact path and of r's store
  const int cpl = p.cells.cpl;
  double* const s_wave = s_hist + (size_t)wave * (int_cells_wave_bytes(G, cpl) / sizeof(double));
  const WaveImage im = int_image<L>(s_wave, wave_g0, mtx.n_groups, slot, j, lane);

  WRegs<W_BF16> wr;
  float v[N];
  int_load<W_BF16, EMA, kSpread, G>(p, mtx, im, e0, wr, v);
  const IntRange rg = int_range<L, SYM, W_BF16, kSpread>(wr);

  // ---- this group's cells: lane j owns cells [j cpl, (j + 1) cpl) -----------
  // Groups are int_cells_stride(cpl) cells apart, an odd number, so that the
  // same cell of the wavefront's groups falls in different LDS banks.  The
  // wavefront clears its whole area, 16 bytes per lane and step.
  double* hist = s_wave + (size_t)slot * int_cells_stride<L>(cpl) * 2;
  double* mine = hist + 2 * j * cpl;
  {
    const int n16 = GPW * int_cells_stride<L>(cpl);
    uint4* z = reinterpret_cast<uint4*>(s_wave);
#pragma unroll 1
    for (int i = lane; i < n16; i += 64) z[i] = make_uint4(0u, 0u, 0u, 0u);
  }

  // ---- h and h w of every weight into its cell, as exact integers --------------
  // h and h w are scaled by powers of two that bring the group's largest |h|
  // and |h| max|w| below 2^B, B = 51, rounded to integers and added as int64:
  // every cell sum is exact (below 2^58), whatever the order of the atomics,
  // and is rounded once to fp64 in the scan.  Clips whose codes agree on the
  // whole group get bit-identical moments, so their scores tie exactly and the
  // lowest index wins, as in the exact definition.  A term loses at most
  // 2^-52 of the largest one; the fit below checks what that can do to it.
  constexpr int B = 51;
  float hmax = 0.0f;
#pragma unroll
  for (int i = 0; i < N; i++) hmax = fmaxf(hmax, v[i]);
  hmax = M::max(hmax);
  const float wabs = SYM ? rg.mx : fmaxf(fabsf(rg.mn), fabsf(rg.mx));
  // 2^eh > hmax and 2^ew > max |w| (frexp exponents)
  const int eh = __builtin_amdgcn_frexp_expf(hmax), ew = __builtin_amdgcn_frexp_expf(wabs);
  const double sh = __builtin_amdgcn_ldexp(1.0, B - eh), shw = __builtin_amdgcn_ldexp(1.0, B - eh - ew);
  double Svww = 0.0;
  wave_lds_fence();  // the cells are clear

  // ---- the cell of every weight (four bucket reads in flight at a time) -----
  // Thresholds outside u's bucket lie on the far side of u and the table's
  // padding is NaN, so cmax compares never pass the last threshold.
  uint32_t cells[N / 4];  // four cells per register, one byte each
  auto bin = [&](auto cmax_tag) {
    constexpr int C = decltype(cmax_tag)::value;
#pragma unroll
    for (int c4 = 0; c4 < N / 4; c4++) {
      float u[4];
      uint4 e[4];
#pragma unroll
      for (int t = 0; t < 4; t++) {
        u[t] = int_u<SYM>(wr.get(4 * c4 + t), rg);
        e[t] = s_bucket[cell_bucket(u[t])];
      }
      uint32_t packed = 0;
#pragma unroll
      for (int t = 0; t < 4; t++) {
        uint32_t cell = e[t].x + (u[t] >= as_f32(e[t].y) ? 1u : 0u);
        if constexpr (C > 1) cell += (u[t] >= as_f32(e[t].z) ? 1u : 0u);
        if constexpr (C > 2) cell += (u[t] >= as_f32(e[t].w) ? 1u : 0u);
        packed |= cell << (8 * t);
      }
      cells[c4] = packed;
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  const int cmax = p.cells.cmax;
  if (cmax == 1)
    bin(std::integral_constant<int, 1>{});
  else if (cmax == 2)
    bin(std::integral_constant<int, 2>{});
  else
    bin(std::integral_constant<int, 3>{});

  // ---- h and h w of every weight into its cell --------------------------------
#pragma unroll
  for (int i = 0; i < N; i++) {
    const int cell = (int)((cells[i >> 2] >> (8 * (i & 3))) & 0xffu);
    const double V = (double)v[i], Wd = (double)wr.get(i);
    const double VW = V * Wd;
    Svww = __builtin_fma(VW, Wd, Svww);
    uint64_t* c64 = reinterpret_cast<uint64_t*>(hist + 2 * cell);
    __hip_atomic_fetch_add(c64, scaled_to_i64(V, sh), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
    __hip_atomic_fetch_add(c64 + 1, scaled_to_i64(VW, shw), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
  }
  wave_lds_fence();

  // A weight among merged thresholds (rare) lies in the unsafe cell, where the
  // cell does not fix every clip's code: its group takes the exact path below
  // unless its saliency is 0 (h >= 0, so the cell's sum of h is 0 exactly when
  // every weight in it has h = 0, and those weights add nothing to any moment).
  const int ucell = p.cells.unsafe_cell;
  // (read with the suffix pass's access type, which then cannot move above it)
  const bool group_unsafe = ucell >= 0 && reinterpret_cast<const ulonglong2*>(hist)[ucell].x != 0;

  // ---- suffix sums over the cells (exact integer cells, rounded once to fp64):
  // the chunk totals first, then the members above this one, then a second
  // pass that writes the suffix sums.  The lane's cells are read four at a
  // time, all four reads in flight before the first is used; an index past
  // the lane's last cell reads that cell again and contributes nothing, and
  // in the second pass (from the top down) its write to that cell comes
  // before the cell's own.
  {
    // one access type for the reads and the writes: the writes may not be
    // moved above reads of the same cell
    ulonglong2* mc = reinterpret_cast<ulonglong2*>(mine);
    uint64_t ih = 0, iw = 0;  // exact integer chunk totals
#pragma unroll 1
    for (int b = 0; b < cpl; b += 4) {
      ulonglong2 t[4];
#pragma unroll
      for (int c = 0; c < 4; c++) t[c] = mc[min(b + c, cpl - 1)];
#pragma unroll
      for (int c = 0; c < 4; c++) {
        const bool in = b + c < cpl;
        ih += in ? t[c].x : 0ull;
        iw += in ? t[c].y : 0ull;
      }
    }
    double eh2 = members_excl_suffix<L>(i64_to_double(ih), j), ew2 = members_excl_suffix<L>(i64_to_double(iw), j);
#pragma unroll 1
    for (int b = (cpl - 1) & ~3; b >= 0; b -= 4) {
      ulonglong2 t[4];
#pragma unroll
      for (int c = 0; c < 4; c++) t[c] = mc[min(b + c, cpl - 1)];
#pragma unroll
      for (int c = 3; c >= 0; c--) {
        const bool in = b + c < cpl;
        eh2 += in ? i64_to_double(t[c].x) : 0.0;
        ew2 += in ? i64_to_double(t[c].y) : 0.0;
        mc[min(b + c, cpl - 1)] = make_ulonglong2((unsigned long long)__double_as_longlong(eh2),
                                                  (unsigned long long)__double_as_longlong(ew2));
      }
    }
  }
  wave_lds_fence();

  // back from the integer scale (exact: powers of two)
  const double rsh = __builtin_amdgcn_ldexp(1.0, eh - B), rshw = __builtin_amdgcn_ldexp(1.0, eh + ew - B);
  IntMoments mo;
  {
    const double2 tot = *reinterpret_cast<const double2*>(hist);  // cell 0's suffix: the whole group
    mo.Sv = tot.x * rsh;
    mo.Svw = tot.y * rshw;
  }
  mo.Svww = M::sum(Svww);
  mo.thr = 1e-12 * mo.Sv * mo.Sv * (double)QMAX * (double)QMAX;
  mo.rSv = rcp_f64(mo.Sv);
  // each term of sum h and of sum h w is off by at most half a unit of its
  // fixed point; the sums and the fit's products carry fp64 roundings
  mo.qh = 0.5 * (double)G * rsh;
  mo.qhw = 0.5 * (double)G * rshw;
  mo.rel = 0x1p-47;
  mo.wabs = (double)wabs;
  int_fit_bounds<QMAX>(mo);

  // ---- the clips this lane owns: moments from NB suffix sums ------------------
  auto moments = [&](int k, double& A0, double& A1, double& A2) {
    A0 = A1 = A2 = 0.0;
    const uint4 tw4 = *reinterpret_cast<const uint4*>(s_tp + k * kCellSteps);
    const uint32_t tw[4] = {tw4.x, tw4.y, tw4.z, tw4.w};
#pragma unroll
    for (int b = 1; b <= NB; b++) {
      const int c = (int)((tw[(b - 1) >> 2] >> (8 * ((b - 1) & 3))) & 0xffu);
      const double2 s = *reinterpret_cast<const double2*>(hist + 2 * c);
      A0 += s.x;
      A1 = __builtin_fma((double)(2 * b - 1), s.x, A1);
      A2 += s.y;
    }
    A0 *= rsh;
    A1 *= rsh;
    A2 *= rshw;
    if constexpr (SYM) {  // q = n - Q
      A1 = __builtin_fma((double)QMAX * (double)QMAX, mo.Sv, __builtin_fma(-2.0 * (double)QMAX, A0, A1));
      A2 = __builtin_fma(-(double)QMAX, mo.Svw, A2);
    }
  };

  // Selection.  With fp32 (s, z) the candidate's score is that of its exact
  // fit up to the fp32 rounding of (s, z), a relative 1e-12 or so; the exact
  // fit's score is C - num^2 / (Sv D) (asymmetric: num = Sv A2 - A0 Svw,
  // D = Sv A1 - A0^2; symmetric: C - A2^2 / A1), with C the same for every
  // clip.  So each lane ranks its clips by num^2 / D (cross-multiplied, ties
  // to the lowest index), fits and scores only its best one, and the group's
  // argmin runs over keys made from D / num^2.  Groups with a clip whose fit
  // degenerates (no saliency, all of it on one code), and deployed
  // precisions other than fp32, score every clip (int_fit_score).  A group
  // with a clip whose fit the moments cannot fix accurately enough
  // (int_fit_ill), or with a weight among merged thresholds, evaluates every
  // clip straight from its weights (int_exact_all).
  IntBest best = int_best_init();
  bool full = p.param_dtype != 0;
  bool ill = group_unsafe;
  int bk = -1;
  double bn = 0.0, bd = 1.0;
  if (!full && !group_unsafe) {
    // unrolled: the clips' LDS reads and fp64 chains interleave
#pragma unroll
    for (int t = 0; t < OWN; t++) {
      const int k = j + L * t;
      if (k < K) {
        double A0, A1, A2;
        moments(k, A0, A1, A2);
        ill |= int_fit_ill<SYM, QMAX>(mo, A0, A1, A2);
        const double D = SYM ? A1 : mo.Sv * A1 - A0 * A0;
        const double num = SYM ? A2 : mo.Sv * A2 - A0 * mo.Svw;
        const bool degenerate = SYM ? (A1 == 0.0) : (mo.Sv == 0.0 || D <= mo.thr);
        const double n2 = num * num;
        if (degenerate) {
          full = true;
        } else if (bk < 0 || n2 * bd > bn * D) {
          bk = k;
          bn = n2;
          bd = D;
        }
      }
    }
  }
  ill = M::max(ill ? 1.0f : 0.0f) > 0.0f;
  if (!ill) {
    if (M::max(full ? 1.0f : 0.0f) > 0.0f) {
#pragma unroll 1
      for (int t = 0; t < OWN; t++) {
        const int k = j + L * t;
        if (k < K) {
          double A0, A1, A2;
          moments(k, A0, A1, A2);
          int_fit_score<SYM, QMAX>(p, k, s_clip[k], rg, mo, A0, A1, A2, best);
        }
      }
      ill = M::max(best.ill ? 1.0f : 0.0f) > 0.0f;
    } else if (bk >= 0) {
      double b0, b1, b2;
      moments(bk, b0, b1, b2);
      int_fit_score<SYM, QMAX>(p, bk, s_clip[bk], rg, mo, b0, b1, b2, best);
      // rank by D / num^2 (num = 0: the worst fit, kept finite)
      best.key = make_key(fmin(bd * rcp_f64(bn), 1e300), bk);
    }
  }
  {
    // The wavefront's cell areas are no longer needed: they stage the
    // flagged groups.  A member lane reads its saliencies again: v' when this
    // kernel stored it, written by another lane of this wavefront, which the
    // workgroup-scope fences make visible (the workgroup's waves share the
    // compute unit's vector cache).
    auto load_h = [&](float (&hv)[N]) {
      if constexpr (EMA != 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      }
      load16<false>(mtx.v, e0, hv);
#pragma unroll
      for (int i = 0; i < N; i++) hv[i] = weight_of(hv[i], p.weighting);
    };
    int_exact_wave<L, SYM, QMAX, kSpread, W_BF16>(p, wr, load_h, rg, s_alpha, s_clip, lane,
                                                  ill && active && !rg.constant, reinterpret_cast<float*>(s_wave),
                                                  best);
  }

  int_finish<W_BF16, BITS, G, SYM, kSpread>(p, mtx, wr, rg, mo.Sv, best, s_alpha, s_win[wave][slot], j, gid, im,
                                         active);
}

template <bool W_BF16, int EMA, int BITS, int G>
hipError_t launch_g(const IntParams& p, hipStream_t s) {
  constexpr int64_t groups_per_block = int_units_per_block(G);
  const int64_t blocks =
      p.batch.n > 1 ? p.batch.total_blocks : (p.n_groups + groups_per_block - 1) / groups_per_block;
  const size_t lds = int_cells_lds_bytes(G, p.cells.cpl);
  const dim3 grid((unsigned)blocks), block(kThreads);
  if (p.symmetric) {
    if constexpr (EMA <= 2) {
      hipLaunchKernelGGL((int_cells_kernel<W_BF16, EMA, BITS, G, true>), grid, block, lds, s, p);
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  hipLaunchKernelGGL((int_cells_kernel<W_BF16, EMA, BITS, G, false>), grid, block, lds, s, p);
  return hipGetLastError();
}

template <bool W_BF16, int EMA, int BITS>
hipError_t launch_b(const IntParams& p, int group, hipStream_t s) {
  return group == 64 ? launch_g<W_BF16, EMA, BITS, 64>(p, s) : launch_g<W_BF16, EMA, BITS, 128>(p, s);
}

template <bool W_BF16, int EMA>
hipError_t launch_e(const IntParams& p, int bits, int group, hipStream_t s) {
  switch (bits) {
    case 2: return launch_b<W_BF16, EMA, 2>(p, group, s);
    case 3: return launch_b<W_BF16, EMA, 3>(p, group, s);
    default: return launch_b<W_BF16, EMA, 4>(p, group, s);
  }
}

template <bool W_BF16>
hipError_t launch_w(const IntParams& p, int bits, int group, int ema_mode, hipStream_t s) {
  switch (ema_mode) {
    case 1: return launch_e<W_BF16, 1>(p, bits, group, s);
    case 2: return launch_e<W_BF16, 2>(p, bits, group, s);
    case 3: return launch_e<W_BF16, 3>(p, bits, group, s);
    case 4: return launch_e<W_BF16, 4>(p, bits, group, s);
    default: return launch_e<W_BF16, 0>(p, bits, group, s);
  }
}

}  // namespace

hipError_t launch_int_cells(const IntParams& p, int bits, int group, bool w_bf16, int ema_mode, hipStream_t s) {
  return w_bf16 ? launch_w<true>(p, bits, group, ema_mode, s) : launch_w<false>(p, bits, group, ema_mode, s);
}

}  // namespace quasar
