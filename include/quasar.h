/*
 * quasar.h -- C ABI of libquasar.so: QUASAR's per-step loss-aware weight
 * reconstruction (arXiv 2608.13966) as HIP kernels for MI355X (gfx950).
 *
 * One call reconstructs one weight matrix W [rows = out, cols = in], row-major,
 * with quantisation groups running along a row (Sec. 3.1: "each row ... is
 * partitioned into groups"; App. B: groups run along the input dimension).
 * For every group it takes the saliency h (Sec. 4.1.1: the EMA of squared
 * gradients, AdamW's second moment v; optionally updated in the same pass from
 * the current gradient g as v = beta2*v + (1-beta2)*g^2, App. A.2), then runs
 * Algorithm 1 (Sec. 4.1.2): for each clip factor f in F, RTN codes on the range
 * [c - f*rho, c + f*rho] (Eq. rtn), the saliency-weighted least-squares
 * dequantiser (s, z) (Eq. ridgefit) and its score sum h (s q + z - w)^2
 * (Eq. fisher-obj); the argmin is kept and emitted as codes, scale, zero and
 * the reconstruction r = s q + z.  NVFP4 (Sec. 4.2) uses 16-element blocks of
 * E2M1 codes, an E4M3 block scale fitted to the same objective (scale only,
 * no zero-point) and an fp32 tensor scale from the tensor absmax.
 *
 * Conventions
 *  - Every data pointer is HIP device memory owned by the caller, except
 *    desc->clip_ratios, which is a host array read during the call.
 *  - The library allocates no memory and keeps no state between calls; it is
 *    reentrant.  Work is enqueued on `stream` (a hipStream_t; NULL = the null
 *    stream) and the call returns without waiting; results are valid once the
 *    caller has synchronised that stream.
 *  - Argument errors are detected on the host before anything is launched; a
 *    call that returns an error has written nothing.  QUASAR_ERR_DEVICE reports
 *    a launch failure; faults during execution surface at the caller's sync.
 *  - Every device pointer must be 16-byte aligned.
 *  - v >= 0 is a precondition (saliency is non-negative, Alg. 1 input); it is
 *    not checked.  NaN or Inf inputs give unspecified (but in-bounds) results.
 *
 * Output layouts (the paper fixes none; these are this library's):
 *  - codes: groups in row-major order, each group's codes contiguous:
 *      INT4 / NVFP4: two per byte, even element in the low nibble;
 *      INT2: four per byte, element 4k+j at bits 2j;
 *      INT3: per group a little-endian bit stream, code i at bits [3i, 3i+3)
 *            (48 bytes per 128-group, 24 per 64-group).
 *    NVFP4 code = (sign << 3) | magnitude index, magnitudes 0, 0.5, 1, 1.5, 2,
 *    3, 4, 6; zero is always +0.
 *  - INT: scales = fp32 s, zeros = fp32 z, one each per group ([rows, cols/group]);
 *    with param_dtype F16/BF16 they hold values exactly representable there.
 *  - NVFP4: scales = one E4M3FN byte per 16-block ([rows, cols/16]); zeros unused;
 *    tensor_scale = one fp32 S_t; the block's dequantiser is S_t * e4m3.
 *  - RUBIN_INT3: blocks in row-major order over [rows/8, cols/64]; codes =
 *    192 bytes per block, the INT3 bit stream of its 512 indices in row-major
 *    order inside the block (element (i, j) of the block is index 64 i + j);
 *    scales = the codebook, 8 E4M3FN bytes per block (entry k at byte k, zero
 *    is +0); zeros and tensor_scale unused; r = codebook[index].
 *  - r: [rows, cols] in W's dtype (fp32 r = fmaf(s, q, z); bf16 = its
 *    round-to-nearest-even).  A constant group (min = max) has codes 0,
 *    s = 0 and z = its value in the deployed precision.
 *  - best_clip: u8 index into clip_ratios per group; err: fp32 score of the
 *    chosen candidate per group.
 */
#ifndef QUASAR_H
#define QUASAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  QUASAR_OK = 0,
  QUASAR_ERR_ARG = -1,       /* NULL required pointer, n_clips, clip ratio or beta2 out of range */
  QUASAR_ERR_SHAPE = -2,     /* rows/cols < 1, cols % group != 0, too many groups */
  QUASAR_ERR_ALIGN = -3,     /* a device pointer is not 16-byte aligned */
  QUASAR_ERR_FORMAT = -4,    /* unsupported format / bits / group / dtype */
  QUASAR_ERR_WORKSPACE = -5, /* workspace missing or smaller than quasar_workspace_bytes() */
  QUASAR_ERR_DEVICE = -6     /* HIP reported an error when launching */
} quasar_status;

typedef enum { QUASAR_F32 = 0, QUASAR_BF16 = 1, QUASAR_F16 = 2 } quasar_dtype;

/* Saliency weighting of the objective (Eq. fisher-obj) and of the fit:
 * QUASAR_WEIGHT_H    h = v, the method's default (Sec. 4.1.1);
 * QUASAR_WEIGHT_H2   h = v*v in fp32, the squared weighting compared in App. A.3;
 * QUASAR_WEIGHT_NONE h = 1, the "scale search only" ablation of Table 5
 *                    (plain least-squares fit, unweighted score). */
typedef enum { QUASAR_WEIGHT_H = 0, QUASAR_WEIGHT_H2 = 1, QUASAR_WEIGHT_NONE = 2 } quasar_weighting;
/* QUASAR_INT: asymmetric INT-b groups with (s, z) (Sec. 3.1, Alg. 1);
 * QUASAR_NVFP4: 16-blocks of E2M1 with E4M3 block scales (Sec. 4.2);
 * QUASAR_RUBIN_INT3: the Rubin INT3 lookup-table format (App. B, Eq. rubin-fit):
 *   blocks of 8 rows x 64 columns (rows % 8 == 0, cols % 64 == 0; desc->bits
 *   = 3, desc->group = 512), 3-bit indices and an 8-entry E4M3 codebook per
 *   block, each entry the saliency-weighted mean of its weights rounded to E4M3
 *   (an index without saliency mass keeps the E4M3 value of its grid level). */
/* QUASAR_INT_SYM: symmetric INT-b groups (Sec. 4.1.2 notes that symmetric
 *   quantisation has a closed form like Eq. ridgefit): r = s q with q in
 *   [-Q, Q], Q = 2^(b-1) - 1, codes on the range [-f m, f m] (m = the group's
 *   max |w|; fp32: q = clamp(rint((w * (1/m)) * (Q/f)), -Q, Q)), the scale
 *   s = sum h q w / sum h q^2 (the RTN scale f m / Q when that sum is 0),
 *   stored codes in b-bit two's complement; zeros may be NULL (else written 0);
 *   an all-zero group has s = 0.  Not available in quasar_adamw_reconstruct. */
typedef enum { QUASAR_INT = 0, QUASAR_NVFP4 = 1, QUASAR_RUBIN_INT3 = 2, QUASAR_INT_SYM = 3 } quasar_format;

#define QUASAR_MAX_CLIPS 16

typedef struct {
  int64_t rows;               /* out features, >= 1 */
  int64_t cols;               /* in features, >= 1, multiple of group */
  int32_t w_dtype;            /* quasar_dtype of W and of r */
  int32_t format;             /* quasar_format */
  int32_t bits;               /* INT, INT_SYM: 2, 3 or 4 (INT: qmax = 2^bits - 1); RUBIN_INT3: 3;
                                 ignored for NVFP4 */
  int32_t group;              /* INT, INT_SYM: 64 or 128; NVFP4: 16; RUBIN_INT3: 512 (8 x 64) */
  const float* clip_ratios;   /* HOST array of n_clips factors, each in (0, 1]; order breaks ties
                                 (the lowest index wins among equal scores) */
  int32_t n_clips;            /* 1 .. QUASAR_MAX_CLIPS */
  int32_t g_dtype;            /* quasar_dtype of g when g != NULL (F32 or BF16) */
  float beta2;                /* EMA decay when g != NULL, in [0.5, 1) */
  int32_t weighting;          /* quasar_weighting; 0 = QUASAR_WEIGHT_H */
  int32_t param_dtype;        /* INT: precision the dequantiser (s, z) is deployed in,
                                 QUASAR_F32 (0), QUASAR_F16 or QUASAR_BF16.  s and z are
                                 rounded (from fp32, to nearest even) before r is formed
                                 and before the candidate is scored, so r is exactly what
                                 the deployed model computes (Sec. 3.1: the result deploys
                                 as an ordinary RTN-quantised model).  The scales/zeros
                                 buffers stay fp32 and hold the rounded values.
                                 NVFP4: must be QUASAR_F32. */
} quasar_desc;

/*
 * Reconstruct one matrix (Alg. 1 for every group; Sec. 4.2 for NVFP4).
 *
 *  W            [rows, cols] in desc->w_dtype (read)
 *  v            [rows, cols] fp32 saliency.  Read only when g == NULL.  When g
 *               != NULL it is read and overwritten in place with
 *               v' = fmaf(beta2, v, (1 - beta2) * (g * g)) (fp32, this order), and
 *               v' is the saliency used.
 *  g            [rows, cols] gradient in desc->g_dtype, or NULL (no EMA)
 *  codes        packed codes, quasar_codes_bytes(desc) bytes (required)
 *  scales       INT: fp32 [rows, cols/group]; NVFP4: u8 E4M3 [rows, cols/16];
 *               RUBIN_INT3: u8 E4M3 codebook [blocks, 8] (required)
 *  zeros        INT: fp32 [rows, cols/group] (required); NVFP4, RUBIN_INT3: unused, pass NULL
 *  r            [rows, cols] in w_dtype, or NULL to skip writing r (export only)
 *  best_clip    u8 [groups] or NULL;  err  fp32 [groups] or NULL
 *  tensor_scale NVFP4: fp32 [1] output S_t = amax / 2688 (required); INT: NULL
 *  tensor_amax  NVFP4: optional fp32 [1] input, the tensor absmax (e.g. tracked
 *               by the optimiser); NULL = computed here with an extra pass over W.
 *               INT: NULL.
 *  workspace    device scratch of at least quasar_workspace_bytes(desc) bytes, or
 *               NULL when that size is 0.  Not read before it is written.
 *  stream       hipStream_t to enqueue on.
 * Returns a quasar_status.
 */
int quasar_reconstruct(const quasar_desc* desc, const void* W, float* v, const void* g,
                       uint8_t* codes, void* scales, float* zeros, void* r, uint8_t* best_clip,
                       float* err, float* tensor_scale, const float* tensor_amax, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * quasar_reconstruct for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments and results without the workspace, whose
 * role a library-owned static device array of 256 bytes per GPU takes (held
 * until the process ends).  Only NVFP4 without tensor_amax uses it; a call
 * that would need more than 256 bytes returns QUASAR_ERR_WORKSPACE.  The call
 * itself allocates nothing (no hipMalloc, no allocating library routine);
 * the array's address is looked up once per device.  Every call on a GPU
 * shares that GPU's array: calls that overlap on one GPU (other streams,
 * other threads) race on it and must be serialised by the caller.  Returns a
 * quasar_status; QUASAR_ERR_DEVICE also when the array's address cannot be
 * obtained.
 */
int quasar_reconstruct_noalloc(const quasar_desc* desc, const void* W, float* v, const void* g, uint8_t* codes,
                               void* scales, float* zeros, void* r, uint8_t* best_clip, float* err,
                               float* tensor_scale, const float* tensor_amax, void* stream);

/*
 * Tensor absmax for NVFP4 (Sec. 4.2: the fp32 tensor scale is set from the
 * tensor's absolute maximum).  Writes max |W| over the whole matrix, as fp32,
 * to amax_out (device, 1 float, 16-byte aligned), for use as the tensor_amax
 * argument of quasar_reconstruct.  desc->format must be QUASAR_NVFP4 (the
 * descriptor's clip fields are validated but unused).  Asynchronous on stream.
 */
int quasar_absmax(const quasar_desc* desc, const void* W, float* amax_out, void* stream);

/*
 * One optimiser step fused with the reconstruction of its result.
 *
 * Every method in the paper trains its latent weights with AdamW (Sec. 6.1),
 * and QUASAR's saliency is AdamW's own second moment (Sec. 4.1.1); at every
 * step the updated latent weights are reconstructed for the next forward pass
 * (Sec. 3.1, Alg. 1).  This call does both in one pass over memory: per
 * element, in fp32 and in this order,
 *     m' = fmaf(beta1, m, (1 - beta1) g)
 *     v' = fmaf(beta2, v, (1 - beta2) (g g))
 *     W' = fmaf(-lr / (1 - beta1^t), m' / fmaf(sqrtf(v'), 1 / sqrt(1 - beta2^t), eps),
 *               W (1 - lr weight_decay))
 * (decoupled weight decay, bias-corrected; 1 - beta in fp32, the three
 * step constants in fp64 then rounded to fp32; sqrtf and the quotient
 * correctly rounded; a bf16 W' is rounded to nearest even), then the
 * reconstruction of W' with saliency v' exactly as quasar_reconstruct
 * (desc->weighting and desc->param_dtype apply; desc->beta2 is ignored).
 */
typedef struct {
  float lr;            /* learning rate, finite, >= 0 */
  float beta1;         /* first-moment decay, in [0, 1) */
  float beta2;         /* second-moment decay, in [0.5, 1) */
  float eps;           /* > 0 */
  float weight_decay;  /* decoupled, finite */
  int64_t step;        /* t >= 1, the step being taken (bias corrections) */
} quasar_adamw;

/*
 *  W            [rows, cols] latent weights in desc->w_dtype, updated in place
 *  m, v         [rows, cols] fp32 optimiser moments, updated in place
 *  g            [rows, cols] gradient in desc->g_dtype (required)
 *  codes, scales, zeros, best_clip, err, tensor_scale: as quasar_reconstruct
 *  r            [rows, cols] or NULL, in r_dtype: QUASAR_BF16 (any W) or
 *               QUASAR_F32 (fp32 W only)
 *  tensor_amax  NVFP4: required, the amax the tensor scale of this step is
 *               taken from (e.g. last step's amax_out); the updated tensor's
 *               own absmax is not known before the pass.  INT: NULL.
 *  amax_out     NVFP4: optional device fp32, receives max |W'| for the next
 *               step (cleared and filled by the call); not the tensor_amax
 *               buffer (QUASAR_ERR_ARG).  INT: NULL.
 * No workspace is needed.  Returns a quasar_status; on error nothing is
 * launched and W, m, v are untouched.
 */
int quasar_adamw_reconstruct(const quasar_desc* desc, const quasar_adamw* opt, void* W, float* m, float* v,
                             const void* g, uint8_t* codes, void* scales, float* zeros, void* r, int r_dtype,
                             uint8_t* best_clip, float* err, float* tensor_scale, const float* tensor_amax,
                             float* amax_out, void* stream);

/* Host-only validation: the status quasar_adamw_reconstruct would return for
 * these arguments (desc->beta2 is ignored, as there). */
int quasar_adamw_check(const quasar_desc* desc, const quasar_adamw* opt, const void* W, const float* m,
                       const float* v, const void* g, const uint8_t* codes, const void* scales,
                       const float* zeros, const void* r, int r_dtype, const uint8_t* best_clip,
                       const float* err, const float* tensor_scale, const float* tensor_amax,
                       const float* amax_out);

/*
 * Several matrices in one launch (e.g. the seven projections of a
 * transformer layer): the same computation as one quasar_reconstruct per
 * matrix, with identical results, but a single grid, so small matrices do not
 * each pay a launch and the tail of one overlaps the others.
 *
 * desc gives everything the matrices share (format, bits, group, clips,
 * dtypes, beta2, weighting, param_dtype); its rows/cols are ignored.  Each
 * quasar_matrix gives a matrix's shape and buffers, with the meaning and
 * requirements of the same-named quasar_reconstruct arguments.  Either every
 * g is NULL or none is.  NVFP4 needs every tensor_amax (no workspace path).
 * 1 <= n_mats <= QUASAR_MAX_BATCH.  Returns a quasar_status; on error nothing
 * is launched.
 */
#define QUASAR_MAX_BATCH 16
typedef struct {
  int64_t rows, cols;
  const void* W;
  float* v;
  const void* g;
  uint8_t* codes;
  void* scales;
  float* zeros;
  void* r;
  uint8_t* best_clip;
  float* err;
  float* tensor_scale;
  const float* tensor_amax;
} quasar_matrix;

int quasar_reconstruct_batch(const quasar_desc* desc, const quasar_matrix* mats, int n_mats, void* stream);

/* Host-only validation: the status quasar_reconstruct_batch would return. */
int quasar_batch_check(const quasar_desc* desc, const quasar_matrix* mats, int n_mats);

/*
 * The fused AdamW step and reconstruction of quasar_adamw_reconstruct over
 * several matrices in one launch (e.g. the seven projections of a transformer
 * layer), with the same results as one call per matrix.  desc, opt and r_dtype
 * are shared (desc's rows/cols and beta2 are ignored); each
 * quasar_adamw_matrix gives a matrix's shape and buffers with the meaning and
 * requirements of the same-named quasar_adamw_reconstruct arguments (W is
 * updated in place).  Every amax_out given is cleared before the pass, so none
 * may be any matrix's tensor_amax, and no two may be the same buffer.
 * 1 <= n_mats <= QUASAR_MAX_BATCH.  Returns a quasar_status; on error nothing
 * is launched.
 */
typedef struct {
  int64_t rows, cols;
  void* W;
  float* m;
  float* v;
  const void* g;
  uint8_t* codes;
  void* scales;
  float* zeros;
  void* r;
  uint8_t* best_clip;
  float* err;
  float* tensor_scale;
  const float* tensor_amax;
  float* amax_out;
} quasar_adamw_matrix;

int quasar_adamw_reconstruct_batch(const quasar_desc* desc, const quasar_adamw* opt,
                                   const quasar_adamw_matrix* mats, int n_mats, int r_dtype, void* stream);

/* Host-only validation: the status quasar_adamw_reconstruct_batch would return. */
int quasar_adamw_batch_check(const quasar_desc* desc, const quasar_adamw* opt, const quasar_adamw_matrix* mats,
                             int n_mats, int r_dtype);

/*
 * Tensor absmax (Sec. 4.2, as quasar_absmax) of up to QUASAR_MAX_BATCH NVFP4
 * matrices in one launch, e.g. ahead of quasar_reconstruct_batch.  Of each
 * quasar_matrix only rows, cols and W are read (desc gives the format and W's
 * dtype).  amax_out is a host array of n_mats device pointers (each 16-byte
 * aligned, 1 fp32): amax_out[i] receives max |W| of mats[i] (cleared first,
 * then filled by the pass); no two of them may be the same buffer
 * (QUASAR_ERR_ARG).  Asynchronous on stream; on error nothing is launched.
 */
int quasar_absmax_batch(const quasar_desc* desc, const quasar_matrix* mats, int n_mats, float* const* amax_out,
                        void* stream);

/* Host-only validation: the status quasar_absmax_batch would return. */
int quasar_absmax_batch_check(const quasar_desc* desc, const quasar_matrix* mats, int n_mats,
                              float* const* amax_out);

/* Host-only validation: the status quasar_reconstruct would return for these
 * arguments, without launching anything or touching device memory. */
int quasar_check(const quasar_desc* desc, const void* W, const float* v, const void* g,
                 const uint8_t* codes, const void* scales, const float* zeros, const void* r,
                 const uint8_t* best_clip, const float* err, const float* tensor_scale,
                 const float* tensor_amax, const void* workspace, size_t workspace_bytes);

/* Number of groups (INT), 16-blocks (NVFP4) or 8x64 blocks (RUBIN_INT3) of the
 * matrix; 0 for an invalid desc. */
int64_t quasar_num_groups(const quasar_desc* desc);

/* Which kernel serves INT and INT_SYM calls with this desc (host-only; the
 * result depends on the clip grid, bits and group, not on the shape):
 *  1  the binned kernel: each weight is placed once among the code thresholds
 *     T(k, b) of every clip, and each candidate's moments for the fit of
 *     Eq. ridgefit (Sec. 4.1.2) come from per-group suffix sums over those
 *     cells;
 *  0  the direct kernel: the moments are summed weight by weight for every
 *     clip (grids with many thresholds per group lane, such as INT4 with 8
 *     clips, where it is the faster one; or the environment variable
 *     QUASAR_INT_PATH=direct).  QUASAR_INT_PATH=binned selects the binned
 *     kernel for every grid whose thresholds fit its tables.
 * Both give the same codes, chosen clip and r up to the rounding order of the
 * fp64 moment sums.
 * For RUBIN_INT3 (whose per-clip sums of Eq. rubin-fit, App. B, always come
 * from such cells) it tells how a weight finds its cell:
 *  1  a table of 256 equal slices of the normalised range and at most three
 *     compares (clip grids whose thresholds are spread enough);
 *  0  a binary search over all thresholds (any grid, or the environment
 *     variable QUASAR_RUBIN_PATH=tree).
 * Both give identical results.  A negative quasar_status for an invalid desc
 * or the NVFP4 format. */
int quasar_int_path(const quasar_desc* desc);

/* Bytes of the packed code buffer; 0 for an invalid desc. */
size_t quasar_codes_bytes(const quasar_desc* desc);

/* Bytes of device workspace the call needs (NVFP4 without tensor_amax: 256;
 * otherwise 0). */
size_t quasar_workspace_bytes(const quasar_desc* desc, int has_tensor_amax);

/* Static description of a status code. */
const char* quasar_status_string(int status);

/* Library version, "major.minor.patch". */
const char* quasar_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QUASAR_H */
