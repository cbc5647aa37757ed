/*
 * vcheck.h -- C ABI of the MI355X (gfx950) validation and failure-forensics
 * library. ABI version 1.
 *
 * The library is the engine-owned validator of the paper's debug loop: it
 * compares a candidate operator output with the reference output over every
 * test case (Sec. 3.2, Eq. 1: Validate(K, R, T_ext, tau) = true), produces the
 * numerical-deviation metrics that the same section lists as diagnostic
 * evidence, localizes mismatches (Sec. 4.2, diagnostic instrumentation;
 * Sec. S2.2, NaN/Inf forensics triggering localization), runs output-level
 * degenerate-output detectors on every candidate (Sec. 4.1: integrity
 * checking on every candidate belongs to the engine; Sec. 4.3 anti-cheat),
 * and reduces per-case verdicts and suite match rates over the full case
 * matrix (Sec. 4.3 full-coverage evaluation; Sec. S3.4, P/x = x% matched
 * cases). Only this library's results carry acceptance: the caller cannot
 * make a case pass (Sec. 1 and Sec. 4.1, evidence ownership).
 *
 * ---- Conventions shared by every entry point ----------------------------
 *
 * Element semantics (per case; the view is (R, C) with C = last dimension,
 * R = product of the others; a 0-d tensor is (1, 1)):
 *   - values are decoded exactly (fp32 widened, fp16 per binary16 incl.
 *     subnormals, bf16 = upper half of a binary32 pattern) and compared in
 *     IEEE binary64 with round-to-nearest-even and no fused multiply-add;
 *   - gate for tolerance pair p:  close_p(i) = (c_i == r_i)
 *       or (c_i, r_i finite and |c_i - r_i| <= atol_p + rtol_p * |r_i|)
 *       or (equal_nan_p and c_i, r_i both NaN);  mismatch = not close.
 *     +Inf == +Inf is close, +0 == -0 is close, NaN is never close unless
 *     equal_nan is set;
 *   - metrics run over finite pairs only: d_i = |c_i - r_i|, and
 *     q_i = d_i / |r_i| where r_i != 0; argmax ties go to the smallest index.
 *
 * Memory: every data and output pointer is a DEVICE pointer on the current
 * HIP device; descriptor structs (vc_tensor, vc_case, vc_tol, vc_sweep_opts,
 * vc_sweep_out) are HOST memory and are not referenced after the call
 * returns. The caller owns every buffer, including the workspace (device
 * memory of at least vcheck_workspace_bytes() bytes, any alignment, contents
 * ignored on entry and clobbered); it must keep them alive until the stream
 * has finished the enqueued work. Results are valid after the stream syncs.
 * Input tensors must be contiguous row-major; a data pointer must be aligned
 * to its element size (16-byte alignment takes the fast vectorised path).
 *
 * Errors: every argument is checked on the host before anything is enqueued.
 * On error the call returns a negative vc_status, enqueues nothing and writes
 * no output; vcheck_last_error() gives a thread-local description. VC_OK
 * means the work was enqueued on `stream` (a hipStream_t; NULL = the null
 * stream). HIP launch failures return VC_ERR_HIP with the HIP error string.
 *
 * Determinism: results are bit-identical across runs for identical inputs
 * (fixed-order reductions, no floating-point atomics).
 *
 * Concurrency: calls on different streams may run concurrently as long as
 * they use different workspaces and outputs.
 *
 * Host-side state and blocking. The library keeps, per device and until the
 * process ends: a ring of 8 pinned host buffers of 256 KiB, allocated once
 * (by vcheck_init or by the first call that needs it), from which the first
 * kernel of a one-shot call copies the call's descriptor table (a buffer is
 * reused only after the event recorded behind the call that read it has
 * completed: a thread that issues more than 8 such calls ahead of the GPU
 * waits for the oldest); and the device address of the scratch array of
 * vcheck_sweep_noalloc. Both are guarded by a mutex. A descriptor table larger
 * than 256 KiB (about 1,300 sweep cases) is uploaded with a pageable copy,
 * which returns only once the runtime has taken the bytes (for pageable
 * memory it first waits for the stream's earlier work). Per thread: the last
 * error string and the vcheck_profile_events hook. Nothing else persists
 * between calls; descriptor planning uses the C++ heap.
 */
#ifndef VCHECK_H
#define VCHECK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VCHECK_ABI_VERSION 1
#define VC_MAX_NDIM 8
#define VC_MAX_TOLS 8
#define VC_MAX_INPUTS 8
#define VC_MAX_K 1024

typedef int32_t vc_status;
#define VC_OK 0
#define VC_ERR_NULL (-1)      /* a required pointer is NULL */
#define VC_ERR_DTYPE (-2)     /* unknown dtype, or cand/ref dtypes differ */
#define VC_ERR_SHAPE (-3)     /* bad ndim/shape, or cand/ref shapes differ */
#define VC_ERR_TOL (-4)       /* atol/rtol negative or not finite, bad primary_tol */
#define VC_ERR_TILE (-5)      /* tile_h or tile_w < 1 while a tile map is requested */
#define VC_ERR_K (-6)         /* k < 0, k > VC_MAX_K, or first_k NULL with k > 0 */
#define VC_ERR_WORKSPACE (-7) /* workspace NULL or smaller than required */
#define VC_ERR_LIMIT (-8)     /* n_tols, n_inputs or n_cases outside its range */
#define VC_ERR_HIP (-9)       /* HIP runtime / launch failure */
#define VC_ERR_ALIGN (-10)    /* data pointer not aligned to its element size */
#define VC_ERR_STATE (-11)    /* vcheck_init has not run on the current device, or a
                                 prepared sweep is launched on another device */

typedef enum vc_dtype { VC_F32 = 0, VC_F16 = 1, VC_BF16 = 2 } vc_dtype;

/* Detector flag bits (vc_integrity.flags); each is a conjunction, so each
 * degenerate class raises exactly one of them. n = numel. */
#define VC_FLAG_ALL_ZERO (1u << 0)     /* every cand element is +-0, ref is not */
#define VC_FLAG_CONSTANT (1u << 1)     /* n >= 2, every cand element has the bit pattern
                                          of element 0, cand is not all zero, ref is not
                                          constant */
#define VC_FLAG_INPUT_COPY (1u << 2)   /* cand is a bit copy of an operator input that
                                          ref is not a copy of */
#define VC_FLAG_LOWPREC_BF16 (1u << 3) /* fp32 only: n >= 2, every cand value is
                                          bf16-representable, cand neither constant nor
                                          all zero, ref not all bf16-representable */
#define VC_FLAG_LOWPREC_FP16 (1u << 4) /* fp32 only: as above for binary16, and cand is
                                          not all bf16-representable */

/* Tensor descriptor (host struct; data is a device pointer). */
typedef struct vc_tensor {
  const void *data;
  int32_t dtype; /* vc_dtype */
  int32_t ndim;  /* 0 .. VC_MAX_NDIM */
  int64_t shape[VC_MAX_NDIM];
} vc_tensor; /* 80 bytes */

/* One tolerance pair; atol and rtol finite and >= 0; equal_nan 0 or 1. */
typedef struct vc_tol {
  double atol;
  double rtol;
  int32_t equal_nan;
  int32_t reserved; /* must be 0 */
} vc_tol; /* 24 bytes */

/* Per-case statistics (device-resident output). Counts at the primary pair. */
typedef struct vc_stats {
  uint64_t numel;
  uint64_t mismatches;                      /* at the primary tolerance pair */
  uint64_t nan_cand, inf_cand, nan_ref, inf_ref; /* element counts */
  uint64_t n_finite;    /* pairs with both values finite */
  uint64_t n_rel;       /* finite pairs with r != 0 */
  uint64_t n_rel_undef; /* finite pairs with r == 0 and c != 0 */
  double max_abs;       /* 0.0 when n_finite == 0 */
  int64_t argmax_abs;   /* flat index, -1 when n_finite == 0 */
  double max_rel;       /* exact (correctly rounded quotient) */
  int64_t argmax_rel;   /* -1 when n_rel == 0 */
  double sum_abs;       /* sum of d_i, binary64 accumulation, within 1e-6 relative */
  double sum_rel;       /* sum of q_i, binary64, within 1e-6 relative */
  int32_t case_status;  /* 0, or a negative vc_status for a case that could not run */
  int32_t pass;         /* 1 iff case_status == 0 and mismatches == 0 */
} vc_stats; /* 128 bytes */

/* Degenerate-output detector results (device-resident output). */
typedef struct vc_integrity {
  uint64_t zero_cand, zero_ref;       /* elements equal to +-0 */
  uint64_t eqfirst_cand, eqfirst_ref; /* elements bit-equal to element 0 */
  uint64_t bf16rep_cand, bf16rep_ref; /* fp32 only: low 16 pattern bits zero */
  uint64_t fp16rep_cand, fp16rep_ref; /* fp32 only: exactly representable in binary16
                                         (NaN and +-Inf count as representable) */
  uint32_t flags;                     /* VC_FLAG_* */
  int32_t copy_input;                 /* smallest j raising INPUT_COPY, else -1 */
  uint32_t cand_eq_input_mask;        /* bit j: cand bit-equal to input j (same dtype,
                                         same numel) */
  uint32_t ref_eq_input_mask;         /* bit j: ref bit-equal to input j */
  uint32_t cand_eq_ref;               /* 1 iff cand bit-equal to ref (evidence only) */
  uint32_t reserved;
} vc_integrity; /* 88 bytes */

/* One test case of a sweep (host struct). inputs: host array of n_inputs
 * operator-input descriptors used by the input-copy detector. */
typedef struct vc_case {
  vc_tensor cand;
  vc_tensor ref;
  const vc_tensor *inputs;
  int32_t n_inputs; /* 0 .. VC_MAX_INPUTS */
  int32_t reserved;
} vc_case; /* 176 bytes */

typedef struct vc_sweep_opts {
  int32_t primary_tol;  /* pair used for vc_stats.mismatches, tile maps, first-k */
  int32_t tile_h, tile_w; /* tile geometry, used when out->tile_maps != NULL */
  int32_t k;            /* first-k length, used when out->first_k != NULL */
  int32_t do_integrity; /* 1: run the detectors (out->integ required) */
  int32_t reserved;
} vc_sweep_opts;

/* Sweep outputs (host struct of device pointers). */
typedef struct vc_sweep_out {
  vc_stats *stats;        /* [n_cases], required */
  uint64_t *mismatches;   /* [n_cases * n_tols] case-major, nullable */
  uint8_t *pass;          /* [n_cases * n_tols]: numeric pass per pair, nullable */
  double *match_rate;     /* [n_tols]: certified cases / n_cases, nullable;
                             certified = pass and (no integrity run or flags == 0) */
  double *numeric_rate;   /* [n_tols]: passing cases / n_cases, nullable */
  uint32_t *tile_maps;    /* concatenated per-case tile maps, nullable; case i
                             starts at sum_{j<i} vcheck_tile_count(ref of case j)
                             (cases with a negative case_status keep their slots,
                             which stay 0) */
  int64_t *first_k;       /* [n_cases * k], -1 padded, nullable */
  vc_integrity *integ;    /* [n_cases], required iff do_integrity */
} vc_sweep_out;

/*
 * vcheck_compare -- validate one candidate against its reference at one
 * tolerance pair (Sec. 3.2 Validate; metrics of the diagnostic evidence D).
 *   cand, ref: same dtype and shape.  tol: one pair.
 *   out: device vc_stats.  ws/ws_bytes: workspace (vcheck_workspace_bytes
 *   with the case {cand, ref}, n_tols = 1, opts = NULL).
 */
vc_status vcheck_compare(const vc_tensor *cand, const vc_tensor *ref, const vc_tol *tol,
                         vc_stats *out, void *ws, size_t ws_bytes, void *stream);

/*
 * vcheck_localize -- vcheck_compare plus localization (Sec. 4.2 diagnostic
 * instrumentation; Sec. S2.2 NaN/Inf forensics triggering localization).
 *   tile_map: device uint32[vcheck_tile_count(cand, tile_h, tile_w)],
 *     mismatches per tile_h x tile_w tile of the (R, C) view, row-major
 *     tiles, partial edge tiles included.
 *   first_k: device int64[k], the k smallest mismatching flat indices in
 *     ascending order, -1 padded (may be NULL when k == 0).
 *   out: device vc_stats, nullable.
 *   Workspace: vcheck_workspace_bytes with opts.k = k.
 */
vc_status vcheck_localize(const vc_tensor *cand, const vc_tensor *ref, const vc_tol *tol,
                          int32_t tile_h, int32_t tile_w, uint32_t *tile_map, int32_t k,
                          int64_t *first_k, vc_stats *out, void *ws, size_t ws_bytes,
                          void *stream);

/*
 * vcheck_integrity -- degenerate-output detectors in the same pass as the
 * comparison (integrity hazards: Sec. 1 "degeneration", Sec. 3.3 host-wrapper
 * bypass, Sec. 4.3 anti-cheat, Sec. 4.4 degenerate-round and fp16-ceiling
 * detection, Sec. S2.2 golden-output cache).
 *   inputs: host array of n_inputs (0 .. VC_MAX_INPUTS) operator inputs;
 *     an input takes part in the copy detector when its dtype and numel
 *     match cand's. Input data is read only while cand or ref is still
 *     bit-equal to it.
 *   out: device vc_integrity.  stats: device vc_stats, nullable.
 */
vc_status vcheck_integrity(const vc_tensor *cand, const vc_tensor *ref, const vc_tensor *inputs,
                           int32_t n_inputs, const vc_tol *tol, vc_integrity *out,
                           vc_stats *stats, void *ws, size_t ws_bytes, void *stream);

/*
 * vcheck_sweep -- validate a whole case matrix in one call (Sec. 4.3
 * full-coverage evaluation: per-case pass/fail and match rates over all
 * shapes and dtypes), evaluating n_tols (1 .. VC_MAX_TOLS) tolerance pairs in
 * the same pass. n_cases 0 .. 2^24.
 * A case whose cand/ref dtype or shape differ, or whose pointers are not
 * element-aligned, is a data outcome, not an API error: it gets a negative
 * case_status and pass = 0 (the paper's runtime-failure class), the rest of
 * the batch runs.
 * opts: NULL means primary_tol 0, no tile maps, k = 0, no integrity.
 */
vc_status vcheck_sweep(const vc_case *cases, int32_t n_cases, const vc_tol *tols, int32_t n_tols,
                       const vc_sweep_opts *opts, const vc_sweep_out *out, void *ws,
                       size_t ws_bytes, void *stream);

/* ---- prepared sweeps -------------------------------------------------------
 *
 * The repair loop validates every candidate of an operator against the same
 * case matrix (Sec. 3.2: Validate(K, R, T_ext, tau) for each repaired
 * kernel; Sec. 4.3: full-coverage evaluation of every accepted candidate):
 * the case descriptors do not change between candidates when each candidate
 * writes its outputs into the same buffers. A prepared sweep uploads the
 * case table once; each launch then runs only the streaming and merge
 * kernels, with the results of vcheck_sweep.
 */
typedef struct vc_plan vc_plan; /* opaque, host memory */

/*
 * vcheck_plan_sweep -- check and plan a sweep exactly as vcheck_sweep does
 * (same arguments, same errors), upload its case table into `ws` and clear
 * the workspace parts that must be zero on entry. Blocks until the upload is
 * done (it synchronizes `stream`). On success *plan receives a plan that
 * refers to the descriptors' device pointers, the outputs of `out` and the
 * workspace: the caller keeps all of them alive, and the workspace for this
 * plan's use only, until vcheck_plan_free. Host structs (cases, tols, opts,
 * out) are not referenced after the call. The plan belongs to the current
 * device.
 */
vc_status vcheck_plan_sweep(const vc_case *cases, int32_t n_cases, const vc_tol *tols,
                            int32_t n_tols, const vc_sweep_opts *opts, const vc_sweep_out *out,
                            void *ws, size_t ws_bytes, void *stream, vc_plan **plan);

/*
 * vcheck_plan_launch -- enqueue one evaluation of a prepared sweep on
 * `stream`: the outputs are those of vcheck_sweep over the current contents
 * of the case tensors, valid after the stream syncs. Each launch leaves the
 * workspace ready for the next one, so launches of one plan must not
 * overlap (use one stream, or order the streams). Errors: VC_ERR_NULL,
 * VC_ERR_STATE (current device is not the plan's), VC_ERR_HIP. After a
 * VC_ERR_HIP, free the plan and prepare a new one.
 */
vc_status vcheck_plan_launch(vc_plan *plan, void *stream);

/* Frees a plan (NULL is accepted). Does not wait for launches in flight:
 * the workspace and outputs must stay alive until they are done. */
vc_status vcheck_plan_free(vc_plan *plan);

/* ---- library set-up and the allocation-free sweep -------------------------- */

/* Set-up for the current device: allocates the pinned staging ring (once)
 * and takes the device address of vcheck_sweep_noalloc's scratch array.
 * Idempotent; call it once per device (with that device current) before
 * vcheck_sweep_noalloc. Errors: VC_ERR_HIP. */
vc_status vcheck_init(void);

/* Bytes of device scratch per device that vcheck_sweep_noalloc works in. */
#define VC_NOALLOC_SCRATCH_BYTES (64ull << 20)

/*
 * vcheck_sweep_noalloc -- vcheck_sweep for callers that cannot allocate
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. Same arguments and results as vcheck_sweep except the
 * workspace: the library's static device scratch array of
 * VC_NOALLOC_SCRATCH_BYTES bytes on the current device. The call allocates
 * no device or pinned memory (vcheck_init must have run on the device:
 * VC_ERR_STATE otherwise). It rejects, before enqueueing anything, a sweep
 * whose workspace (vcheck_workspace_bytes) exceeds VC_NOALLOC_SCRATCH_BYTES
 * or whose case table exceeds one 256 KiB staging buffer (VC_ERR_LIMIT).
 * Every call on a device shares that device's scratch, whose contents the
 * next call overwrites: calls that overlap on one device (other streams,
 * other threads) race and must be serialized by the caller.
 */
vc_status vcheck_sweep_noalloc(const vc_case *cases, int32_t n_cases, const vc_tol *tols,
                               int32_t n_tols, const vc_sweep_opts *opts,
                               const vc_sweep_out *out, void *stream);

/* ---- tensor-statistics probe ---------------------------------------------
 *
 * The multi-level tensor statistics that the engine's diagnostic
 * instrumentation records at pipeline boundaries when a repair attempt has
 * failed (Sec. 4.2, diagnostic instrumentation; the instrumentation panel of
 * the mechanisms figure: tensor-statistic probes). One call probes a batch of
 * tensors in one pass over HBM. Per tensor, over its elements in flat order:
 *   nan, inf, zero      counts of NaN, of +-Inf and of +-0 elements;
 *   n_finite            finite elements (zeros included);
 *   min, max            smallest / largest finite value, the value of the
 *                       element itself (+0 and -0 compare equal);
 *   argmin, argmax      first flat index holding it (-1, and min = max = 0,
 *                       when no element is finite);
 *   sum, sum_sq, sum_abs binary64 sums of x, x*x and |x| over finite values
 *                       (summation order unspecified: each differs from the
 *                       exact sum by at most 1e-6 times the sum of its terms'
 *                       magnitudes);
 *   hist[b]             finite non-zero values with binary exponent
 *                       e = floor(log2 |x|) in bin b = e - VC_HIST_EMIN + 1,
 *                       clamped to [0, VC_HIST_BINS - 1] (bin 0 gathers
 *                       e < VC_HIST_EMIN, the last bin e >= VC_HIST_EMIN + 62).
 * mean = sum / n_finite, the standard deviation and the mean magnitude
 * follow from these. */
#define VC_HIST_BINS 64
#define VC_HIST_EMIN (-40)

typedef struct vc_tstats {
  uint64_t numel, nan, inf, zero, n_finite;
  double min, max;
  int64_t argmin, argmax;
  double sum, sum_sq, sum_abs;
  uint64_t hist[VC_HIST_BINS];
} vc_tstats;

/* Statistics of tensors[0 .. n_tensors) (device data, any storage type, any
 * element-aligned pointer; 16-byte alignment takes the vectorised path) into
 * out[0 .. n_tensors) (device vc_tstats, one per tensor, in order).
 * Workspace: vcheck_tensor_stats_workspace for the same tensors.
 * Errors: VC_ERR_NULL (tensors, out or a data pointer of a non-empty tensor
 * NULL), VC_ERR_DTYPE, VC_ERR_SHAPE, VC_ERR_ALIGN (pointer not aligned to the
 * element size), VC_ERR_LIMIT (n_tensors outside 0 .. 2^20, or a tensor of
 * 2^34 elements or more), VC_ERR_WORKSPACE, VC_ERR_HIP. n_tensors = 0 enqueues
 * nothing. */
vc_status vcheck_tensor_stats(const vc_tensor *tensors, int32_t n_tensors, vc_tstats *out,
                              void *workspace, size_t ws_bytes, void *stream);

/* Workspace bytes for vcheck_tensor_stats over the same tensors. */
vc_status vcheck_tensor_stats_workspace(const vc_tensor *tensors, int32_t n_tensors,
                                        size_t *bytes);

/* ---- near-pass statistics -------------------------------------------------
 *
 * Evidence for the near-pass and fp16-ceiling rules of the adaptive
 * scheduling (Sec. 4.4) and for precision failures such as Table 1's (a
 * binary32 accumulation against a reference that rounds to binary16 at every
 * step): how far the failing elements are from the tolerance, and how many
 * grid steps apart the two outputs are. Per case, at one tolerance pair,
 * over the elements where cand and ref are both finite, with d = |c - r|
 * and t = atol + rtol*|r| in binary64 (each operation rounded):
 *   n_pairs       such elements; n_fail those with d > t;
 *   n_zero_tol    elements with t == 0 and d > 0 (unbounded ratio);
 *   max_ratio     largest binary64 d / t over elements with t > 0, at the
 *                 first flat index argmax_ratio (0 and -1 when none);
 *   ratio_hist[b] failing elements with t > 0 and floor(log2(d / t)) = b
 *                 (the last bin: b >= 31);
 *   ulp_hist[b]   elements by their distance on the grid: binary16 for
 *                 binary32 and binary16 storage, bfloat16 for bfloat16
 *                 storage (both values rounded to the grid, nearest, ties to
 *                 even; -0 and +0 are one grid value); bin 0 distance 0, bin
 *                 b in 1..16 distances in [2^(b-1), 2^b), bin 17 elements
 *                 with a value beyond the grid's finite range;
 *   max_ulp_fail  largest grid distance among failing elements (0 if none,
 *                 0xffffffff when one lies beyond the grid's range).
 * A case fails only within one grid step (the fp16 ceiling) when
 * n_fail > 0 and max_ulp_fail <= 1 and no non-finite element mismatches. */
#define VC_RATIO_BINS 32
#define VC_ULP_BINS 18

typedef struct vc_nearpass {
  uint64_t numel, n_pairs, n_fail, n_zero_tol;
  double max_ratio;
  int64_t argmax_ratio;
  uint32_t max_ulp_fail, reserved;
  uint64_t ratio_hist[VC_RATIO_BINS];
  uint64_t ulp_hist[VC_ULP_BINS];
} vc_nearpass;

/* Near-pass statistics of cases[0 .. n_cases) at tolerance `tol` (its
 * equal_nan is ignored: only finite pairs count) into out[0 .. n_cases)
 * (device vc_nearpass, in case order); inputs are not read. Workspace:
 * vcheck_nearpass_workspace. Errors: VC_ERR_NULL, VC_ERR_DTYPE and
 * VC_ERR_SHAPE (also for a case whose cand and ref differ in dtype or
 * shape), VC_ERR_ALIGN, VC_ERR_TOL, VC_ERR_LIMIT (n_cases outside
 * 0 .. 2^20, or a case of 2^31 elements or more), VC_ERR_WORKSPACE,
 * VC_ERR_HIP. n_cases = 0 enqueues nothing. */
vc_status vcheck_nearpass(const vc_case *cases, int32_t n_cases, const vc_tol *tol,
                          vc_nearpass *out, void *workspace, size_t ws_bytes, void *stream);

/* Workspace bytes for vcheck_nearpass over the same cases. */
vc_status vcheck_nearpass_workspace(const vc_case *cases, int32_t n_cases, size_t *bytes);

/* ---- content hash ---------------------------------------------------------
 *
 * Content hashes of tensors, for the immutable evidence of a full-coverage
 * evaluation (Sec. 4.3: acceptance backed by full-coverage evidence; the
 * per-case pass/fail record; Sec. S4 reproducibility artifacts). With w_i
 * the i-th 64-bit word of the tensor's storage (bytes 8i .. 8i+7 read
 * little-endian, the last word zero-padded), n elements and storage code D:
 *   H = M(0x243F6A8885A308D3 ^ (D << 56) ^ n) + sum_i M(w_i ^ (i * G)) mod 2^64,
 * G = 0x9E3779B97F4A7C15 and M the 64-bit finalizer of the SplitMix64
 * generator (z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
 * z *= 0x94D049BB133111EB; z ^= z >> 31). Not cryptographic: it detects
 * changed, reordered or truncated outputs between evaluations. */

/* Hashes of tensors[0 .. n_tensors) into out[0 .. n_tensors) (device
 * uint64_t; overwritten). Workspace: vcheck_content_hash_workspace. Errors
 * as for vcheck_tensor_stats. n_tensors = 0 enqueues nothing. */
vc_status vcheck_content_hash(const vc_tensor *tensors, int32_t n_tensors, uint64_t *out,
                              void *workspace, size_t ws_bytes, void *stream);

/* Workspace bytes for vcheck_content_hash over the same tensors. */
vc_status vcheck_content_hash_workspace(const vc_tensor *tensors, int32_t n_tensors,
                                        size_t *bytes);

/* Profiling hook (tracing): the next vcheck_compare / _localize / _integrity /
 * _sweep / _tensor_stats / _nearpass / _content_hash call made on this thread
 * records `begin_event` on its stream just before its first streaming-kernel
 * launch and `end_event` just after its last one, so hipEventElapsedTime
 * gives the duration of the streaming kernels alone (without the prologue
 * and the merge kernels). Both are hipEvent_t handles created by the caller;
 * the hook is consumed by that one call. Pass NULL, NULL to clear it.
 * Returns VC_OK, or VC_ERR_NULL when only one of the two is NULL. */
vc_status vcheck_profile_events(void *begin_event, void *end_event);

/* Workspace bytes for a sweep over `cases` (also for the single-case entry
 * points: one case, n_tols = 1, opts carrying k and, for vcheck_localize,
 * the tile geometry). opts->tile_h and opts->tile_w of 1 or more size the
 * workspace for tile maps of that geometry (4 bytes per tile); 0 (or opts
 * NULL) for a call without tile maps. Returns VC_OK and writes *bytes, or
 * an error status for arguments the sweep would reject. */
vc_status vcheck_workspace_bytes(const vc_case *cases, int32_t n_cases, int32_t n_tols,
                                 const vc_sweep_opts *opts, size_t *bytes);

/* Number of tiles of t's (R, C) view: ceil(R/tile_h) * ceil(C/tile_w);
 * -1 for an invalid descriptor or tile size. */
int64_t vcheck_tile_count(const vc_tensor *t, int32_t tile_h, int32_t tile_w);

/* Static description of a status code. */
const char *vcheck_status_str(vc_status status);

/* Thread-local description of the last error on this thread ("" if none). */
const char *vcheck_last_error(void);

/* VCHECK_ABI_VERSION of the loaded library. */
int32_t vcheck_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* VCHECK_H */
