/*
 * vcheck_oracle.h -- CPU oracle for candidate-vs-reference validation.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library. The product path never
 * calls it, and this oracle shares no code, header, table or helper with the
 * HIP implementation.
 *
 * What it computes (one plain loop per case, flat row-major index order, all
 * floating point in IEEE binary64 with round-to-nearest-even, no fused
 * multiply-add):
 *
 *   Validate(K, R, T, tau) of the problem formulation (Sec. 3.2, Eq. 1 and the
 *   conditions after it): every element of a candidate output is compared with
 *   the reference output under the tolerance gate |c - r| <= atol + rtol*|r|,
 *   together with the numerical-deviation metrics that the same section lists
 *   as diagnostic evidence (counts, NaN/Inf, max abs/rel error, error sums),
 *   the localization data of Sec. 4.2 (per-tile mismatch map, first failing
 *   indices), output-level degenerate-output detectors for the integrity
 *   hazards of Sec. 1 and Sec. 4.3, and the per-case pass/fail and suite match
 *   rate of the full-coverage evaluation (Sec. 4.3, Sec. S3.4).
 *
 * Parity status: every output of this oracle is pinned by the CPU test suite
 * (library routines, closed forms of the synthetic workloads, invariants and
 * hand-built boundary cases); see the pin list in the test module header.
 */
#ifndef VCHECK_ORACLE_H
#define VCHECK_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_F32 = 0, ORC_F16 = 1, ORC_BF16 = 2 };

enum {
  ORC_FLAG_ALL_ZERO = 1u << 0,
  ORC_FLAG_CONSTANT = 1u << 1,
  ORC_FLAG_INPUT_COPY = 1u << 2,
  ORC_FLAG_LOWPREC_BF16 = 1u << 3,
  ORC_FLAG_LOWPREC_FP16 = 1u << 4
};

typedef struct orc_stats {
  uint64_t numel;
  uint64_t mismatches; /* at the primary tolerance pair */
  uint64_t nan_cand, inf_cand, nan_ref, inf_ref;
  uint64_t n_finite, n_rel, n_rel_undef;
  double max_abs;
  int64_t argmax_abs;
  double max_rel;
  int64_t argmax_rel;
  double sum_abs, sum_rel;
} orc_stats;

typedef struct orc_integrity {
  uint64_t zero_cand, zero_ref, eqfirst_cand, eqfirst_ref;
  uint64_t bf16rep_cand, bf16rep_ref, fp16rep_cand, fp16rep_ref;
  uint32_t flags;
  int32_t copy_input;
  uint32_t cand_eq_input_mask, ref_eq_input_mask;
  uint32_t cand_eq_ref;
  uint32_t reserved;
} orc_integrity;

/* Decode n elements of the given storage type to binary64 (exact). */
void orc_decode(int32_t dtype, const void *src, int64_t n, double *dst);

/* Validate one case. cand/ref hold rows*cols elements of `dtype`, row-major.
 * mismatches[n_tols] receives the mismatch count of every tolerance pair.
 * tile_map (nullable) receives ceil(rows/tile_h)*ceil(cols/tile_w) counters
 * and is zeroed first; first_k (nullable) receives k indices, -1 padded.
 * integ (nullable) enables the degenerate-output detectors; inputs[j] is the
 * j-th operator input (input_dtype[j], input_numel[j]). Returns 0, or -1 on
 * an argument the oracle cannot evaluate. */
int32_t orc_validate(int32_t dtype, const void *cand, const void *ref, int64_t rows,
                     int64_t cols, int32_t n_tols, const double *atol, const double *rtol,
                     const int32_t *equal_nan, int32_t primary, uint64_t *mismatches,
                     orc_stats *st, int32_t tile_h, int32_t tile_w, uint32_t *tile_map,
                     int32_t k, int64_t *first_k, int32_t n_inputs,
                     const void *const *inputs, const int32_t *input_dtype,
                     const int64_t *input_numel, orc_integrity *integ);

/* Tensor-statistics probe of one tensor (the multi-level tensor statistics
 * that the engine's diagnostic instrumentation records at pipeline
 * boundaries, Sec. 4.2, and the tensor-statistic probes of the mechanism
 * figure's instrumentation panel). Over the n elements in flat order:
 * counts of NaN, of infinities, of zeros (+0 and -0) and of finite values;
 * the smallest and largest finite value with the first index holding each
 * (0 and -1 when no value is finite; +0 and -0 compare equal, and the value
 * reported is the element's own); binary64 sums of x, x*x and |x| over the
 * finite values, accumulated in index order; and a histogram of the finite
 * non-zero values by binary exponent e = floor(log2 |x|): bin
 * e - ORC_HIST_EMIN + 1 clamped to [0, ORC_HIST_BINS - 1], so bin 0 gathers
 * e < ORC_HIST_EMIN and the last bin e >= ORC_HIST_EMIN + ORC_HIST_BINS - 2. */
enum { ORC_HIST_BINS = 64, ORC_HIST_EMIN = -40 };

typedef struct orc_tstats {
  uint64_t numel, nan, inf, zero, n_finite;
  double min, max;
  int64_t argmin, argmax;
  double sum, sum_sq, sum_abs;
  uint64_t hist[ORC_HIST_BINS];
} orc_tstats;

void orc_tensor_stats(int32_t dtype, const void *x, int64_t n, orc_tstats *out);

/* Near-pass statistics of one case at one tolerance pair, for the near-pass
 * and fp16-ceiling detection of the adaptive scheduling rules (Sec. 4.4) and
 * the precision failures of Sec. 3.2 (Table 1: a cumsum whose binary32
 * accumulation misses a binary16-rounding reference). Over the pairs where
 * c and r are both finite, with d = |c - r| and t = atol + rtol*|r| in
 * binary64 (each operation rounded):
 *   n_pairs      such pairs; n_fail those with d > t;
 *   n_zero_tol   pairs with t == 0 and d > 0 (violation ratio unbounded);
 *   max_ratio    largest d / t over pairs with t > 0, argmax_ratio its first
 *                index (0 and -1 when there is none);
 *   ratio_hist   failing pairs with t > 0 by floor(log2(d / t)), the last
 *                bin gathering 31 and more;
 *   ulp_hist     pairs by their distance on the grid (binary16 for binary32
 *                and binary16 storage, bfloat16 for bfloat16 storage): both
 *                values rounded to the grid (nearest, ties to even), then the
 *                number of grid values between them; bin 0 distance 0, bin
 *                k in 1..16 distances [2^(k-1), 2^k), bin 17 pairs with a
 *                value beyond the grid's finite range;
 *   max_ulp_fail largest grid distance among failing pairs (0 if none,
 *                0xffffffff when one lies beyond the grid's range). */
enum { ORC_RATIO_BINS = 32, ORC_ULP_BINS = 18 };

typedef struct orc_np {
  uint64_t numel, n_pairs, n_fail, n_zero_tol;
  double max_ratio;
  int64_t argmax_ratio;
  uint32_t max_ulp_fail, reserved;
  uint64_t ratio_hist[ORC_RATIO_BINS];
  uint64_t ulp_hist[ORC_ULP_BINS];
} orc_np;

/* Rounds a finite binary64 value to binary16 (nearest, ties to even) and
 * returns the bit pattern; values beyond the range give +-Inf. */
uint16_t orc_round_binary16(double v);

void orc_nearpass(int32_t dtype, const void *cand, const void *ref, int64_t n, double atol,
                  double rtol, orc_np *out);

/* Content hash of one tensor, for the immutable evidence of a full-coverage
 * evaluation (Sec. 4.3: per-case results backed by full-coverage evidence;
 * Sec. S4 reproducibility artifacts): with w_i the i-th 64-bit word of the
 * tensor's storage (bytes 8i .. 8i+7 read little-endian, the last word
 * zero-padded; ceil(n * size / 8) words), n elements and storage code D,
 *   H = M(0x243F6A8885A308D3 ^ (D << 56) ^ n) + sum_i M(w_i ^ (i * G))
 * modulo 2^64, where G = 0x9E3779B97F4A7C15 and M is the 64-bit finalizer of
 * the SplitMix64 generator (Steele, Lea and Flood, 2014):
 *   z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
 *   z *= 0x94D049BB133111EB; z ^= z >> 31.
 * The sum is order-free, so any partition of the words hashes alike. */
uint64_t orc_content_hash(int32_t dtype, const void *x, int64_t n);

/* The finalizer M above. */
uint64_t orc_splitmix_finalize(uint64_t z);

/* Suite verdict over n_cases x n_tols mismatch counts (case-major).
 * status[c] < 0 marks a case that could not be evaluated (it fails).
 * flags[c] (nullable) are the detector flags; certification requires 0.
 * pass[c*n_tols+p] = 1 iff the case passes numerically at pair p;
 * rate[p] = certified cases / n_cases (0 when n_cases == 0). */
void orc_suite(int32_t n_cases, int32_t n_tols, const uint64_t *mismatches,
               const int32_t *status, const uint32_t *flags, uint8_t *pass, double *rate);

#ifdef __cplusplus
}
#endif
#endif
