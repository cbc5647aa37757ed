/*
 * vcheck_oracle.c -- plain, slow, obviously correct CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path. It shares no code
 * with the HIP implementation. Build: gcc -std=c11 -O2 -ffp-contract=off
 * -fno-fast-math -shared -fPIC (the -ffp-contract=off keeps every product and
 * sum separately rounded, as the definition below requires).
 *
 * Definition followed, per case (the view is (rows, cols), cols = last dim):
 *  1. decode c_i, r_i exactly to binary64;
 *  2. classify NaN / Inf of every element;
 *  3. gate, for every tolerance pair p (Sec. 3.2: Validate with tolerance tau;
 *     Sec. S2.2: every numerical case must pass the benchmark tolerance):
 *       close_p(i) = (c_i == r_i)
 *                 or (c_i, r_i finite and |c_i - r_i| <= atol_p + rtol_p*|r_i|)
 *                 or (equal_nan_p and c_i, r_i both NaN);
 *  4. numerical-deviation metrics over finite pairs (Sec. 3.2, the evidence D):
 *     max / argmax / sum of d_i = |c_i - r_i|, and of q_i = d_i / |r_i| where
 *     r_i != 0; argmax ties go to the smallest index;
 *  5. localization at the primary pair (Sec. 4.2 diagnostic instrumentation,
 *     Sec. S2.2 NaN/Inf forensics triggering localization): mismatches per
 *     tile_h x tile_w tile of the (rows, cols) view, and the k smallest
 *     mismatching flat indices in ascending order;
 *  6. degenerate-output detectors for the integrity hazards (Sec. 1
 *     "degeneration", Sec. 3.3 host-wrapper bypass, Sec. 4.3 anti-cheat,
 *     Sec. 4.4 degenerate-round and fp16-ceiling detection, Sec. S2.2
 *     golden-output cache): all-zero, constant fill, bit copy of an operator
 *     input, and a reduced-precision signature;
 *  7. per-case verdict and suite match rate (Sec. 4.3 full-coverage evidence:
 *     per-case pass/fail and match rates; Sec. S3.4: P/x = x% matched cases).
 */
#include "vcheck_oracle.h"

#include <math.h>
#include <string.h>

/* ---- step 1: exact decode ------------------------------------------------ */

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
static double decode_binary16(uint16_t h) {
  int sign = h >> 15;
  int expo = (h >> 10) & 0x1f;
  int frac = h & 0x3ff;
  double v;
  if (expo == 0) {
    v = ldexp((double)frac, -24); /* subnormal: frac * 2^-24 */
  } else if (expo == 31) {
    v = frac ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + frac), expo - 25); /* (1 + frac/2^10) * 2^(expo-15) */
  }
  return sign ? -v : v;
}

/* bfloat16: the upper half of a binary32 pattern. */
static double decode_bfloat16(uint16_t h) {
  uint32_t w = (uint32_t)h << 16;
  float f;
  memcpy(&f, &w, sizeof f);
  return (double)f;
}

static double decode_one(int32_t dtype, const void *base, int64_t i) {
  if (dtype == ORC_F32) {
    float f;
    memcpy(&f, (const char *)base + 4 * i, 4);
    return (double)f;
  }
  uint16_t h;
  memcpy(&h, (const char *)base + 2 * i, 2);
  return dtype == ORC_F16 ? decode_binary16(h) : decode_bfloat16(h);
}

/* Raw storage pattern of element i (for the bitwise detectors). */
static uint32_t bits_of(int32_t dtype, const void *base, int64_t i) {
  if (dtype == ORC_F32) {
    uint32_t w;
    memcpy(&w, (const char *)base + 4 * i, 4);
    return w;
  }
  uint16_t h;
  memcpy(&h, (const char *)base + 2 * i, 2);
  return h;
}

void orc_decode(int32_t dtype, const void *src, int64_t n, double *dst) {
  for (int64_t i = 0; i < n; i++) dst[i] = decode_one(dtype, src, i);
}

/* ---- step 6 helpers: exact representability of a binary32 value --------- */

/* bfloat16 keeps the upper 16 bits of a binary32 pattern. */
static int bf16_representable(uint32_t w) { return (w & 0xffffu) == 0; }

/* binary16 holds +-0, +-Inf, NaN, normals 2^-14 <= |v| <= 65504 with 10
 * fraction bits, and subnormals that are integer multiples of 2^-24. */
static int fp16_representable(uint32_t w) {
  float f;
  memcpy(&f, &w, sizeof f);
  if (f == 0.0f || isinf(f) || isnan(f)) return 1;
  double a = fabs((double)f);
  if (a >= 0x1p-14 && a <= 65504.0) return (w & 0x1fffu) == 0;
  if (a >= 0x1p-24 && a < 0x1p-14) {
    double s = a * 0x1p24;
    return s == floor(s);
  }
  return 0;
}

/* ---- one case ------------------------------------------------------------ */

int32_t orc_validate(int32_t dtype, const void *cand, const void *ref, int64_t rows,
                     int64_t cols, int32_t n_tols, const double *atol, const double *rtol,
                     const int32_t *equal_nan, int32_t primary, uint64_t *mismatches,
                     orc_stats *st, int32_t tile_h, int32_t tile_w, uint32_t *tile_map,
                     int32_t k, int64_t *first_k, int32_t n_inputs,
                     const void *const *inputs, const int32_t *input_dtype,
                     const int64_t *input_numel, orc_integrity *integ) {
  if (dtype < ORC_F32 || dtype > ORC_BF16 || rows < 0 || cols < 0 || n_tols < 1 ||
      primary < 0 || primary >= n_tols || n_inputs < 0 || n_inputs > 32)
    return -1;
  if (tile_map && (tile_h < 1 || tile_w < 1)) return -1;
  if (first_k && k < 0) return -1;

  const int64_t n = rows * cols;
  const int64_t tiles_r = tile_map ? (rows + tile_h - 1) / tile_h : 0;
  const int64_t tiles_c = tile_map ? (cols + tile_w - 1) / tile_w : 0;
  int64_t n_found = 0;

  memset(st, 0, sizeof *st);
  st->numel = (uint64_t)n;
  st->argmax_abs = -1;
  st->argmax_rel = -1;
  for (int32_t p = 0; p < n_tols; p++) mismatches[p] = 0;
  if (tile_map)
    for (int64_t t = 0; t < tiles_r * tiles_c; t++) tile_map[t] = 0;

  for (int64_t i = 0; i < n; i++) {
    /* 1. decode */
    const double c = decode_one(dtype, cand, i);
    const double r = decode_one(dtype, ref, i);

    /* 2. classify */
    /* isinf may return -1 for -Inf, so normalise every class test to 0/1 */
    const int c_nan = isnan(c) != 0, c_inf = isinf(c) != 0;
    const int r_nan = isnan(r) != 0, r_inf = isinf(r) != 0;
    st->nan_cand += c_nan;
    st->inf_cand += c_inf;
    st->nan_ref += r_nan;
    st->inf_ref += r_inf;
    const int finite = !c_nan && !c_inf && !r_nan && !r_inf;

    /* 3. gate, every tolerance pair */
    const double d = fabs(c - r);
    for (int32_t p = 0; p < n_tols; p++) {
      const double t = atol[p] + rtol[p] * fabs(r);
      const int close = (c == r) || (finite && d <= t) || (equal_nan[p] && c_nan && r_nan);
      if (close) continue;
      mismatches[p] += 1;
      if (p != primary) continue;
      /* 5. localization at the primary pair */
      if (tile_map) {
        const int64_t row = i / cols, col = i % cols;
        tile_map[(row / tile_h) * tiles_c + col / tile_w] += 1;
      }
      if (first_k && n_found < k) first_k[n_found++] = i;
    }

    /* 4. metrics over finite pairs */
    if (finite) {
      st->n_finite += 1;
      st->sum_abs += d;
      if (st->argmax_abs < 0 || d > st->max_abs) {
        st->max_abs = d;
        st->argmax_abs = i;
      }
      if (r != 0.0) {
        const double q = d / fabs(r);
        st->n_rel += 1;
        st->sum_rel += q;
        if (st->argmax_rel < 0 || q > st->max_rel) {
          st->max_rel = q;
          st->argmax_rel = i;
        }
      } else if (c != 0.0) {
        st->n_rel_undef += 1;
      }
    }
  }
  st->mismatches = mismatches[primary];
  if (first_k)
    for (int64_t j = n_found; j < k; j++) first_k[j] = -1;

  /* 6. degenerate-output detectors */
  if (integ) {
    memset(integ, 0, sizeof *integ);
    uint32_t eq_cand = 0, eq_ref = 0; /* bit j: still bit-equal to input j */
    for (int32_t j = 0; j < n_inputs; j++)
      if (input_dtype[j] == dtype && input_numel[j] == n) {
        eq_cand |= 1u << j;
        eq_ref |= 1u << j;
      }
    int cand_eq_ref = 1;
    const uint32_t first_cand = n > 0 ? bits_of(dtype, cand, 0) : 0;
    const uint32_t first_ref = n > 0 ? bits_of(dtype, ref, 0) : 0;
    for (int64_t i = 0; i < n; i++) {
      const uint32_t bc = bits_of(dtype, cand, i), br = bits_of(dtype, ref, i);
      integ->zero_cand += decode_one(dtype, cand, i) == 0.0;
      integ->zero_ref += decode_one(dtype, ref, i) == 0.0;
      integ->eqfirst_cand += bc == first_cand;
      integ->eqfirst_ref += br == first_ref;
      if (dtype == ORC_F32) {
        integ->bf16rep_cand += bf16_representable(bc);
        integ->bf16rep_ref += bf16_representable(br);
        integ->fp16rep_cand += fp16_representable(bc);
        integ->fp16rep_ref += fp16_representable(br);
      }
      if (bc != br) cand_eq_ref = 0;
      for (int32_t j = 0; j < n_inputs; j++) {
        const uint32_t bx = bits_of(dtype, inputs[j], i);
        if ((eq_cand >> j & 1u) && bc != bx) eq_cand &= ~(1u << j);
        if ((eq_ref >> j & 1u) && br != bx) eq_ref &= ~(1u << j);
      }
    }
    integ->cand_eq_input_mask = eq_cand;
    integ->ref_eq_input_mask = eq_ref;
    integ->cand_eq_ref = (uint32_t)cand_eq_ref;

    const uint64_t un = (uint64_t)n;
    uint32_t flags = 0;
    if (integ->zero_cand == un && n >= 1 && integ->zero_ref < un) flags |= ORC_FLAG_ALL_ZERO;
    if (integ->eqfirst_cand == un && n >= 2 && integ->zero_cand < un &&
        integ->eqfirst_ref < un)
      flags |= ORC_FLAG_CONSTANT;
    integ->copy_input = -1;
    for (int32_t j = 0; j < n_inputs; j++)
      if ((eq_cand >> j & 1u) && !(eq_ref >> j & 1u)) {
        flags |= ORC_FLAG_INPUT_COPY;
        integ->copy_input = j;
        break;
      }
    if (dtype == ORC_F32 && integ->bf16rep_cand == un && n >= 2 && integ->zero_cand < un &&
        integ->eqfirst_cand < un && integ->bf16rep_ref < un)
      flags |= ORC_FLAG_LOWPREC_BF16;
    if (dtype == ORC_F32 && integ->fp16rep_cand == un && integ->bf16rep_cand < un && n >= 2 &&
        integ->zero_cand < un && integ->eqfirst_cand < un && integ->fp16rep_ref < un)
      flags |= ORC_FLAG_LOWPREC_FP16;
    integ->flags = flags;
  }
  return 0;
}

/* ---- step 7: suite verdict ---------------------------------------------- */

void orc_suite(int32_t n_cases, int32_t n_tols, const uint64_t *mismatches,
               const int32_t *status, const uint32_t *flags, uint8_t *pass, double *rate) {
  for (int32_t p = 0; p < n_tols; p++) {
    int64_t certified = 0;
    for (int32_t c = 0; c < n_cases; c++) {
      const int ok = status[c] >= 0 && mismatches[(int64_t)c * n_tols + p] == 0;
      pass[(int64_t)c * n_tols + p] = (uint8_t)ok;
      if (ok && (!flags || flags[c] == 0)) certified += 1;
    }
    rate[p] = n_cases > 0 ? (double)certified / (double)n_cases : 0.0;
  }
}

/* ---- tensor-statistics probe ---------------------------------------------- */

/* Histogram bin of a finite non-zero value: frexp gives x = m * 2^p with
 * 0.5 <= |m| < 1, so floor(log2 |x|) = p - 1 exactly. */
static int hist_bin(double x) {
  int p = 0;
  (void)frexp(x, &p);
  const int b = (p - 1) - ORC_HIST_EMIN + 1;
  return b < 0 ? 0 : (b > ORC_HIST_BINS - 1 ? ORC_HIST_BINS - 1 : b);
}

void orc_tensor_stats(int32_t dtype, const void *x, int64_t n, orc_tstats *out) {
  memset(out, 0, sizeof *out);
  out->numel = (uint64_t)n;
  out->argmin = out->argmax = -1;
  for (int64_t i = 0; i < n; ++i) {
    const double v = decode_one(dtype, x, i);
    if (isnan(v)) {
      out->nan++;
      continue;
    }
    if (isinf(v)) {
      out->inf++;
      continue;
    }
    out->n_finite++;
    if (v == 0.0) out->zero++;
    if (out->argmin < 0 || v < out->min) {
      out->min = v;
      out->argmin = i;
    }
    if (out->argmax < 0 || v > out->max) {
      out->max = v;
      out->argmax = i;
    }
    out->sum += v;
    out->sum_sq += v * v;
    out->sum_abs += fabs(v);
    if (v != 0.0) out->hist[hist_bin(v)]++;
  }
}

/* ---- near-pass statistics -------------------------------------------------- */

/* Nearest binary16 (ties to even) of a finite binary64 value, written from
 * the format's definition: 1 sign, 5 exponent (bias 15), 10 fraction bits;
 * the grid spacing is 2^(e-10) for |v| in [2^e, 2^(e+1)), e >= -14, and
 * 2^-24 below 2^-14; magnitudes that round beyond 65504 become Inf. */
uint16_t orc_round_binary16(double v) {
  const uint16_t sign = signbit(v) ? 0x8000u : 0u;
  double a = fabs(v);
  if (a == 0.0) return sign;
  int p = 0;
  (void)frexp(a, &p); /* a = m * 2^p, 0.5 <= m < 1: exponent e = p - 1 */
  int e = p - 1;
  if (e < -14) e = -14; /* subnormal range: spacing 2^-24 */
  const double spacing = ldexp(1.0, e - 10);
  double k = a / spacing; /* exact: a power-of-two scaling */
  double kr = floor(k);
  const double frac = k - kr;
  if (frac > 0.5 || (frac == 0.5 && fmod(kr, 2.0) != 0.0)) kr += 1.0;
  const double r = kr * spacing;
  if (r > 65504.0) return (uint16_t)(sign | 0x7c00u);
  /* encode r exactly */
  if (r < ldexp(1.0, -14)) return (uint16_t)(sign | (uint16_t)(r / ldexp(1.0, -24)));
  int q = 0;
  const double m = frexp(r, &q); /* r = m * 2^q */
  const uint16_t expo = (uint16_t)(q - 1 + 15);
  const uint16_t fracb = (uint16_t)((m * 2.0 - 1.0) * 1024.0);
  return (uint16_t)(sign | (uint16_t)(expo << 10) | fracb);
}

/* Position on the ordered grid: -0 and +0 coincide. */
static int64_t grid_key(uint16_t h) {
  const int64_t mag = h & 0x7fff;
  return (h & 0x8000u) ? -mag : mag;
}

/* Grid pattern of a finite storage value: binary16 for binary32 values
 * (rounded), the stored pattern for 16-bit storage. Returns 0 when the
 * rounded value is beyond the grid's finite range. */
static int grid_of(int32_t dtype, const void *base, int64_t i, uint16_t *h) {
  if (dtype == ORC_F32) {
    *h = orc_round_binary16(decode_one(dtype, base, i));
  } else {
    *h = (uint16_t)bits_of(dtype, base, i);
  }
  const uint16_t expo_mask = dtype == ORC_BF16 ? 0x7f80u : 0x7c00u;
  return (*h & expo_mask) != expo_mask;
}

void orc_nearpass(int32_t dtype, const void *cand, const void *ref, int64_t n, double atol,
                  double rtol, orc_np *out) {
  memset(out, 0, sizeof *out);
  out->numel = (uint64_t)n;
  out->argmax_ratio = -1;
  for (int64_t i = 0; i < n; ++i) {
    const double c = decode_one(dtype, cand, i);
    const double r = decode_one(dtype, ref, i);
    if (!isfinite(c) || !isfinite(r)) continue;
    out->n_pairs++;
    const double d = fabs(c - r);
    const double t = atol + rtol * fabs(r);
    const int fail = d > t;
    if (fail) out->n_fail++;
    if (t == 0.0) {
      if (d > 0.0) out->n_zero_tol++;
    } else {
      const double q = d / t;
      if (out->argmax_ratio < 0 || q > out->max_ratio) {
        out->max_ratio = q;
        out->argmax_ratio = i;
      }
      if (fail) {
        int p = 0;
        (void)frexp(q, &p); /* q >= 1: floor(log2 q) = p - 1 */
        const int b = p - 1 > ORC_RATIO_BINS - 1 ? ORC_RATIO_BINS - 1 : p - 1;
        out->ratio_hist[b]++;
      }
    }
    uint16_t hc = 0, hr = 0;
    const int in_c = grid_of(dtype, cand, i, &hc), in_r = grid_of(dtype, ref, i, &hr);
    uint32_t dist;
    if (in_c && in_r) {
      const int64_t g = grid_key(hc) - grid_key(hr);
      dist = (uint32_t)(g < 0 ? -g : g);
      int bin = 0;
      while (bin < 16 && (dist >> bin) != 0) bin++; /* bin = bit length of dist */
      out->ulp_hist[bin]++;
    } else {
      dist = 0xffffffffu;
      out->ulp_hist[ORC_ULP_BINS - 1]++;
    }
    if (fail && dist > out->max_ulp_fail) out->max_ulp_fail = dist;
  }
}

/* ---- content hash ------------------------------------------------------------ */

uint64_t orc_splitmix_finalize(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

uint64_t orc_content_hash(int32_t dtype, const void *x, int64_t n) {
  uint64_t h = orc_splitmix_finalize(0x243F6A8885A308D3ull ^ ((uint64_t)dtype << 56) ^ (uint64_t)n);
  const int64_t nbytes = n * (dtype == ORC_F32 ? 4 : 2);
  const unsigned char *p = (const unsigned char *)x;
  for (int64_t i = 0; 8 * i < nbytes; ++i) {
    /* word i: bytes 8i .. 8i+7, little-endian, missing bytes zero */
    uint64_t w = 0;
    for (int b = 0; b < 8 && 8 * i + b < nbytes; ++b) w |= (uint64_t)p[8 * i + b] << (8 * b);
    h += orc_splitmix_finalize(w ^ ((uint64_t)i * 0x9E3779B97F4A7C15ull));
  }
  return h;
}
