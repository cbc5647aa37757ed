// vcheck_kernels.hip -- gfx950 kernels of the validation library.
//
// One streaming pass over (cand, ref) computes, per case, everything the
// engine-owned validation and forensics need (Sec. 3.2 Validate and the
// numerical-deviation evidence; Sec. 4.2 localization; Sec. 4.3 integrity and
// full-coverage evidence): the tolerance gate for up to 8 pairs, NaN/Inf
// counts, exact max/argmax of |c-r| and |c-r|/|r|, binary64 error sums, the
// per-tile mismatch map, the ordered first-k mismatch indices and the
// degenerate-output detector counts.
//
// Work decomposition: a case is cut into chunks of 4 * U elements; one block
// (4 waves) owns one chunk and streams it front to back: a step is 64 lanes x
// 16 bytes (one fully coalesced 1 KiB non-temporal load per tensor) and the
// four waves take steps round robin, so the block's loads always target one
// contiguous stretch of memory (this interleave reads HBM markedly faster
// than one contiguous range per wave). The loop is unrolled twice so the
// next step's loads are in flight while the current step is evaluated.
// Per-wave results carry chunk offsets, so ties and first-k are resolved by
// index, not by which wave saw an element first.
//
// Exactness. The definition is binary64 on exactly decoded values (every
// storage type widens exactly to binary32, and binary32 to binary64). Each
// step first runs a fast path that evaluates the gate, |c - r| and |r| in
// binary64 exactly as the definition (separately rounded rtol*|r| and
// atol + (.), no contraction anywhere in this file), keeps the lane maximum
// of |c - r| in binary64 and tests every element against the wave's exact
// running maximum of |c - r|/|r| with the exact sign test
// fma(-M, |r|, d) > 0 <=> d/|r| > M. Only an element that strictly beats a
// running maximum reaches the update path (a correctly rounded division and a
// wave reduction that keeps the smallest index on ties), so ties cost
// nothing. The fast path assumes every value finite and every r non-zero
// (checked through the finiteness of the lane's quotient estimates); a step
// that breaks this is evaluated element by element with the class tests (the
// exact path) from the registers it already holds. Only sum_rel uses binary32
// quotient estimates (relative error below 5e-7, within the 1e-6 contract).
// Counts come from wave ballots and popcounts; no floating-point atomics are
// used, so every result is bit-reproducible.
#pragma clang fp contract(off)

#include "vcheck_internal.h"

namespace vck {
namespace {

template <int DT>
struct Tr;
template <>
struct Tr<VC_F32> {
  static constexpr int V = 4;
  static constexpr int ES = 4;
};
template <>
struct Tr<VC_F16> {
  static constexpr int V = 8;
  static constexpr int ES = 2;
};
template <>
struct Tr<VC_BF16> {
  static constexpr int V = 8;
  static constexpr int ES = 2;
};

// 16 bytes of raw storage held by one lane.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Raw storage pattern of element j (0 <= j < V) of a 16-byte vector.
template <int DT>
__device__ __forceinline__ uint32_t elem(const u32x4 &x, int j) {
  if constexpr (Tr<DT>::ES == 4) {
    return j == 0 ? x[0] : j == 1 ? x[1] : j == 2 ? x[2] : x[3];
  } else {
    const int w = j >> 1;
    const uint32_t v = w == 0 ? x[0] : w == 1 ? x[1] : w == 2 ? x[2] : x[3];
    return (j & 1) ? (v >> 16) : (v & 0xffffu);
  }
}

// Exact widening of one storage pattern to binary32 / binary64.
template <int DT>
__device__ __forceinline__ float dec32(uint32_t raw) {
  if constexpr (DT == VC_F32) {
    return __uint_as_float(raw);
  } else if constexpr (DT == VC_F16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)raw);
  } else {
    return __uint_as_float(raw << 16);
  }
}
template <int DT>
__device__ __forceinline__ double dec64(uint32_t raw) {
  return (double)dec32<DT>(raw);
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ uint32_t popc(uint64_t m) { return (uint32_t)__popcll(m); }
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Loads through global-address-space pointers (the data pointers come from
// the case table, so the compiler cannot infer it; generic loads would also
// wait on the LDS counter).
#define VCK_GLOBAL __attribute__((address_space(1)))
#define VCK_CONST __attribute__((address_space(4)))

// Streamed data is read once: non-temporal loads keep it from displacing
// reused lines in the caches.
__device__ __forceinline__ u32x4 load16(const uint8_t *p) {
  return __builtin_nontemporal_load((const VCK_GLOBAL u32x4 *)(p));
}

// Element loads of positions idx0 .. idx0+V-1 below `end` (others read 0).
template <int DT>
__device__ __forceinline__ u32x4 load_guarded(const uint8_t *base, uint64_t idx0, uint64_t end) {
  uint32_t v[Tr<DT>::V];
#pragma unroll
  for (int j = 0; j < Tr<DT>::V; ++j) {
    const uint64_t i = idx0 + j;
    uint32_t x = 0;
    if (i < end) {
      if constexpr (Tr<DT>::ES == 4) x = *(const VCK_GLOBAL uint32_t *)(base + i * 4);
      else x = *(const VCK_GLOBAL uint16_t *)(base + i * 2);
    }
    v[j] = x;
  }
  u32x4 r;
  if constexpr (Tr<DT>::ES == 4) {
    r[0] = v[0];
    r[1] = v[1];
    r[2] = v[2];
    r[3] = v[3];
  } else {
    r[0] = v[0] | (v[1] << 16);
    r[1] = v[2] | (v[3] << 16);
    r[2] = v[4] | (v[5] << 16);
    r[3] = v[6] | (v[7] << 16);
  }
  return r;
}

struct WaveOut {
  uint32_t mism[VC_MAX_TOLS];
  uint32_t nan_c, inf_c, nan_r, inf_r, n_fin, n_rel, n_rel_undef, eq_bits;
  uint32_t nfound, zc, zr, efc, efr, bfc, bfr, hfc, hfr;
  uint32_t amax_abs, amax_rel;
  double max_abs, max_rel, sum_abs, sum_rel;
};

// Member-wise copy of a case descriptor read through the constant address
// space (scalar loads).
__device__ __forceinline__ DevCase load_case(const VCK_CONST DevCase *t) {
  DevCase d;
  d.cand = t->cand;
  d.ref = t->ref;
#pragma unroll
  for (int q = 0; q < VC_MAX_INPUTS; ++q) d.inp[q] = t->inp[q];
  d.numel = t->numel;
  d.cols = t->cols;
  d.chunk_begin = t->chunk_begin;
  d.tile_off = t->tile_off;
  d.tiles_c = t->tiles_c;
  d.n_chunks = t->n_chunks;
  d.status = t->status;
  d.inp_mask = t->inp_mask;
  d.vec_ok = t->vec_ok;
  d.orig = t->orig;
  d.dtype = t->dtype;
  d.unit_elems = t->unit_elems;
  d.reserved = 0;
  return d;
}

__device__ __forceinline__ void max_merge(double &v, uint32_t &i, double ov, uint32_t oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

__device__ __forceinline__ double readfirstlane_f64(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Wave-wide (largest value, smallest index) of the lanes' (v, i), returned
// as wave-uniform values. Lanes with nothing pass v = -1 (real values are
// >= 0) and i = 0xffffffff.
__device__ __forceinline__ void wave_max(double &v, uint32_t &i) {
#pragma unroll
  for (int m = kWaveSize / 2; m >= 1; m >>= 1) {
    const double ov = __shfl_xor(v, m);
    const uint32_t oi = __shfl_xor(i, m);
    max_merge(v, i, ov, oi);
  }
  v = readfirstlane_f64(v);
  i = __builtin_amdgcn_readfirstlane(i);
}

#ifndef VCK_WAVES_PER_EU
#define VCK_WAVES_PER_EU 4
#endif

template <int DT, int NT, bool INTEG>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(VCK_WAVES_PER_EU)))
void main_kernel(const Params P) {
  constexpr int V = Tr<DT>::V;
  constexpr int ES = Tr<DT>::ES;
  constexpr uint32_t ITER = kWaveSize * V;  // elements per wave step
  constexpr uint32_t ALL = (1u << V) - 1u;

  __shared__ uint32_t s_win[kTileWindow];   // block tile-count window
  __shared__ uint32_t s_merged[VC_MAX_K];   // first-k merge of the four waves
  __shared__ WaveOut s_out[kWavesPerBlock];
  // counters touched only by the exact path, per wave (kept out of scalar
  // registers): nan_c, inf_c, nan_r, inf_r, n_fin, n_rel, n_rel_undef
  __shared__ uint32_t s_rare[kWavesPerBlock][8];

  const uint32_t lane = threadIdx.x & (kWaveSize - 1);
  // wave index: uniform per wave (keeps every range bound in scalar registers)
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  const uint64_t chunk = P.chunk_lo + blockIdx.x;

  // Locate the case: the last table entry whose first chunk is <= chunk
  // (scalar loads through the constant address space).
  const VCK_CONST DevCase *table = (const VCK_CONST DevCase *)P.cases;
  uint64_t ci = 0;
  if (table != nullptr) {
    uint64_t lo = P.case_lo, hi = P.case_hi - 1;
    while (lo < hi) {
      const uint64_t mid = (lo + hi + 1) / 2;
      if (table[mid].chunk_begin <= chunk) lo = mid;
      else hi = mid - 1;
    }
    ci = lo;
  }
  // a value copy (an lvalue selecting between the table and the by-value
  // argument would force the whole argument struct into private memory)
  DevCase dcs;
  if (table != nullptr) dcs = load_case(table + ci);
  else dcs = P.single;
  const uint8_t *const cand = dcs.cand;
  const uint8_t *const ref = dcs.ref;
  const uint64_t numel = dcs.numel;
  const uint64_t cols = dcs.cols;
  const uint64_t tiles_c = dcs.tiles_c;
  const uint64_t tile_off = dcs.tile_off;
  const uint64_t chunk_begin = dcs.chunk_begin;
  const bool vec = dcs.vec_ok != 0;
  const uint32_t inp_mask = dcs.inp_mask;
  const uint64_t U = P.unit_elems;
  const uint64_t cstart = (chunk - chunk_begin) * (4 * U);
  const uint64_t cend = min(cstart + 4 * U, numel);
  const int prim = P.primary;
  // Params fields used by the step lambdas, as locals: the lambdas capture by
  // reference, and a captured by-value argument would live in private memory.
  const int32_t kk = P.k;
  const bool do_tiles = P.do_tiles != 0;
  const uint32_t eqnan_mask = P.eqnan_mask;
  uint32_t *const tile_maps = P.tile_maps;
  // tolerance pairs in registers (constant indices only: a runtime index into
  // the kernel-argument struct would copy it to private memory)
  double atol[NT], rtol[NT];
#pragma unroll
  for (int p = 0; p < NT; ++p) {
    atol[p] = P.atol[p];
    rtol[p] = P.rtol[p];
  }


  // per-lane binary64 sums
  double acc_abs = 0.0, acc_rel = 0.0;
  // wave-uniform exact running maxima (value, chunk offset)
  double best_abs = -1.0, best_rel = -1.0;
  uint32_t arg_abs = 0xffffffffu, arg_rel = 0xffffffffu;
  // merge lane-local candidates into the wave's running maximum
  auto merge_abs = [&](double v, uint32_t i) __attribute__((always_inline)) {
    wave_max(v, i);
    max_merge(best_abs, arg_abs, v, i);
  };
  auto merge_rel = [&](double v, uint32_t i) __attribute__((always_inline)) {
    wave_max(v, i);
    max_merge(best_rel, arg_rel, v, i);
  };
  // wave-uniform counters
  uint32_t mism[NT];
#pragma unroll
  for (int p = 0; p < NT; ++p) mism[p] = 0;
  uint32_t fast_steps = 0;  // steps committed by the fast path
  if (lane < 8) s_rare[wave][lane] = 0;
  uint32_t zc = 0, zr = 0, efc = 0, efr = 0, bfc = 0, bfr = 0, hfc = 0, hfr = 0;
  uint64_t diff_cr = 0;
  uint32_t eqc = INTEG ? inp_mask : 0u, eqr = eqc;
  uint32_t nfound = 0;
  uint32_t first_c = 0, first_r = 0;
  if constexpr (INTEG) {
    if (numel > 0) {
      if constexpr (ES == 4) {
        first_c = *(const VCK_GLOBAL uint32_t *)cand;
        first_r = *(const VCK_GLOBAL uint32_t *)ref;
      } else {
        first_c = *(const VCK_GLOBAL uint16_t *)cand;
        first_r = *(const VCK_GLOBAL uint16_t *)ref;
      }
    }
  }

  // Tile window: LDS counters for the tile-id range this chunk can touch.
  const uint32_t th = (uint32_t)P.tile_h, tw = (uint32_t)P.tile_w;
  bool win_ok = false;
  uint64_t win_base = 0;
  if (do_tiles) {
    const uint64_t row_lo = cstart / cols, row_hi = (cend - 1) / cols;
    uint64_t t_min, t_max;
    if (row_lo == row_hi) {
      t_min = (row_lo / th) * tiles_c + (cstart - row_lo * cols) / tw;
      t_max = (row_lo / th) * tiles_c + (cend - 1 - row_lo * cols) / tw;
    } else {
      t_min = (row_lo / th) * tiles_c;
      t_max = (row_hi / th) * tiles_c + tiles_c - 1;
    }
    win_ok = (t_max - t_min) < (uint64_t)kTileWindow;
    win_base = t_min;
    if (win_ok)
      for (uint32_t e = threadIdx.x; e < (uint32_t)kTileWindow; e += kBlockThreads) s_win[e] = 0;
    __syncthreads();
  }
  uint32_t *const stage =
      P.stage + ((uint64_t)chunk * kWavesPerBlock + wave) * (uint64_t)(kk > 0 ? kk : 0);

  // Localization of the primary-pair mismatches given by per-lane bit mask
  // pb (bit j = element i0 + j): ordered first-k staging and tile counts.
  auto localize = [&](uint32_t pb, uint64_t i0) __attribute__((always_inline)) {
    const uint32_t off0 = (uint32_t)(i0 - cstart);
    if (kk > 0 && nfound < (uint32_t)kk) {
      uint32_t before = 0, total = 0;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const uint64_t b = ballot((pb >> j) & 1u);
        before += lanes_below(b);
        total += popc(b);
      }
      uint32_t pos = nfound + before;
      uint32_t bits = pb;
      while (bits != 0) {
        const int j = __builtin_ctz(bits);
        bits &= bits - 1;
        if (pos < (uint32_t)kk) stage[pos] = off0 + j;
        ++pos;
      }
      nfound = min(nfound + total, (uint32_t)kk);
    }
    if (do_tiles) {
      uint32_t bits = pb;
      while (bits != 0) {
        const int j = __builtin_ctz(bits);
        bits &= bits - 1;
        const uint64_t i = i0 + j;
        const uint64_t row = i / cols;
        const uint64_t col = i - row * cols;
        const uint64_t t = (row / th) * tiles_c + col / tw;
        if (win_ok && t >= win_base && t - win_base < (uint64_t)kTileWindow)
          atomicAdd(&s_win[t - win_base], 1u);
        else
          atomicAdd(&tile_maps[tile_off + t], 1u);
      }
    }
  };

  // Exact binary64 evaluation of one step (element by element).
  auto exact_step = [&](const u32x4 &cq, const u32x4 &rq, uint32_t vmask, uint64_t i0) __attribute__((always_inline)) {
    const uint32_t off0 = (uint32_t)(i0 - cstart);
    uint32_t pb = 0;
    uint32_t nan_c_step = 0, nan_r_step = 0, inf_c_step = 0, inf_r_step = 0;
    uint32_t fin_step = 0, rel_step = 0, undef_step = 0;
    double lb_abs = -1.0, lb_rel = -1.0;  // lane-local maxima of this step
    uint32_t li_abs = 0xffffffffu, li_rel = 0xffffffffu;
#pragma unroll 1
    for (int j = 0; j < V; ++j) {
      const bool valid = (vmask >> j) & 1u;
      const double c = dec64<DT>(elem<DT>(cq, j));
      const double r = dec64<DT>(elem<DT>(rq, j));
      const bool c_nan = __builtin_isnan(c), c_inf = __builtin_isinf(c);
      const bool r_nan = __builtin_isnan(r), r_inf = __builtin_isinf(r);
      nan_c_step += popc(ballot(valid && c_nan));
      inf_c_step += popc(ballot(valid && c_inf));
      nan_r_step += popc(ballot(valid && r_nan));
      inf_r_step += popc(ballot(valid && r_inf));
      const bool fin = valid && !(c_nan || c_inf || r_nan || r_inf);
      const double d = __builtin_fabs(c - r);
      const double a = __builtin_fabs(r);
#pragma unroll
      for (int p = 0; p < NT; ++p) {
        const double t = atol[p] + rtol[p] * a;
        const bool close =
            (c == r) || (fin && d <= t) || (((eqnan_mask >> p) & 1u) && c_nan && r_nan);
        const bool f = valid && !close;
        mism[p] += popc(ballot(f));
        if (p == prim && f) pb |= 1u << j;
      }
      const bool relok = fin && r != 0.0;
      fin_step += popc(ballot(fin));
      rel_step += popc(ballot(relok));
      undef_step += popc(ballot(fin && r == 0.0 && c != 0.0));
      if (fin) {
        acc_abs += d;
        if (d > lb_abs) {
          lb_abs = d;
          li_abs = off0 + j;
        }
      }
      if (relok) {
        const double q = d / a;
        acc_rel += q;
        if (q > lb_rel) {
          lb_rel = q;
          li_rel = off0 + j;
        }
      }
    }
    merge_abs(lb_abs, li_abs);
    merge_rel(lb_rel, li_rel);
    if (lane == 0) {
      uint32_t *const rc = s_rare[wave];
      rc[0] += nan_c_step;
      rc[1] += inf_c_step;
      rc[2] += nan_r_step;
      rc[3] += inf_r_step;
      rc[4] += fin_step;
      rc[5] += rel_step;
      rc[6] += undef_step;
    }
    if constexpr (DT == VC_F32) {
      // NaN is binary16-representable: count it with the representability tests
      hfc += nan_c_step;
      hfr += nan_r_step;
    }
    if (ballot(pb != 0) != 0) localize(pb, i0);
  };

  // Fast path for a full step; returns false (and changes nothing) when the
  // step holds a NaN, an infinity or a zero reference (the exact path then
  // does the per-element class tests). The gate, the running maxima and
  // sum_abs are exact binary64; the lane's quotient estimates feed sum_rel.
  auto fast_step = [&](const u32x4 &cq, const u32x4 &rq, uint64_t i0) __attribute__((always_inline)) -> bool {
    float sq0 = 0.f, sq1 = 0.f;
    double sa = 0.0;
    uint32_t fcnt[NT];
#pragma unroll
    for (int p = 0; p < NT; ++p) fcnt[p] = 0;
    uint64_t pany = 0;
    // lanes with an element whose |c - r| exceeds best_abs / whose exact
    // quotient exceeds best_rel (per-element compares into wave masks; a
    // per-lane OR would be rewritten by the compiler into a max reduction)
    uint64_t absm = 0, relm = 0;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const float c32 = dec32<DT>(elem<DT>(cq, j));
      const float r32 = dec32<DT>(elem<DT>(rq, j));
      const double c = c32, r = r32;
      const double d = __builtin_fabs(c - r);
      const double a = __builtin_fabs(r);
#pragma unroll
      for (int p = 0; p < NT; ++p) {
        const double t = atol[p] + rtol[p] * a;
        const uint64_t f = ballot(!(d <= t));
        fcnt[p] += popc(f);
        if (p == prim) pany |= f;
      }
      sa += d;
      absm |= ballot(d > best_abs);
      relm |= ballot(__builtin_fma(-best_rel, a, d) > 0.0);
      const float q = __builtin_fabsf((float)d * __builtin_amdgcn_rcpf(r32));
      if (j & 1) sq1 += q;
      else sq0 += q;
    }
    // finite iff every c and r of the lane is finite and every r != 0
    if (ballot(!__builtin_isfinite(sq0 + sq1)) != 0) return false;
#pragma unroll
    for (int p = 0; p < NT; ++p) mism[p] += fcnt[p];
    ++fast_steps;
    acc_abs += sa;
    acc_rel += (double)sq0 + (double)sq1;
    const uint32_t off0 = (uint32_t)(i0 - cstart);
    const uint64_t lane_bit = 1ull << lane;
    if (absm != 0) {
      double lb = -1.0;
      uint32_t li = 0xffffffffu;
      if (absm & lane_bit) {
#pragma unroll
        for (int j = 0; j < V; ++j) {  // lane max, smallest j on ties
          const double d = __builtin_fabs(dec64<DT>(elem<DT>(cq, j)) - dec64<DT>(elem<DT>(rq, j)));
          if (d > lb) {
            lb = d;
            li = off0 + j;
          }
        }
      }
      merge_abs(lb, li);
    }
    if (relm != 0) {
      double lb = -1.0;
      uint32_t li = 0xffffffffu;
      if (relm & lane_bit) {
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const double r = dec64<DT>(elem<DT>(rq, j));
          const double d = __builtin_fabs(dec64<DT>(elem<DT>(cq, j)) - r);
          const double a = __builtin_fabs(r);
          // exact sign test: d / a > best_rel  <=>  d - best_rel * a > 0
          if (__builtin_fma(-best_rel, a, d) > 0.0) {
            const double q = d / a;
            if (q > lb) {
              lb = q;
              li = off0 + j;
            }
          }
        }
      }
      merge_rel(lb, li);
    }
    if (pany != 0) {
      uint32_t pb = 0;
#pragma unroll 1
      for (int j = 0; j < V; ++j) {
        const double r = dec64<DT>(elem<DT>(rq, j));
        const double d = __builtin_fabs(dec64<DT>(elem<DT>(cq, j)) - r);
        double t = 0.0;
#pragma unroll
        for (int p = 0; p < NT; ++p)
          if (p == prim) t = atol[p] + rtol[p] * __builtin_fabs(r);
        if (!(d <= t)) pb |= 1u << j;
      }
      localize(pb, i0);
    }
    return true;
  };

  // Degenerate-output detector counts of one step (bitwise; NaN handling of
  // the binary16 test is added by the exact path).
  auto integ_step = [&](const u32x4 &cq, const u32x4 &rq, uint32_t vmask, bool full,
                        uint64_t i0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const bool valid = (vmask >> j) & 1u;
      const uint32_t c = elem<DT>(cq, j), r = elem<DT>(rq, j);
      const float cf = dec32<DT>(c), rf = dec32<DT>(r);
      zc += popc(ballot(valid && cf == 0.0f));
      zr += popc(ballot(valid && rf == 0.0f));
      efc += popc(ballot(valid && c == first_c));
      efr += popc(ballot(valid && r == first_r));
      if constexpr (DT == VC_F32) {
        bfc += popc(ballot(valid && (c & 0xffffu) == 0));
        bfr += popc(ballot(valid && (r & 0xffffu) == 0));
        hfc += popc(ballot(valid && (float)(_Float16)cf == cf));
        hfr += popc(ballot(valid && (float)(_Float16)rf == rf));
      }
      diff_cr |= ballot(valid && c != r);
    }
    // operator inputs: read only while cand or ref is still bit-equal
    uint32_t need = eqc | eqr;
    while (need != 0) {
      const int jx = __builtin_ctz(need);
      need &= need - 1;
      const uint8_t *xp = nullptr;
#pragma unroll
      for (int q = 0; q < VC_MAX_INPUTS; ++q)
        if (q == jx) xp = dcs.inp[q];
      const u32x4 xq = (vec && full) ? load16(xp + i0 * ES) : load_guarded<DT>(xp, i0, cend);
      bool dc = false, dr = false;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const bool valid = (vmask >> j) & 1u;
        const uint32_t x = elem<DT>(xq, j);
        dc |= valid && elem<DT>(cq, j) != x;
        dr |= valid && elem<DT>(rq, j) != x;
      }
      if (ballot(dc) != 0) eqc &= ~(1u << jx);
      if (ballot(dr) != 0) eqr &= ~(1u << jx);
    }
  };

  auto step = [&](const u32x4 &cq, const u32x4 &rq, uint64_t i0) __attribute__((always_inline)) {
    if (!fast_step(cq, rq, i0)) exact_step(cq, rq, ALL, i0);
    if constexpr (INTEG) integ_step(cq, rq, ALL, true, i0);
  };

  // Steps of ITER elements; wave w takes steps w, w+4, w+8, ... of the chunk,
  // so the block streams its chunk front to back, one KiB per wave and tensor.
  const uint64_t n_steps = (cend - cstart) / ITER;  // full steps in the chunk
  const uint64_t n_full = n_steps > wave ? (n_steps - wave + 3) / 4 : 0;
  const uint64_t lane_off = (uint64_t)lane * V;
  auto step_i0 = [&](uint64_t st) __attribute__((always_inline)) { return cstart + (wave + 4 * st) * ITER + lane_off; };
  if (vec) {
    // Two steps per trip with the next step's loads in flight. The loads are
    // unconditional (past the end they re-read the last step, a cache hit) so
    // the wait counters stay exact across the loop.
    const uint8_t *const cb = cand + cstart * ES;  // block-uniform bases
    const uint8_t *const rb = ref + cstart * ES;
    const uint32_t lane_b = lane * 16u;
    const uint64_t last = n_full > 0 ? n_full - 1 : 0;
    auto off = [&](uint64_t st) __attribute__((always_inline)) {
      return (uint32_t)((wave + 4 * min(st, last)) * ITER * ES) + lane_b;
    };
    u32x4 ca = {0, 0, 0, 0}, ra = ca, cn = ca, rn = ca;
    if (n_full > 0) {
      ca = load16(cb + off(0));
      ra = load16(rb + off(0));
    }
    for (uint64_t st = 0; st < n_full; st += 2) {
      cn = load16(cb + off(st + 1));
      rn = load16(rb + off(st + 1));
      step(ca, ra, step_i0(st));
      if (st + 1 >= n_full) break;
      ca = load16(cb + off(st + 2));
      ra = load16(rb + off(st + 2));
      step(cn, rn, step_i0(st + 1));
    }
  } else {
    for (uint64_t st = 0; st < n_full; ++st) {
      const uint64_t i0 = step_i0(st);
      const u32x4 cq = load_guarded<DT>(cand, i0, cend);
      const u32x4 rq = load_guarded<DT>(ref, i0, cend);
      step(cq, rq, i0);
    }
  }
  if ((cend - cstart) % ITER != 0 && n_steps % 4 == wave) {
    const uint64_t i0 = cstart + n_steps * ITER + lane_off;
    const u32x4 ct = load_guarded<DT>(cand, i0, cend);
    const u32x4 rt = load_guarded<DT>(ref, i0, cend);
    uint32_t vmask = 0;
#pragma unroll
    for (int j = 0; j < V; ++j) vmask |= (i0 + j < cend ? 1u : 0u) << j;
    exact_step(ct, rt, vmask, i0);
    if constexpr (INTEG) integ_step(ct, rt, vmask, false, i0);
  }


  // wave reduction (fixed butterfly order)
#pragma unroll
  for (int m = kWaveSize / 2; m >= 1; m >>= 1) {
    acc_abs += __shfl_xor(acc_abs, m);
    acc_rel += __shfl_xor(acc_rel, m);
  }
  if (lane == 0) {
    WaveOut &o = s_out[wave];
#pragma unroll
    for (int p = 0; p < VC_MAX_TOLS; ++p) o.mism[p] = p < NT ? mism[p] : 0u;
    const uint32_t *const rc = s_rare[wave];
    o.nan_c = rc[0];
    o.inf_c = rc[1];
    o.nan_r = rc[2];
    o.inf_r = rc[3];
    o.n_fin = rc[4] + fast_steps * ITER;
    o.n_rel = rc[5] + fast_steps * ITER;
    o.n_rel_undef = rc[6];
    o.eq_bits = (diff_cr == 0 ? kEqCandRef : 0u) | (eqc << kEqCandInpShift) |
                (eqr << kEqRefInpShift);
    o.nfound = nfound;
    o.zc = zc;
    o.zr = zr;
    o.efc = efc;
    o.efr = efr;
    o.bfc = bfc;
    o.bfr = bfr;
    o.hfc = hfc;
    o.hfr = hfr;
    o.max_abs = best_abs;
    o.amax_abs = arg_abs;
    o.max_rel = best_rel;
    o.amax_rel = arg_rel;
    o.sum_abs = acc_abs;
    o.sum_rel = acc_rel;
  }
  __syncthreads();
  // flush the tile window (all four waves are done with it)
  if (do_tiles && win_ok) {
    for (uint32_t e = threadIdx.x; e < (uint32_t)kTileWindow; e += kBlockThreads) {
      const uint32_t v = s_win[e];
      if (v != 0) atomicAdd(&tile_maps[tile_off + win_base + e], v);
    }
  }
  // Merge the four waves' ascending first-k lists (disjoint index sets) into
  // the k smallest: an entry's rank is its position in its own list plus the
  // number of smaller entries in the other three.
  uint32_t merged = 0;
  if (kk > 0) {
    const uint32_t k = (uint32_t)kk;
    uint32_t nf[kWavesPerBlock], total = 0;
    for (int w = 0; w < kWavesPerBlock; ++w) {
      nf[w] = s_out[w].nfound;
      total += nf[w];
    }
    if (total > 0) {
      const uint32_t *base = P.stage + (uint64_t)chunk * kWavesPerBlock * k;
      for (uint32_t e = threadIdx.x; e < kWavesPerBlock * k; e += kBlockThreads) {
        const uint32_t w = e / k, i = e % k;
        if (i >= nf[w]) continue;
        const uint32_t x = base[w * k + i];
        uint32_t rank = i;
        for (uint32_t v = 0; v < (uint32_t)kWavesPerBlock; ++v) {
          if (v == w) continue;
          uint32_t lo = 0, hi = nf[v];  // count of list v below x
          while (lo < hi) {
            const uint32_t mid = (lo + hi) / 2;
            if (base[v * k + mid] < x) lo = mid + 1;
            else hi = mid;
          }
          rank += lo;
        }
        if (rank < k) s_merged[rank] = x;
      }
      merged = min(total, k);
      __syncthreads();
      for (uint32_t e = threadIdx.x; e < merged; e += kBlockThreads)
        P.stage[(uint64_t)chunk * kWavesPerBlock * k + e] = s_merged[e];
    }
  }
  if (threadIdx.x == 0) {
    ChunkRec rec;
    const WaveOut &w0 = s_out[0];
#pragma unroll
    for (int p = 0; p < VC_MAX_TOLS; ++p) rec.mism[p] = w0.mism[p];
    rec.nan_c = w0.nan_c;
    rec.inf_c = w0.inf_c;
    rec.nan_r = w0.nan_r;
    rec.inf_r = w0.inf_r;
    rec.n_fin = w0.n_fin;
    rec.n_rel = w0.n_rel;
    rec.n_rel_undef = w0.n_rel_undef;
    rec.eq_bits = w0.eq_bits;
    rec.zero_c = w0.zc;
    rec.zero_r = w0.zr;
    rec.eqf_c = w0.efc;
    rec.eqf_r = w0.efr;
    rec.bf_c = w0.bfc;
    rec.bf_r = w0.bfr;
    rec.f16_c = w0.hfc;
    rec.f16_r = w0.hfr;
    rec.max_abs = w0.max_abs;
    rec.amax_abs = w0.amax_abs;
    rec.max_rel = w0.max_rel;
    rec.amax_rel = w0.amax_rel;
    rec.sum_abs = w0.sum_abs;
    rec.sum_rel = w0.sum_rel;
    for (int w = 1; w < kWavesPerBlock; ++w) {
      const WaveOut &o = s_out[w];
#pragma unroll
      for (int p = 0; p < VC_MAX_TOLS; ++p) rec.mism[p] += o.mism[p];
      rec.nan_c += o.nan_c;
      rec.inf_c += o.inf_c;
      rec.nan_r += o.nan_r;
      rec.inf_r += o.inf_r;
      rec.n_fin += o.n_fin;
      rec.n_rel += o.n_rel;
      rec.n_rel_undef += o.n_rel_undef;
      rec.eq_bits &= o.eq_bits;
      rec.zero_c += o.zc;
      rec.zero_r += o.zr;
      rec.eqf_c += o.efc;
      rec.eqf_r += o.efr;
      rec.bf_c += o.bfc;
      rec.bf_r += o.bfr;
      rec.f16_c += o.hfc;
      rec.f16_r += o.hfr;
      max_merge(rec.max_abs, rec.amax_abs, o.max_abs, o.amax_abs);
      max_merge(rec.max_rel, rec.amax_rel, o.max_rel, o.amax_rel);
      rec.sum_abs += o.sum_abs;
      rec.sum_rel += o.sum_rel;
    }
    rec.nfound[0] = merged;
    for (int w = 1; w < kWavesPerBlock; ++w) rec.nfound[w] = 0;
    rec.pad0 = rec.pad1 = 0;
    P.recs[chunk] = rec;
  }
}

// ---------------------------------------------------------------- finalize

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
#pragma unroll
  for (int m = kWaveSize / 2; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

__device__ __forceinline__ double wave_sum_f64(double x) {
#pragma unroll
  for (int m = kWaveSize / 2; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

struct FinScratch {
  uint64_t u[kWavesPerBlock];
  double d[kWavesPerBlock];
  uint64_t idx[kWavesPerBlock];
  uint32_t scan[kBlockThreads];
  uint32_t eq[kWavesPerBlock];
};

// Block-wide sums in a fixed order: wave butterfly, then waves 0..3.
__device__ uint64_t block_sum_u64(FinScratch &s, uint64_t x) {
  x = wave_sum_u64(x);
  const uint32_t lane = threadIdx.x & (kWaveSize - 1), wave = threadIdx.x / kWaveSize;
  __syncthreads();
  if (lane == 0) s.u[wave] = x;
  __syncthreads();
  uint64_t t = 0;
  for (int w = 0; w < kWavesPerBlock; ++w) t += s.u[w];
  return t;
}

__device__ double block_sum_f64(FinScratch &s, double x) {
  x = wave_sum_f64(x);
  const uint32_t lane = threadIdx.x & (kWaveSize - 1), wave = threadIdx.x / kWaveSize;
  __syncthreads();
  if (lane == 0) s.d[wave] = x;
  __syncthreads();
  double t = 0.0;
  for (int w = 0; w < kWavesPerBlock; ++w) t += s.d[w];
  return t;
}

// Block-wide (max value, smallest index); idx = UINT64_MAX marks "none".
__device__ void block_max(FinScratch &s, double &v, uint64_t &idx) {
#pragma unroll
  for (int m = kWaveSize / 2; m >= 1; m >>= 1) {
    const double ov = __shfl_xor(v, m);
    const uint64_t oi = __shfl_xor(idx, m);
    if (ov > v || (ov == v && oi < idx)) {
      v = ov;
      idx = oi;
    }
  }
  const uint32_t lane = threadIdx.x & (kWaveSize - 1), wave = threadIdx.x / kWaveSize;
  __syncthreads();
  if (lane == 0) {
    s.d[wave] = v;
    s.idx[wave] = idx;
  }
  __syncthreads();
  v = s.d[0];
  idx = s.idx[0];
  for (int w = 1; w < kWavesPerBlock; ++w)
    if (s.d[w] > v || (s.d[w] == v && s.idx[w] < idx)) {
      v = s.d[w];
      idx = s.idx[w];
    }
}

__device__ uint32_t block_and_u32(FinScratch &s, uint32_t x) {
#pragma unroll
  for (int m = kWaveSize / 2; m >= 1; m >>= 1) x &= __shfl_xor(x, m);
  const uint32_t lane = threadIdx.x & (kWaveSize - 1), wave = threadIdx.x / kWaveSize;
  __syncthreads();
  if (lane == 0) s.eq[wave] = x;
  __syncthreads();
  uint32_t t = 0xffffffffu;
  for (int w = 0; w < kWavesPerBlock; ++w) t &= s.eq[w];
  return t;
}

// Exclusive prefix of x over the block (thread order); returns the total too.
__device__ uint32_t block_exscan_u32(FinScratch &s, uint32_t x, uint32_t &total) {
  __syncthreads();
  s.scan[threadIdx.x] = x;
  __syncthreads();
  for (uint32_t off = 1; off < (uint32_t)kBlockThreads; off <<= 1) {
    const uint32_t v = threadIdx.x >= off ? s.scan[threadIdx.x - off] : 0u;
    __syncthreads();
    s.scan[threadIdx.x] += v;
    __syncthreads();
  }
  total = s.scan[kBlockThreads - 1];
  return s.scan[threadIdx.x] - x;
}

__global__ __launch_bounds__(kBlockThreads) void finalize_kernel(const Params P) {
  __shared__ FinScratch s;
  const uint64_t ci = P.case_lo + blockIdx.x;
  DevCase cs;
  if (P.cases != nullptr) cs = load_case((const VCK_CONST DevCase *)P.cases + ci);
  else cs = P.single;
  const uint32_t oi = cs.orig;
  const int nt = P.n_tols;
  const uint64_t CH = 4ull * cs.unit_elems;
  const uint32_t n_chunks = cs.n_chunks;

  uint64_t mism[VC_MAX_TOLS];
  for (int p = 0; p < VC_MAX_TOLS; ++p) mism[p] = 0;
  uint64_t cnt[7] = {0, 0, 0, 0, 0, 0, 0};
  uint64_t ic[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  double sa = 0.0, sr = 0.0;
  double mav = -1.0, mrv = -1.0;
  uint64_t mai = UINT64_MAX, mri = UINT64_MAX;
  uint32_t eqb = 0xffffffffu;
  for (uint32_t c = threadIdx.x; c < n_chunks; c += kBlockThreads) {
    const ChunkRec &r = P.recs[cs.chunk_begin + c];
    for (int p = 0; p < VC_MAX_TOLS; ++p) mism[p] += r.mism[p];
    cnt[0] += r.nan_c;
    cnt[1] += r.inf_c;
    cnt[2] += r.nan_r;
    cnt[3] += r.inf_r;
    cnt[4] += r.n_fin;
    cnt[5] += r.n_rel;
    cnt[6] += r.n_rel_undef;
    ic[0] += r.zero_c;
    ic[1] += r.zero_r;
    ic[2] += r.eqf_c;
    ic[3] += r.eqf_r;
    ic[4] += r.bf_c;
    ic[5] += r.bf_r;
    ic[6] += r.f16_c;
    ic[7] += r.f16_r;
    eqb &= r.eq_bits;
    sa += r.sum_abs;
    sr += r.sum_rel;
    if (r.amax_abs != 0xffffffffu) {
      const uint64_t gi = (uint64_t)c * CH + r.amax_abs;
      if (r.max_abs > mav || (r.max_abs == mav && gi < mai)) {
        mav = r.max_abs;
        mai = gi;
      }
    }
    if (r.amax_rel != 0xffffffffu) {
      const uint64_t gi = (uint64_t)c * CH + r.amax_rel;
      if (r.max_rel > mrv || (r.max_rel == mrv && gi < mri)) {
        mrv = r.max_rel;
        mri = gi;
      }
    }
  }
  for (int p = 0; p < VC_MAX_TOLS; ++p) mism[p] = block_sum_u64(s, mism[p]);
  for (int q = 0; q < 7; ++q) cnt[q] = block_sum_u64(s, cnt[q]);
  for (int q = 0; q < 8; ++q) ic[q] = block_sum_u64(s, ic[q]);
  sa = block_sum_f64(s, sa);
  sr = block_sum_f64(s, sr);
  block_max(s, mav, mai);
  block_max(s, mrv, mri);
  eqb = block_and_u32(s, eqb);

  const bool ok = cs.status == 0;
  if (!ok) {
    for (int p = 0; p < VC_MAX_TOLS; ++p) mism[p] = 0;
    for (int q = 0; q < 7; ++q) cnt[q] = 0;
    for (int q = 0; q < 8; ++q) ic[q] = 0;
    sa = sr = 0.0;
    mai = mri = UINT64_MAX;
    eqb = 0;
  }
  const uint64_t n = ok ? cs.numel : 0;

  // ordered first-k: walk chunks in order, waves in order
  if (P.first_k != nullptr && P.k > 0) {
    const uint32_t k = (uint32_t)P.k;
    int64_t *const fk = P.first_k + (uint64_t)oi * k;
    uint32_t carry = 0;
    if (ok) {
      for (uint32_t b = 0; b < n_chunks && carry < k; b += kBlockThreads) {
        const uint32_t c = b + threadIdx.x;
        uint32_t cntc = 0;
        const ChunkRec *r = c < n_chunks ? &P.recs[cs.chunk_begin + c] : nullptr;
        if (r != nullptr)
          for (int w = 0; w < kWavesPerBlock; ++w) cntc += r->nfound[w];
        uint32_t total;
        const uint32_t ex = block_exscan_u32(s, cntc, total);
        if (cntc != 0 && carry + ex < k) {
          uint32_t pos = carry + ex;
          for (int w = 0; w < kWavesPerBlock && pos < k; ++w) {
            const uint32_t *st = P.stage + ((cs.chunk_begin + c) * kWavesPerBlock + w) * k;
            for (uint32_t e = 0; e < r->nfound[w] && pos < k; ++e, ++pos)
              fk[pos] = (int64_t)((uint64_t)c * CH + st[e]);
          }
        }
        carry = min(carry + total, k);
      }
    }
    for (uint32_t pos = carry + threadIdx.x; pos < k; pos += kBlockThreads) fk[pos] = -1;
  }

  if (threadIdx.x != 0) return;
  const int prim = P.primary;
  vc_stats st;
  st.numel = cs.numel;
  st.mismatches = mism[prim];
  st.nan_cand = cnt[0];
  st.inf_cand = cnt[1];
  st.nan_ref = cnt[2];
  st.inf_ref = cnt[3];
  st.n_finite = cnt[4];
  st.n_rel = cnt[5];
  st.n_rel_undef = cnt[6];
  st.max_abs = mai == UINT64_MAX ? 0.0 : mav;
  st.argmax_abs = mai == UINT64_MAX ? -1 : (int64_t)mai;
  st.max_rel = mri == UINT64_MAX ? 0.0 : mrv;
  st.argmax_rel = mri == UINT64_MAX ? -1 : (int64_t)mri;
  st.sum_abs = sa;
  st.sum_rel = sr;
  st.case_status = cs.status;
  st.pass = (ok && mism[prim] == 0) ? 1 : 0;
  if (P.stats != nullptr) P.stats[oi] = st;
  for (int p = 0; p < nt; ++p) {
    const uint8_t pass = (ok && mism[p] == 0) ? 1 : 0;
    P.ws_pass[(uint64_t)oi * nt + p] = pass;
    if (P.pass_out != nullptr) P.pass_out[(uint64_t)oi * nt + p] = pass;
    if (P.mismatches != nullptr) P.mismatches[(uint64_t)oi * nt + p] = mism[p];
  }
  uint32_t flags = 0;
  if (P.do_integ) {
    vc_integrity g;
    g.zero_cand = ic[0];
    g.zero_ref = ic[1];
    g.eqfirst_cand = ic[2];
    g.eqfirst_ref = ic[3];
    g.bf16rep_cand = ic[4];
    g.bf16rep_ref = ic[5];
    g.fp16rep_cand = ic[6];
    g.fp16rep_ref = ic[7];
    const uint32_t inp_mask = ok ? cs.inp_mask : 0u;
    const uint32_t eq_c = (eqb >> kEqCandInpShift) & 0xffu & inp_mask;
    const uint32_t eq_r = (eqb >> kEqRefInpShift) & 0xffu & inp_mask;
    g.cand_eq_input_mask = eq_c;
    g.ref_eq_input_mask = eq_r;
    g.cand_eq_ref = ok ? (eqb & kEqCandRef) : 0u;
    g.copy_input = -1;
    if (ok) {
      const bool f32 = cs.dtype == VC_F32;
      if (ic[0] == n && n >= 1 && ic[1] < n) flags |= VC_FLAG_ALL_ZERO;
      if (ic[2] == n && n >= 2 && ic[0] < n && ic[3] < n) flags |= VC_FLAG_CONSTANT;
      const uint32_t copy = eq_c & ~eq_r;
      if (copy != 0) {
        flags |= VC_FLAG_INPUT_COPY;
        g.copy_input = __builtin_ctz(copy);
      }
      if (f32 && ic[4] == n && n >= 2 && ic[0] < n && ic[2] < n && ic[5] < n)
        flags |= VC_FLAG_LOWPREC_BF16;
      if (f32 && ic[6] == n && ic[4] < n && n >= 2 && ic[0] < n && ic[2] < n && ic[7] < n)
        flags |= VC_FLAG_LOWPREC_FP16;
    }
    g.flags = flags;
    g.reserved = 0;
    if (P.integ != nullptr) P.integ[oi] = g;
  }
  P.ws_flags[oi] = flags;
}

// Suite match rates: certified (and numerically passing) cases per pair.
__global__ __launch_bounds__(kBlockThreads) void rates_kernel(const Params P) {
  __shared__ FinScratch s;
  const int nt = P.n_tols;
  for (int p = 0; p < nt; ++p) {
    uint64_t cert = 0, num = 0;
    for (uint64_t c = threadIdx.x; c < (uint64_t)P.n_cases; c += kBlockThreads) {
      const bool pass = P.ws_pass[c * nt + p] != 0;
      num += pass;
      cert += pass && (!P.do_integ || P.ws_flags[c] == 0);
    }
    cert = block_sum_u64(s, cert);
    num = block_sum_u64(s, num);
    if (threadIdx.x == 0) {
      const double n = (double)P.n_cases;
      if (P.match_rate != nullptr) P.match_rate[p] = P.n_cases > 0 ? (double)cert / n : 0.0;
      if (P.numeric_rate != nullptr) P.numeric_rate[p] = P.n_cases > 0 ? (double)num / n : 0.0;
    }
  }
}

__global__ void fill_u32_kernel(uint32_t *p, uint64_t n) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

template <int DT, int NT, bool INTEG>
hipError_t launch_main_t(const Params &p, uint64_t n_chunks, hipStream_t s) {
  hipLaunchKernelGGL((main_kernel<DT, NT, INTEG>), dim3((uint32_t)n_chunks), dim3(kBlockThreads),
                     0, s, p);
  return hipGetLastError();
}

template <int DT, bool INTEG>
hipError_t launch_main_nt(int nt_class, const Params &p, uint64_t n_chunks, hipStream_t s) {
  switch (nt_class) {
    case 1: return launch_main_t<DT, 1, INTEG>(p, n_chunks, s);
    case 2: return launch_main_t<DT, 2, INTEG>(p, n_chunks, s);
    case 4: return launch_main_t<DT, 4, INTEG>(p, n_chunks, s);
    default: return launch_main_t<DT, 8, INTEG>(p, n_chunks, s);
  }
}

template <int DT>
hipError_t launch_main_dt(int nt_class, int integ, const Params &p, uint64_t n_chunks,
                          hipStream_t s) {
  return integ ? launch_main_nt<DT, true>(nt_class, p, n_chunks, s)
               : launch_main_nt<DT, false>(nt_class, p, n_chunks, s);
}

}  // namespace

hipError_t launch_fill_u32(uint32_t *p, uint64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const uint64_t blocks = (n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_main(int dtype, int nt_class, int integ, const Params &p, uint64_t n_chunks,
                       hipStream_t s) {
  if (n_chunks == 0) return hipSuccess;
  switch (dtype) {
    case VC_F32: return launch_main_dt<VC_F32>(nt_class, integ, p, n_chunks, s);
    case VC_F16: return launch_main_dt<VC_F16>(nt_class, integ, p, n_chunks, s);
    default: return launch_main_dt<VC_BF16>(nt_class, integ, p, n_chunks, s);
  }
}

hipError_t launch_finalize(const Params &p, uint64_t n_cases_in_table, hipStream_t s) {
  if (n_cases_in_table == 0) return hipSuccess;
  hipLaunchKernelGGL(finalize_kernel, dim3((uint32_t)n_cases_in_table), dim3(kBlockThreads), 0,
                     s, p);
  return hipGetLastError();
}

hipError_t launch_rates(const Params &p, hipStream_t s) {
  hipLaunchKernelGGL(rates_kernel, dim3(1), dim3(kBlockThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace vck
