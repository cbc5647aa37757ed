// vcheck_probe.hip -- gfx950 kernels of the diagnostic statistics and the
// evidence: the tensor-statistics probe, the near-pass statistics and the
// content hash.
//
// The diagnostic instrumentation of the repair loop records multi-level
// tensor statistics at pipeline boundaries (Sec. 4.2; the instrumentation
// panel of the mechanisms figure). One call probes a batch of tensors in one
// streaming pass: counts of NaN, Inf, zero and finite elements, the first
// smallest and largest finite value, binary64 sums of x, x^2 and |x|, and a
// histogram of binary exponents.
//
// Work decomposition: a tensor is cut into chunks of 4 * U elements; one
// block (4 waves) owns one chunk and each wave streams one contiguous
// quarter, one 16-byte load per lane and step. Each block writes one chunk
// record; a merge launch combines up to 256 chunk records per group in a
// fixed order (writing the tensor's statistics when it has one group), and a
// last launch combines the group records of larger tensors. Kernel
// boundaries order the launches; no floating-point atomics are used, so the
// results are bit-reproducible.
//
// Histogram: 32-bit counters in LDS, slot-major, one column per lane
// position that the block's four waves share (the increments are LDS
// atomics): the counter of slot b for lane l is word 64 b + l, so the 64
// lanes of one increment always hit 64 different banks. Slots 0..63 are the
// bins, slot 64 counts the zeros of the usual steps (binary16 zeros go to
// slot 16 instead, the bin of 2^-25, which no non-zero binary16 value
// reaches). No counter can overflow. The columns are summed when the chunk
// is done.
#pragma clang fp contract(off)

#include "vcheck_internal.h"

namespace vck {
namespace {

constexpr int kPWaves = 4;
constexpr int kPThreads = kPWaves * 64;
constexpr int kPSlots = kHistBins + 1;  // the bins, then the zero slot
// Binary32 exponent field of the bin below binary16's smallest subnormal
// (2^-24 has field 103): binary16 zeros are clamped up to it.
constexpr uint32_t kF16ZeroField = 102;
constexpr uint32_t kF16ZeroBin = kF16ZeroField - 127 - kHistEmin + 1;
static_assert(kF16ZeroBin == 16, "bin of 2^-25");

#define PRB_GLOBAL __attribute__((address_space(1)))

typedef uint32_t p32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 ph2 __attribute__((ext_vector_type(2)));  // a word's two binary16 values

__device__ __forceinline__ p32x4 pload16(const uint8_t *p) {
  return __builtin_nontemporal_load((const PRB_GLOBAL p32x4 *)(p));
}

// Raw buffer resources: the fourth descriptor word of the gfx9 family for
// untyped dword accesses; offsets at or beyond the record count read 0.
constexpr int kBufferWord3 = 0x00020000;
// 16-byte nontemporal load at byte voff + soff of a raw buffer.
__device__ __forceinline__ p32x4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 2 /* nt */);
}

// Exact binary32 value of element j (of V) of a 16-byte vector.
template <int DT>
__device__ __forceinline__ float pdec(const p32x4 &q, int j) {
  if constexpr (DT == VC_F32) {
    return __uint_as_float(q[j]);
  } else {
    const uint32_t w = q[j >> 1];
    const uint32_t h = (j & 1) ? (w >> 16) : (w & 0xffffu);
    if constexpr (DT == VC_BF16) return __uint_as_float(h << 16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
  }
}

// Element loads of indices i0 .. i0 + V - 1 below n (others read as 0).
template <int DT>
__device__ __forceinline__ p32x4 pload_guarded(const uint8_t *base, uint64_t i0, uint64_t n) {
  constexpr int V = DT == VC_F32 ? 4 : 8;
  uint32_t v[V];
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const uint64_t i = i0 + j;
    uint32_t x = 0;
    if (i < n) {
      if constexpr (DT == VC_F32) x = *(const PRB_GLOBAL uint32_t *)(base + i * 4);
      else x = *(const PRB_GLOBAL uint16_t *)(base + i * 2);
    }
    v[j] = x;
  }
  p32x4 r;
  if constexpr (DT == VC_F32) {
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

// Last entry in [0, n) whose value in `first` is <= x (first ascends and
// first[0] <= x), found by one wave: each lane tests one of 64 evenly spaced
// probes and the ballot counts those at or below x, narrowing the range
// 64-fold per round. Uniform result.
__device__ __forceinline__ uint32_t find_first(const uint64_t *first, uint32_t n, uint64_t x) {
  const PRB_GLOBAL uint64_t *f = (const PRB_GLOBAL uint64_t *)first;
  const uint32_t lane = threadIdx.x & 63u;
  uint32_t lo = 0;
  while (n > 64) {
    const uint32_t stride = (n + 63) / 64;
    const uint32_t idx = lo + lane * stride;
    const bool le = lane * stride < n ? f[idx] <= x : false;
    const uint32_t k = (uint32_t)__popcll(__ballot(le)) - 1u;
    lo += k * stride;
    n = min(stride, n - k * stride);
  }
  const bool le = lane < n ? f[lo + lane] <= x : false;
  return lo + (uint32_t)__popcll(__ballot(le)) - 1u;
}

// Wave-wide minimum (MAX = false) or maximum of v, wave-uniform: row shifts
// by 1, 2, 3, 4 and 8 (DPP) leave each row's extreme in its last lane, two
// row broadcasts carry the rows' extremes to lane 63. Lanes with no source
// see the identity (+inf / -inf).
template <int CTRL, int ROWS, bool MAX>
__device__ __forceinline__ float dpp_ext(float v) {
  const uint32_t o = __builtin_amdgcn_update_dpp(MAX ? 0xff800000u : 0x7f800000u,
                                                 __float_as_uint(v), CTRL, ROWS, 0xf, false);
  return MAX ? __builtin_fmaxf(v, __uint_as_float(o)) : __builtin_fminf(v, __uint_as_float(o));
}
template <bool MAX>
__device__ __forceinline__ float wave_ext(float v) {
  v = dpp_ext<0x111, 0xf, MAX>(v);  // row_shr:1
  v = dpp_ext<0x112, 0xf, MAX>(v);  // row_shr:2
  v = dpp_ext<0x113, 0xf, MAX>(v);  // row_shr:3
  v = dpp_ext<0x114, 0xf, MAX>(v);  // row_shr:4
  v = dpp_ext<0x118, 0xf, MAX>(v);  // row_shr:8
  v = dpp_ext<0x142, 0xa, MAX>(v);  // row_bcast:15
  v = dpp_ext<0x143, 0xc, MAX>(v);  // row_bcast:31
  return __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(v), 63));
}

// Wave-wide maximum of v (values -1 or >= 0), wave-uniform, the same way.
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_max_d(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)b, CTRL, ROWS, 0xf, false);
  const uint32_t hi =
      __builtin_amdgcn_update_dpp(0xbff00000u, (uint32_t)(b >> 32), CTRL, ROWS, 0xf, false);
  return __builtin_fmax(v, __longlong_as_double((long long)(((uint64_t)hi << 32) | lo)));
}
__device__ __forceinline__ double wave_max_d(double v) {
  v = dpp_max_d<0x111, 0xf>(v);
  v = dpp_max_d<0x112, 0xf>(v);
  v = dpp_max_d<0x113, 0xf>(v);
  v = dpp_max_d<0x114, 0xf>(v);
  v = dpp_max_d<0x118, 0xf>(v);
  v = dpp_max_d<0x142, 0xa>(v);
  v = dpp_max_d<0x143, 0xc>(v);
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)b, 63);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(b >> 32), 63);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// (value, index) of the smaller / larger of two candidates; equal values
// keep the smaller index; index -1 marks no candidate.
__device__ __forceinline__ void pick_min(double &v, int64_t &i, double v2, int64_t i2) {
  if (i2 < 0) return;
  if (i < 0 || v2 < v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}
__device__ __forceinline__ void pick_max(double &v, int64_t &i, double v2, int64_t i2) {
  if (i2 < 0) return;
  if (i < 0 || v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

// One step of a 64-bit DPP pattern: the value CTRL moves in (lanes with no
// source, or outside the rows ROWS enables, see id).
template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t dpp64(uint64_t x, uint64_t id) {
  const uint32_t lo = __builtin_amdgcn_update_dpp((uint32_t)id, (uint32_t)x, CTRL, ROWS, 0xf, false);
  const uint32_t hi =
      __builtin_amdgcn_update_dpp((uint32_t)(id >> 32), (uint32_t)(x >> 32), CTRL, ROWS, 0xf, false);
  return (uint64_t)hi << 32 | lo;
}

// Wave-wide reduction of a 64-bit value with op, wave-uniform, in a fixed
// order: row shifts by 1, 2, 4 and 8 and two row broadcasts (an inclusive
// scan whose last lane holds the result); id is op's identity.
template <typename Op>
__device__ __forceinline__ uint64_t wave_reduce64(uint64_t x, uint64_t id, Op op) {
  x = op(x, dpp64<0x111, 0xf>(x, id));  // row_shr:1
  x = op(x, dpp64<0x112, 0xf>(x, id));  // row_shr:2
  x = op(x, dpp64<0x114, 0xf>(x, id));  // row_shr:4
  x = op(x, dpp64<0x118, 0xf>(x, id));  // row_shr:8
  x = op(x, dpp64<0x142, 0xa>(x, id));  // row_bcast:15
  x = op(x, dpp64<0x143, 0xc>(x, id));  // row_bcast:31
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, 63);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), 63);
  return (uint64_t)hi << 32 | lo;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
  return wave_reduce64(x, 0ull, [](uint64_t a, uint64_t b) { return a + b; });
}
__device__ __forceinline__ double wave_sum_f64(double x) {
  return __longlong_as_double((long long)wave_reduce64(
      (uint64_t)__double_as_longlong(x), 0ull, [](uint64_t a, uint64_t b) {
        return (uint64_t)__double_as_longlong(__longlong_as_double((long long)a) +
                                              __longlong_as_double((long long)b));
      }));
}
// The wave's (value, index) extreme among lanes with index >= 0: the
// smallest (MAX = false) or largest value, then the smallest index holding
// it; index -1 when no lane has one.
template <bool MAX>
__device__ __forceinline__ void wave_pick(double &v, int64_t &i) {
  const double none = MAX ? -__builtin_inf() : __builtin_inf();
  const double x = i >= 0 ? v : none;
  const double e = __longlong_as_double((long long)wave_reduce64(
      (uint64_t)__double_as_longlong(x), (uint64_t)__double_as_longlong(none),
      [](uint64_t a, uint64_t b) {
        const double da = __longlong_as_double((long long)a), db = __longlong_as_double((long long)b);
        return (uint64_t)__double_as_longlong(MAX ? __builtin_fmax(da, db) : __builtin_fmin(da, db));
      }));
  const uint64_t k = wave_reduce64((i >= 0 && x == e) ? (uint64_t)i : UINT64_MAX, UINT64_MAX,
                                   [](uint64_t a, uint64_t b) { return a < b ? a : b; });
  v = e;
  i = k == UINT64_MAX ? -1 : (int64_t)k;
}

// LDS of the streaming kernel: the histogram columns while streaming, the
// per-thread partials of the chunk afterwards (counts, binary32 extremes and
// their offsets from the chunk's first element all fit 32 bits), so that
// eight blocks fit one compute unit.
constexpr uint32_t kNoOff = 0xffffffffu;  // no finite element yet
struct alignas(16) ChunkLds {
  union {
    uint32_t hist[kPSlots * 64];
    struct {
      double d[3][kPThreads];
      float v[2][kPThreads];
      uint32_t o[2][kPThreads];
      uint32_t n[4][kPThreads];
    };
  };
  uint32_t tensor;
};

// LDS of the merge launches.
struct ProbeLds {
  // per-thread partials
  double d[3][kPThreads];
  double mv[2][kPThreads];
  int64_t mi[2][kPThreads];
  uint64_t c[4][kPThreads];
  // per-wave totals of block_reduce
  uint64_t wc[4][kPWaves];
  double wd[3][kPWaves], wv[2][kPWaves];
  int64_t wi[2][kPWaves];
  uint32_t tensor;
};

// Fixed-order reduction of the per-thread partials in s (256 threads; each
// thread's own slots) into a record (valid in thread 0): DPP wave
// reductions, then the four waves in order.
__device__ void block_reduce(ProbeLds &s, ProbeRec &r) {
  const uint32_t t = threadIdx.x, lane = t & 63u, wave = t >> 6;
  uint64_t c[4];
  double d[3], v[2];
  int64_t i[2];
#pragma unroll
  for (int f = 0; f < 4; ++f) c[f] = wave_sum_u64(s.c[f][t]);
#pragma unroll
  for (int f = 0; f < 3; ++f) d[f] = wave_sum_f64(s.d[f][t]);
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    v[f] = s.mv[f][t];
    i[f] = s.mi[f][t];
  }
  wave_pick<false>(v[0], i[0]);
  wave_pick<true>(v[1], i[1]);
  if (lane == 0) {
#pragma unroll
    for (int f = 0; f < 4; ++f) s.wc[f][wave] = c[f];
#pragma unroll
    for (int f = 0; f < 3; ++f) s.wd[f][wave] = d[f];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      s.wv[f][wave] = v[f];
      s.wi[f][wave] = i[f];
    }
  }
  __syncthreads();
  if (t == 0) {
    uint64_t cc[4] = {0, 0, 0, 0};
    double dd[3] = {0.0, 0.0, 0.0};
    double mn = 0.0, mx = 0.0;
    int64_t imn = -1, imx = -1;
    for (int w = 0; w < kPWaves; ++w) {
#pragma unroll
      for (int f = 0; f < 4; ++f) cc[f] += s.wc[f][w];
#pragma unroll
      for (int f = 0; f < 3; ++f) dd[f] += s.wd[f][w];
      pick_min(mn, imn, s.wv[0][w], s.wi[0][w]);
      pick_max(mx, imx, s.wv[1][w], s.wi[1][w]);
    }
    r.nan = cc[0];
    r.inf = cc[1];
    r.zero = cc[2];
    r.fin = cc[3];
    r.sum = dd[0];
    r.sum_sq = dd[1];
    r.sum_abs = dd[2];
    r.argmin = imn;
    r.argmax = imx;
    r.min = imn < 0 ? 0.0 : mn;
    r.max = imx < 0 ? 0.0 : mx;
  }
}

// (value, offset) of the smaller (MAX = false) or larger of two binary32
// candidates; equal values keep the smaller offset; kNoOff marks none.
template <bool MAX>
__device__ __forceinline__ void pick_off(float &v, uint32_t &o, float v2, uint32_t o2) {
  if (o2 == kNoOff) return;
  if (o == kNoOff || (MAX ? v2 > v : v2 < v) || (v2 == v && o2 < o)) {
    v = v2;
    o = o2;
  }
}

// Fixed-order tree reduction of the per-thread partials of the chunk that
// starts at element c0 into its record, written by thread 0. Its levels
// below 64 threads occupy one wave, so it costs fewer vector instructions
// than the DPP form that the merge launches use.
__device__ void chunk_reduce(ChunkLds &s, uint64_t c0, ProbeRec *rec) {
  const uint32_t t = threadIdx.x;
  for (uint32_t w = kPThreads / 2; w >= 1; w >>= 1) {
    __syncthreads();
    if (t < w) {
#pragma unroll
      for (int f = 0; f < 3; ++f) s.d[f][t] += s.d[f][t + w];
#pragma unroll
      for (int f = 0; f < 4; ++f) s.n[f][t] += s.n[f][t + w];
      pick_off<false>(s.v[0][t], s.o[0][t], s.v[0][t + w], s.o[0][t + w]);
      pick_off<true>(s.v[1][t], s.o[1][t], s.v[1][t + w], s.o[1][t + w]);
    }
  }
  __syncthreads();
  if (t == 0) {
    rec->nan = s.n[0][0];
    rec->inf = s.n[1][0];
    rec->zero = s.n[2][0];
    rec->fin = s.n[3][0];
    rec->argmin = s.o[0][0] == kNoOff ? -1 : (int64_t)(c0 + s.o[0][0]);
    rec->argmax = s.o[1][0] == kNoOff ? -1 : (int64_t)(c0 + s.o[1][0]);
    rec->min = s.o[0][0] == kNoOff ? 0.0 : (double)s.v[0][0];
    rec->max = s.o[1][0] == kNoOff ? 0.0 : (double)s.v[1][0];
    rec->sum = s.d[0][0];
    rec->sum_sq = s.d[1][0];
    rec->sum_abs = s.d[2][0];
    rec->pad[0] = 0;
  }
}

// Stream one chunk: per-lane partials, then the chunk record.
template <int DT>
__device__ void probe_chunk(ChunkLds &s, const ProbeTensor &T, uint64_t c0, uint64_t c1,
                            uint32_t U, ProbeRec *rec) {
  constexpr int V = DT == VC_F32 ? 4 : 8;
  constexpr int ES = DT == VC_F32 ? 4 : 2;
  constexpr uint32_t ITER = 64 * V;
  const uint32_t t = threadIdx.x, lane = t & 63u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(t >> 6);
  for (uint32_t w = t; w < (uint32_t)(kPSlots * 64); w += kPThreads) s.hist[w] = 0;
  __syncthreads();
  // lane's column; col[64 * b] is its counter of slot b
  uint32_t *const col = s.hist + lane;
  const uint64_t w0 = min(c0 + (uint64_t)wave * U, c1), w1 = min(w0 + U, c1);
  const bool vec = ((uintptr_t)T.data % 16) == 0;
  uint32_t n_nan = 0, n_inf = 0, n_zero = 0, n_fin = 0;
  uint32_t n_usual = 0;  // usual steps (uniform): V finite elements per lane each
  float mn = __builtin_inff(), mx = -__builtin_inff();
  uint32_t imn = kNoOff, imx = kNoOff;  // offsets from c0
  double sm = 0.0, sq = 0.0, sa = 0.0;
  // the wave's extremes so far (uniform; +inf / -inf before any finite
  // element)
  float wmn = __builtin_inff(), wmx = -__builtin_inff();
  // Usual step: every element finite (and all below w1). Binary16 screens
  // on the packed halves with the NaN-propagating minimum and maximum
  // (v_pk_minimum3_f16 / v_pk_maximum3_f16; -0 orders below +0, which no
  // comparison below can tell apart): a NaN or an infinity among the
  // elements shows in the step's smallest or largest value, which the step
  // keeps for its extremes screen. The other types test the packed words: an
  // exponent field of all ones carries into the sign bit when its lowest
  // bit is added.
  auto is_usual = [&](const p32x4 &q, float &smn, float &smx) {
    if constexpr (DT == VC_F16) {
      // (each word is copied to a scalar before the cast: a cast of the
      // vector element itself reads the vector's first word)
      const uint32_t u0 = q[0], u1 = q[1], u2 = q[2], u3 = q[3];
      const ph2 h0 = __builtin_bit_cast(ph2, u0), h1 = __builtin_bit_cast(ph2, u1);
      const ph2 h2 = __builtin_bit_cast(ph2, u2), h3 = __builtin_bit_cast(ph2, u3);
      const ph2 lo = __builtin_elementwise_minimum(__builtin_elementwise_minimum(h0, h1),
                                                   __builtin_elementwise_minimum(h2, h3));
      const ph2 hi = __builtin_elementwise_maximum(__builtin_elementwise_maximum(h0, h1),
                                                   __builtin_elementwise_maximum(h2, h3));
      smn = (float)__builtin_elementwise_minimum(lo[0], lo[1]);
      smx = (float)__builtin_elementwise_maximum(hi[0], hi[1]);
      return __ballot(!(smn >= -65504.0f && smx <= 65504.0f)) == 0;
    } else {
      constexpr uint32_t kMag = DT == VC_F32 ? 0x7fffffffu : 0x7fff7fffu;
      constexpr uint32_t kTop = DT == VC_F32 ? 0x80000000u : 0x80008000u;
      constexpr uint32_t kCarry = DT == VC_F32 ? 0x00800000u : 0x00800080u;
      uint32_t nf = 0;
#pragma unroll
      for (int w = 0; w < 4; ++w) nf |= (q[w] & kMag) + kCarry;
      return __ballot((nf & kTop) != 0) == 0;
    }
  };
  // A usual step adds to the sums, counts and histogram with no branch per
  // element (a zero is counted in the zero slot). When no element lies
  // beyond the wave's extremes no lane's first minimum or maximum can change
  // (an element equal to an extreme comes after it); otherwise the lanes
  // take their new extremes by selects, in index order, and the wave's
  // extremes are raised.
  auto usual_step = [&](const p32x4 &q, uint32_t o0, float smn, float smx) {
    float x[V];
#pragma unroll
    for (int j = 0; j < V; ++j) x[j] = pdec<DT>(q, j);
    ++n_usual;
    if constexpr (DT == VC_F16) {
      // Binary16: the step's sums are formed in binary32 before one
      // binary64 addition per sum. A product of two binary16 values is exact in
      // binary32 and every partial sum stays inside its range, so a
      // step's sum of 8 terms errs by at most 7 * 2^-24 of the sum of
      // the terms' magnitudes. Bins: binary16 exponents (subnormals
      // included, through the exact binary32 value) lie inside the
      // histogram's range, so no clamping; a zero (field 0) is raised
      // to field kF16ZeroField, the zero slot.
      // counter of exponent field e: col_f[64 e] (fields 102 .. 142)
      uint32_t *const col_f = col - 64 * (127 + kHistEmin - 1);
      float f1 = x[0], f2 = 0.0f, f3 = 0.0f;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        if (j > 0) f1 += x[j];
        f2 = __builtin_fmaf(x[j], x[j], f2);
        f3 += __builtin_fabsf(x[j]);
        const uint32_t e = max((__float_as_uint(x[j]) >> 23) & 0xffu, kF16ZeroField);
        atomicAdd(col_f + 64 * e, 1u);
      }
      sm += (double)f1;
      sq += (double)f2;
      sa += (double)f3;
    } else {
      smn = __builtin_inff();
      smx = -__builtin_inff();
#pragma unroll
      for (int j = 0; j < V; ++j) {
        smn = __builtin_fminf(smn, x[j]);
        smx = __builtin_fmaxf(smx, x[j]);
        const double xd = (double)x[j];
        sm += xd;
        sq = __builtin_fma(xd, xd, sq);
        sa += __builtin_fabs(xd);
        const int e = (int)((__float_as_uint(x[j]) >> 23) & 0xffu);
        const int bin =
            x[j] == 0.0f ? kHistBins : min(max(e - 127 - kHistEmin + 1, 0), kHistBins - 1);
        atomicAdd(col + 64 * bin, 1u);
      }
    }
    if (__ballot(smn < wmn || smx > wmx) != 0) {
      // every element is finite: the first one beats the lane's +inf /
      // -inf start, so no "no extreme yet" test is needed
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const bool lo = x[j] < mn, hi = x[j] > mx;
        mn = lo ? x[j] : mn;
        imn = lo ? o0 + (uint32_t)j : imn;
        mx = hi ? x[j] : mx;
        imx = hi ? o0 + (uint32_t)j : imx;
      }
      wmn = wave_ext<false>(mn);
      wmx = wave_ext<true>(mx);
    }
  };
  // Any other step, element by element (elements from w1 on are skipped).
  const uint32_t ow1 = (uint32_t)(w1 - c0);
  auto elem_step = [&](const p32x4 &q, uint32_t o0) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      if (o0 + (uint32_t)j >= ow1) break;
      const float x = pdec<DT>(q, j);
      const bool isn = x != x;
      const bool isi = __builtin_fabsf(x) == __builtin_inff();
      n_nan += isn ? 1u : 0u;
      n_inf += isi ? 1u : 0u;
      if (isn || isi) continue;
      ++n_fin;
      const uint32_t o = o0 + (uint32_t)j;
      if (x < mn || imn == kNoOff) {
        mn = x;
        imn = o;
      }
      if (x > mx || imx == kNoOff) {
        mx = x;
        imx = o;
      }
      const double xd = (double)x;
      sm += xd;
      sq = __builtin_fma(xd, xd, sq);  // x*x is exact in binary64
      sa += __builtin_fabs(xd);
      if (x == 0.0f) {
        ++n_zero;
      } else {
        const uint32_t e = (__float_as_uint(x) >> 23) & 0xffu;
        const int bin = e == 0 ? 0 : min(max((int)e - 127 - kHistEmin + 1, 0), kHistBins - 1);
        atomicAdd(col + 64 * bin, 1u);
      }
    }
    // raise the wave's extremes to the lanes' (lanes with no finite element
    // hold +inf / -inf)
    wmn = wave_ext<false>(mn);
    wmx = wave_ext<true>(mx);
  };
  // The full steps through a buffer resource over them (a wave's range is
  // at most 128 KiB: 32-bit offsets, uniform ones in scalar registers),
  // each step's loads issued one step ahead (the last step loads itself
  // again: no branch for it). Runs of usual steps take an inner loop of
  // their own.
  const uint32_t nst = vec ? (uint32_t)((w1 - w0) / ITER) : 0u;
  if (nst > 0) {
    constexpr uint32_t SB = ITER * ES;  // bytes per step
    const uint32_t last = (nst - 1) * SB;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(T.data + w0 * ES), (short)0, (int)(nst * SB), kBufferWord3);
    const uint32_t loff = lane * 16u;                           // lane's bytes in a step
    const uint32_t ol = (uint32_t)(w0 - c0) + lane * (uint32_t)V;  // lane's first offset
    uint32_t k = 0;  // the step's first byte
    p32x4 qn = bload16(rs, loff, 0u);
    while (true) {
      p32x4 q = qn;
      qn = bload16(rs, loff, min(k + SB, last));
      float smn = 0.0f, smx = 0.0f;  // (binary16: set by the screen)
      bool usual = is_usual(q, smn, smx);
      while (usual) {
        usual_step(q, ol + k / ES, smn, smx);
        k += SB;
        if (k > last) break;
        q = qn;
        qn = bload16(rs, loff, min(k + SB, last));
        usual = is_usual(q, smn, smx);
      }
      if (usual) break;  // (past the last step)
      elem_step(q, ol + k / ES);
      k += SB;
      if (k > last) break;
    }
  }
  for (uint64_t b = w0 + (uint64_t)nst * ITER; b < w1; b += ITER) {
    const uint64_t i0 = b + (uint64_t)lane * V;
    const p32x4 q = pload_guarded<DT>(T.data, i0, w1);
    elem_step(q, (uint32_t)(i0 - c0));
  }
  n_fin += V * n_usual;
  __syncthreads();  // every wave's counts are in
  // zeros of the usual steps: wave 0 adds the zero slot's column
  constexpr uint32_t kZeroSlot = DT == VC_F16 ? kF16ZeroBin : (uint32_t)kHistBins;
  if (wave == 0) n_zero += col[64 * kZeroSlot];
  // histogram: thread t sums the columns 16 q .. 16 q + 15 of bin t / 4
  // (q = t % 4), and a quad's four sums are added by DPP (integer sums:
  // any order gives the same total)
  {
    const uint32_t bin = t >> 2;
    const p32x4 *src = (const p32x4 *)(s.hist + 64 * bin + 16 * (t & 3u));
    uint32_t h = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const p32x4 v = src[k];
      h += (v[0] + v[1]) + (v[2] + v[3]);
    }
    h += __builtin_amdgcn_update_dpp(0u, h, 0xb1, 0xf, 0xf, false);  // quad_perm 1,0,3,2
    h += __builtin_amdgcn_update_dpp(0u, h, 0x4e, 0xf, 0xf, false);  // quad_perm 2,3,0,1
    if ((t & 3u) == 0) rec->hist[bin] = DT == VC_F16 && bin == kF16ZeroBin ? 0u : h;
  }
  __syncthreads();  // the columns are dead from here: the partials reuse them
  s.n[0][t] = n_nan;
  s.n[1][t] = n_inf;
  s.n[2][t] = n_zero;
  s.n[3][t] = n_fin;
  s.d[0][t] = sm;
  s.d[1][t] = sq;
  s.d[2][t] = sa;
  s.v[0][t] = mn;
  s.o[0][t] = imn;
  s.v[1][t] = mx;
  s.o[1][t] = imx;
  chunk_reduce(s, c0, rec);
}

__global__ __launch_bounds__(kPThreads) void probe_kernel(const ProbeParams P) {
  __shared__ ChunkLds s;
  const uint64_t chunk = blockIdx.x;
  if (threadIdx.x < 64) {
    const uint32_t ti = find_first(P.chunk_first, (uint32_t)P.n_tensors, chunk);
    if (threadIdx.x == 0) s.tensor = ti;
  }
  __syncthreads();
  const ProbeTensor T = P.tensors[__builtin_amdgcn_readfirstlane(s.tensor)];
  const uint64_t CH = 4ull * P.unit;
  const uint64_t c0 = (chunk - T.chunk_begin) * CH;
  const uint64_t c1 = min(c0 + CH, T.numel);
  ProbeRec *const rec = P.recs + chunk;
  switch (T.dtype) {
    case VC_F32: probe_chunk<VC_F32>(s, T, c0, max(c0, c1), P.unit, rec); break;
    case VC_F16: probe_chunk<VC_F16>(s, T, c0, max(c0, c1), P.unit, rec); break;
    default: probe_chunk<VC_BF16>(s, T, c0, max(c0, c1), P.unit, rec); break;
  }
}

// Sum of one 32-bit field over records part, part + 4, ... below n, with the
// loads of eight records issued before their additions (integer sums: any
// order gives the same total).
template <typename Rec, typename F>
__device__ __forceinline__ uint64_t strided_sum(const Rec *recs, uint32_t part, uint32_t n, F field) {
  uint64_t h = 0;
  uint32_t i = part;
  for (; i + 28 < n; i += 32) {
    uint32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = field(recs[i + 4 * u]);
#pragma unroll
    for (int u = 0; u < 8; ++u) h += v[u];
  }
  for (; i < n; i += 4) h += field(recs[i]);
  return h;
}

// Merges records recs[0 .. n) (n <= 256) in a fixed order; thread 0 gets the
// totals in r, threads 0..63 the histogram bins in hist.
__device__ void merge_recs(ProbeLds &s, const ProbeRec *recs, uint32_t n, ProbeRec &r,
                           uint64_t &hist) {
  const uint32_t t = threadIdx.x;
  const bool has = t < n;
  const ProbeRec *const x = recs + (has ? t : 0);
  s.c[0][t] = has ? x->nan : 0;
  s.c[1][t] = has ? x->inf : 0;
  s.c[2][t] = has ? x->zero : 0;
  s.c[3][t] = has ? x->fin : 0;
  s.d[0][t] = has ? x->sum : 0.0;
  s.d[1][t] = has ? x->sum_sq : 0.0;
  s.d[2][t] = has ? x->sum_abs : 0.0;
  s.mv[0][t] = has ? x->min : 0.0;
  s.mi[0][t] = has ? x->argmin : -1;
  s.mv[1][t] = has ? x->max : 0.0;
  s.mi[1][t] = has ? x->argmax : -1;
  block_reduce(s, r);
  // histogram: thread t sums bin t % 64 over records t / 64, t / 64 + 4, ...
  const uint32_t bin = t & 63u, part = t >> 6;
  const uint64_t h = strided_sum(recs, part, n, [&](const ProbeRec &x) { return x.hist[bin]; });
  __syncthreads();
  s.c[0][t] = h;
  __syncthreads();
  hist = t < 64 ? s.c[0][t] + s.c[0][t + 64] + s.c[0][t + 128] + s.c[0][t + 192] : 0;
}

__device__ void write_out(vc_tstats *o, const ProbeTensor &T, const ProbeRec &r, uint64_t h) {
  const uint32_t t = threadIdx.x;
  if (t < (uint32_t)kHistBins) o->hist[t] = h;
  if (t == 0) {
    o->numel = T.numel;
    o->nan = r.nan;
    o->inf = r.inf;
    o->zero = r.zero;
    o->n_finite = r.fin;
    o->min = r.min;
    o->max = r.max;
    o->argmin = r.argmin;
    o->argmax = r.argmax;
    o->sum = r.sum;
    o->sum_sq = r.sum_sq;
    o->sum_abs = r.sum_abs;
  }
}

// One block per group: the group's chunk records; a tensor with one group
// gets its statistics here, a larger one a group record.
__global__ __launch_bounds__(kPThreads) void probe_merge_kernel(const ProbeParams P) {
  __shared__ ProbeLds s;
  const uint64_t g = blockIdx.x;
  if (threadIdx.x < 64) {
    const uint32_t ti = find_first(P.group_first, (uint32_t)P.n_tensors, g);
    if (threadIdx.x == 0) s.tensor = ti;
  }
  __syncthreads();
  const uint32_t ti = s.tensor;
  const ProbeTensor T = P.tensors[ti];
  const uint64_t gl = g - P.group_first[ti];
  const uint64_t first = T.chunk_begin + gl * kProbeGroupChunks;
  const uint32_t n = (uint32_t)min((uint64_t)kProbeGroupChunks,
                                   T.chunk_begin + T.n_chunks - first);
  ProbeRec r;
  uint64_t h;
  merge_recs(s, P.recs + first, n, r, h);
  if (T.n_chunks <= kProbeGroupChunks) {
    write_out(P.out + ti, T, r, h);
    return;
  }
  ProbeRec *const gr = P.grecs + g;
  if (threadIdx.x < (uint32_t)kHistBins) gr->hist[threadIdx.x] = (uint32_t)h;
  if (threadIdx.x == 0) {
    gr->nan = r.nan;
    gr->inf = r.inf;
    gr->zero = r.zero;
    gr->fin = r.fin;
    gr->argmin = r.argmin;
    gr->argmax = r.argmax;
    gr->min = r.min;
    gr->max = r.max;
    gr->sum = r.sum;
    gr->sum_sq = r.sum_sq;
    gr->sum_abs = r.sum_abs;
    gr->pad[0] = 0;
  }
}

// One block per tensor: the group records of a tensor with several groups.
__global__ __launch_bounds__(kPThreads) void probe_final_kernel(const ProbeParams P) {
  __shared__ ProbeLds s;
  const uint32_t ti = blockIdx.x;
  const ProbeTensor T = P.tensors[ti];
  if (T.n_chunks <= kProbeGroupChunks) return;
  const uint32_t n_groups = (T.n_chunks + kProbeGroupChunks - 1) / kProbeGroupChunks;
  ProbeRec r;
  uint64_t h;
  merge_recs(s, P.grecs + P.group_first[ti], n_groups, r, h);
  write_out(P.out + ti, T, r, h);
}

// ---------------------------------------------------------------- near-pass
//
// Per case: finite pairs, failures, zero-tolerance violations, the largest
// violation ratio d / t with its first index, and histograms of the ratio's
// binary exponent (failures) and of the distance on the binary16 / bfloat16
// grid. Same decomposition as the probe: one block per chunk, each wave one
// contiguous quarter; chunk records merged per group of 256, then per case.
// The largest ratio is tracked per lane under a wave-uniform threshold (the
// wave's best so far): an element becomes a candidate only when its exact
// ratio beats the threshold (fma(-T, t, d) > 0, whose sign is exact), so the
// binary64 division runs for candidates and failing elements only.

// Histogram slots: the ratio bins, then the grid-distance bins.
constexpr int kNpSlots = kRatioBins + kUlpBins;

// LDS of the near-pass streaming kernel: the histogram columns while
// streaming (as the probe's: 32-bit counters, slot-major, one column per
// lane position that the block's waves share), the per-thread partials of
// the chunk afterwards (32-bit counts and offsets from the chunk's first
// element).
struct alignas(16) NpChunkLds {
  union {
    uint32_t hist[kNpSlots * 64];
    struct {
      uint32_t c[3][kPThreads];
      double mv[kPThreads];
      uint32_t mo[kPThreads];
      uint32_t mu[kPThreads];
    };
  };
  uint32_t item;
};

// LDS of the near-pass merge launches.
struct NpLds {
  // per-thread partials
  uint64_t c[3][kPThreads];
  double mv[kPThreads];
  int64_t mi[kPThreads];
  uint32_t mu[kPThreads];
  // per-wave totals of np_reduce
  uint64_t wc[3][kPWaves];
  double wv[kPWaves];
  int64_t wi[kPWaves];
  uint32_t wu[kPWaves];
  uint32_t item;
};

__device__ __forceinline__ void np_pick(double &v, int64_t &i, double v2, int64_t i2) {
  if (i2 < 0) return;
  if (i < 0 || v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

// Fixed-order reduction of the partials in s (each thread's own slots) into
// r (valid in thread 0): DPP wave reductions, then the four waves in order.
__device__ void np_reduce(NpLds &s, NpRec &r) {
  const uint32_t t = threadIdx.x, lane = t & 63u, wave = t >> 6;
  uint64_t c[3];
#pragma unroll
  for (int f = 0; f < 3; ++f) c[f] = wave_sum_u64(s.c[f][t]);
  double v = s.mv[t];
  int64_t i = s.mi[t];
  wave_pick<true>(v, i);
  const uint32_t u = (uint32_t)wave_reduce64(s.mu[t], 0ull,
                                             [](uint64_t a, uint64_t b) { return a > b ? a : b; });
  if (lane == 0) {
#pragma unroll
    for (int f = 0; f < 3; ++f) s.wc[f][wave] = c[f];
    s.wv[wave] = v;
    s.wi[wave] = i;
    s.wu[wave] = u;
  }
  __syncthreads();
  if (t == 0) {
    uint64_t cc[3] = {0, 0, 0};
    double mv = 0.0;
    int64_t mi = -1;
    uint32_t mu = 0;
    for (int w = 0; w < kPWaves; ++w) {
#pragma unroll
      for (int f = 0; f < 3; ++f) cc[f] += s.wc[f][w];
      np_pick(mv, mi, s.wv[w], s.wi[w]);
      mu = max(mu, s.wu[w]);
    }
    r.n_pairs = cc[0];
    r.n_fail = cc[1];
    r.n_zero_tol = cc[2];
    r.argmax_ratio = mi;
    r.max_ratio = mi < 0 ? 0.0 : mv;
    r.max_ulp_fail = mu;
  }
}

// Fixed-order tree reduction of the per-thread partials of the chunk that
// starts at element c0 into its record, written by thread 0 (as the probe's
// chunk_reduce): the largest ratio keeps the smaller offset among equal
// values.
__device__ void np_chunk_reduce(NpChunkLds &s, uint64_t c0, NpRec *rec) {
  const uint32_t t = threadIdx.x;
  for (uint32_t w = kPThreads / 2; w >= 1; w >>= 1) {
    __syncthreads();
    if (t < w) {
#pragma unroll
      for (int f = 0; f < 3; ++f) s.c[f][t] += s.c[f][t + w];
      const uint32_t o2 = s.mo[t + w];
      if (o2 != kNoOff) {
        const double v = s.mv[t], v2 = s.mv[t + w];
        const uint32_t o = s.mo[t];
        if (o == kNoOff || v2 > v || (v2 == v && o2 < o)) {
          s.mv[t] = v2;
          s.mo[t] = o2;
        }
      }
      s.mu[t] = max(s.mu[t], s.mu[t + w]);
    }
  }
  __syncthreads();
  if (t == 0) {
    rec->n_pairs = s.c[0][0];
    rec->n_fail = s.c[1][0];
    rec->n_zero_tol = s.c[2][0];
    rec->argmax_ratio = s.mo[0] == kNoOff ? -1 : (int64_t)(c0 + s.mo[0]);
    rec->max_ratio = s.mo[0] == kNoOff ? 0.0 : s.mv[0];
    rec->max_ulp_fail = s.mu[0];
    rec->pad0 = 0;
  }
}

// Largest binary32 value <= x, for x >= 0 (FLT_MAX beyond the range).
__device__ __forceinline__ float np_f32_below(double x) {
  if (x >= 3.4028234663852886e38) return 3.40282347e38f;
  float f = (float)x;
  if ((double)f > x) f = __uint_as_float(__float_as_uint(f) - 1u);
  return f;
}

// Grid pattern of element j: binary16 rounding of a binary32 value, the
// stored pattern for 16-bit storage.
template <int DT>
__device__ __forceinline__ uint32_t grid_bits(const p32x4 &q, int j) {
  if constexpr (DT == VC_F32) {
    const _Float16 h = (_Float16)__uint_as_float(q[j]);  // nearest, ties to even
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
  } else {
    const uint32_t w = q[j >> 1];
    return (j & 1) ? (w >> 16) : (w & 0xffffu);
  }
}

// Grid distances of the two 16-bit patterns of a word pair, per 16-bit half:
// the patterns become ordered keys (0x8000 + m for +m, 0x8000 - m for -m:
// both zeros map to 0x8000; a finite binary16 or bfloat16 magnitude is at
// most 0x7f7f, so a key fits 16 bits), and the distance is the larger key
// minus the smaller (packed 16-bit operations).
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
typedef int16_t i16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t grid_key2(uint32_t w) {
  const uint32_t sg = __builtin_bit_cast(uint32_t, __builtin_bit_cast(i16x2, w) >> (int16_t)15);
  const u16x2 x = __builtin_bit_cast(u16x2, w ^ (sg | 0x80008000u));
  return __builtin_bit_cast(uint32_t, x - __builtin_bit_cast(u16x2, sg));
}
__device__ __forceinline__ uint32_t grid_dist2(uint32_t c, uint32_t r) {
  const u16x2 x = __builtin_bit_cast(u16x2, grid_key2(c)), y = __builtin_bit_cast(u16x2, grid_key2(r));
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(x, y) - __builtin_elementwise_min(x, y));
}

template <int DT>
__device__ void np_chunk(NpChunkLds &s, const NpCase &C, uint64_t c0, uint64_t c1, uint32_t U,
                         double atol, double rtol, NpRec *rec) {
  constexpr int V = DT == VC_F32 ? 4 : 8;
  constexpr int ES = DT == VC_F32 ? 4 : 2;
  constexpr uint32_t ITER = 64 * V;
  constexpr uint32_t kExpMask = DT == VC_BF16 ? 0x7f80u : 0x7c00u;
  const uint32_t t = threadIdx.x, lane = t & 63u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(t >> 6);
  for (uint32_t w = t; w < (uint32_t)(kNpSlots * 64); w += kPThreads) s.hist[w] = 0;
  __syncthreads();
  // lane's column; col[64 * b] is its counter of slot b
  uint32_t *const col = s.hist + lane;
  const uint64_t w0 = min(c0 + (uint64_t)wave * U, c1), w1 = min(w0 + U, c1);
  const uint32_t ow1 = (uint32_t)(w1 - c0);
  const bool vec = ((uintptr_t)C.cand % 16) == 0 && ((uintptr_t)C.ref % 16) == 0;
  uint32_t n_pairs = 0, n_fail = 0, n_zt = 0, mu = 0;
  uint32_t n_usual = 0;  // usual steps (uniform): V finite pairs per lane each
  double lb = -1.0, T = -1.0;  // lane best ratio, wave threshold (-1: none)
  // Binary32 screen of the usual step. alo, rlo: the pair lowered by 2^-20
  // and rounded down, so fma(|r|, rlo, alo) <= atol + rtol |r| = t despite
  // its rounding; tm = min(1, T lowered by 2^-20 and rounded down), so the
  // rounded product tm * that <= min(1, T) * t. |c - r| in binary32 is
  // within a relative 2^-23 of the exact difference (exact for 16-bit
  // storage unless the exponents lie far apart; gradual underflow keeps a
  // subnormal difference of binary32 values exact or within that bound), so
  // |c - r|32 * (1 + 2^-21) <= tm * fma(|r|, rlo, alo) proves d <= t and
  // d <= T t: the pair neither fails nor beats the largest ratio. A NaN or
  // an infinity in either value makes the test fail (the comparison with 0
  // of a NaN is false; an infinite difference exceeds a finite bound, and an
  // infinite bound comes with an infinite difference: inf - inf is NaN), so
  // a step that passes it holds finite pairs only.
  const float alo = np_f32_below(atol - atol * 0x1p-20);
  const float rlo = np_f32_below(rtol - rtol * 0x1p-20);
  constexpr float kDUp = 1.0f + 0x1p-21f;
  float tm = 0.0f;
  // Binary16 storage screens with the difference taken in binary16 (packed:
  // it is within a relative 2^-11 of c - r, exact when small, and a NaN or an
  // infinity when either value is one or the difference leaves the range)
  // and min(1, T) folded into the lowered pair: am = m atol and rm = m rtol,
  // m = min(1, T), each lowered by 2^-20 and rounded down, so
  // fma(|r|, rm, am) < m t; then |c - r|16 * (1 + 2^-10) <= fma(|r|, rm, am)
  // proves |c - r| < m t. (A binary16 difference that is not zero is at
  // least 2^-24, so a bound that rounds in the subnormal range cannot pass a
  // non-zero difference.)
  constexpr float kDUp16 = 1.0f + 0x1p-10f;
  float am = 0.0f, rm = 0.0f;
  uint32_t li = kNoOff;
  // Usual step (T >= 0, every pair passes the screen): it only counts its
  // pairs and their grid distances, with no exit.
  // (the step's largest test value, by the NaN-propagating maximum, so one
  // comparison decides; c - r as an fma with 1, which takes 16-bit operands
  // as they are)
  auto is_usual = [&](const p32x4 &cq, const p32x4 &rq) {
    float m = -__builtin_inff();
    if constexpr (DT == VC_F16) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t cw = cq[w], rw = rq[w];
        const ph2 ch = __builtin_bit_cast(ph2, cw), rh = __builtin_bit_cast(ph2, rw);
        const ph2 dh = ch - rh;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const float tl = __builtin_fmaf(__builtin_fabsf((float)rh[h]), rm, am);
          m = __builtin_elementwise_maximum(
              m, __builtin_fmaf(__builtin_fabsf((float)dh[h]), kDUp16, -tl));
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const float rf = pdec<DT>(rq, j);
        const float d = __builtin_fabsf(pdec<DT>(cq, j) - rf);
        const float tl = __builtin_fmaf(__builtin_fabsf(rf), rlo, alo);
        m = __builtin_elementwise_maximum(m, __builtin_fmaf(d, kDUp, -(tm * tl)));
      }
    }
    return __ballot(!(m <= 0.0f)) == 0;
  };
  // Grid-distance bin of a usual pair, slot kRatioBins + bit length of the
  // distance (0 for equal patterns): for 16-bit storage the distances of a
  // word's two pairs come packed, and a half's bit length is 16 minus the
  // leading zeros of the half placed above a set bit 15.
  uint32_t *const col_u = col + 64 * (kRatioBins + 16);
  auto usual_step = [&](const p32x4 &cq, const p32x4 &rq) {
    ++n_usual;
    if constexpr (DT != VC_F32) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t d = grid_dist2(cq[w], rq[w]);
        atomicAdd(col_u - 64 * __builtin_clz((d << 16) | 0x8000u), 1u);
        atomicAdd(col_u - 64 * __builtin_clz(d | 0x8000u), 1u);
      }
    } else {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const uint32_t hc = grid_bits<DT>(cq, j), hr = grid_bits<DT>(rq, j);
        const uint32_t dist = ((hc ^ hr) & 0x8000u) ? (hc & 0x7fffu) + (hr & 0x7fffu)
                                                    : (uint32_t)abs((int)hc - (int)hr);
        // binary32 values beyond the binary16 range sit outside the grid
        const int ubin = ((hc & kExpMask) == kExpMask || (hr & kExpMask) == kExpMask)
                             ? kRatioBins + kUlpBins - 1
                             : kRatioBins + 31 - __builtin_clz(2u * dist + 1u);
        atomicAdd(col + 64 * ubin, 1u);
      }
    }
  };
  // Any other step, pair by pair in binary64 (pairs from w1 on are skipped).
  auto elem_step = [&](const p32x4 &cq, const p32x4 &rq, uint32_t o0) {
    bool cand_any = false;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const float cf = pdec<DT>(cq, j), rf = pdec<DT>(rq, j);
      const bool fin = o0 + (uint32_t)j < ow1 && __builtin_fabsf(cf) <= 3.40282347e38f &&
                       __builtin_fabsf(rf) <= 3.40282347e38f;
      if (!fin) continue;
      ++n_pairs;
      const double r = (double)rf;
      const double d = __builtin_fabs((double)cf - r);
      const double tt = atol + rtol * __builtin_fabs(r);
      const bool fail = d > tt;
      n_fail += fail ? 1u : 0u;
      if (tt == 0.0) {
        n_zt += d > 0.0 ? 1u : 0u;
      } else if (fail || T < 0.0 || __builtin_fma(-T, tt, d) > 0.0) {
        const double qr = d / tt;
        if (qr > lb || li == kNoOff) {
          lb = qr;
          li = o0 + (uint32_t)j;
          cand_any = true;
        }
        if (fail) {
          const int e = (int)((__double_as_longlong(qr) >> 52) & 0x7ff) - 1023;  // qr >= 1
          atomicAdd(col + 64 * min(e, kRatioBins - 1), 1u);
        }
      }
      const uint32_t hc = grid_bits<DT>(cq, j), hr = grid_bits<DT>(rq, j);
      const bool inside = (hc & kExpMask) != kExpMask && (hr & kExpMask) != kExpMask;
      const int kc = (hc & 0x8000u) ? -(int)(hc & 0x7fffu) : (int)(hc & 0x7fffu);
      const int kr = (hr & 0x8000u) ? -(int)(hr & 0x7fffu) : (int)(hr & 0x7fffu);
      const uint32_t dist = (uint32_t)abs(kc - kr);
      const int ub = inside ? (dist == 0 ? 0 : 32 - __builtin_clz(dist)) : kUlpBins - 1;
      atomicAdd(col + 64 * (kRatioBins + ub), 1u);
      if (fail) mu = max(mu, inside ? dist : 0xffffffffu);
    }
    if (__ballot(cand_any) != 0) {  // raise the wave threshold
      T = wave_max_d(li == kNoOff ? -1.0 : lb);
      tm = T >= 1.0 ? 1.0f : np_f32_below(T - T * 0x1p-20);
      const double mt = T >= 1.0 ? 1.0 : T;
      am = np_f32_below(mt * atol - mt * atol * 0x1p-20);
      rm = np_f32_below(mt * rtol - mt * rtol * 0x1p-20);
    }
  };
  // The full steps through buffer resources over the wave's range (as the
  // probe's), each step's loads issued one step ahead; runs of usual steps
  // take an inner loop of their own.
  const uint32_t nst = vec ? (uint32_t)((w1 - w0) / ITER) : 0u;
  if (nst > 0) {
    constexpr uint32_t SB = ITER * ES;  // bytes per step and tensor
    const uint32_t last = (nst - 1) * SB;
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(C.cand + w0 * ES), (short)0, (int)(nst * SB), kBufferWord3);
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(C.ref + w0 * ES), (short)0, (int)(nst * SB), kBufferWord3);
    const uint32_t loff = lane * 16u;
    const uint32_t ol = (uint32_t)(w0 - c0) + lane * (uint32_t)V;
    uint32_t k = 0;
    p32x4 cn = bload16(rc, loff, 0u), rn = bload16(rr, loff, 0u);
    while (true) {
      p32x4 cq = cn, rq = rn;
      cn = bload16(rc, loff, min(k + SB, last));
      rn = bload16(rr, loff, min(k + SB, last));
      bool usual = T >= 0.0 && is_usual(cq, rq);
      while (usual) {
        usual_step(cq, rq);
        k += SB;
        if (k > last) break;
        cq = cn;
        rq = rn;
        cn = bload16(rc, loff, min(k + SB, last));
        rn = bload16(rr, loff, min(k + SB, last));
        usual = is_usual(cq, rq);
      }
      if (usual) break;  // (past the last step)
      elem_step(cq, rq, ol + k / ES);
      k += SB;
      if (k > last) break;
    }
  }
  for (uint64_t b = w0 + (uint64_t)nst * ITER; b < w1; b += ITER) {
    const uint64_t i0 = b + (uint64_t)lane * V;
    const p32x4 cq = pload_guarded<DT>(C.cand, i0, w1);
    const p32x4 rq = pload_guarded<DT>(C.ref, i0, w1);
    elem_step(cq, rq, (uint32_t)(i0 - c0));
  }
  n_pairs += V * n_usual;
  // histograms: thread t < 200 sums the columns 16 q .. 16 q + 15 of slot
  // t / 4 (q = t % 4), and a quad's four sums are added by DPP
  __syncthreads();
  {
    const uint32_t slot = t >> 2;
    uint32_t h = 0;
    if (slot < (uint32_t)kNpSlots) {
      const p32x4 *src = (const p32x4 *)(s.hist + 64 * slot + 16 * (t & 3u));
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const p32x4 v = src[k];
        h += (v[0] + v[1]) + (v[2] + v[3]);
      }
    }
    h += __builtin_amdgcn_update_dpp(0u, h, 0xb1, 0xf, 0xf, false);  // quad_perm 1,0,3,2
    h += __builtin_amdgcn_update_dpp(0u, h, 0x4e, 0xf, 0xf, false);  // quad_perm 2,3,0,1
    if ((t & 3u) == 0 && slot < (uint32_t)kNpSlots) {
      if (slot < (uint32_t)kRatioBins) rec->ratio_hist[slot] = h;
      else rec->ulp_hist[slot - kRatioBins] = h;
    }
  }
  __syncthreads();  // the columns are dead from here: the partials reuse them
  s.c[0][t] = n_pairs;
  s.c[1][t] = n_fail;
  s.c[2][t] = n_zt;
  s.mv[t] = lb;
  s.mo[t] = li;
  s.mu[t] = mu;
  np_chunk_reduce(s, c0, rec);
}

__global__ __launch_bounds__(kPThreads) void nearpass_kernel(const NpParams P) {
  __shared__ NpChunkLds s;
  const uint64_t chunk = blockIdx.x;
  if (threadIdx.x < 64) {
    const uint32_t ci = find_first(P.chunk_first, (uint32_t)P.n_cases, chunk);
    if (threadIdx.x == 0) s.item = ci;
  }
  __syncthreads();
  const NpCase C = P.cases[__builtin_amdgcn_readfirstlane(s.item)];
  const uint64_t CH = 4ull * P.unit;
  const uint64_t c0 = (chunk - C.chunk_begin) * CH;
  const uint64_t c1 = max(c0, min(c0 + CH, C.numel));
  NpRec *const rec = P.recs + chunk;
  switch (C.dtype) {
    case VC_F32: np_chunk<VC_F32>(s, C, c0, c1, P.unit, P.atol, P.rtol, rec); break;
    case VC_F16: np_chunk<VC_F16>(s, C, c0, c1, P.unit, P.atol, P.rtol, rec); break;
    default: np_chunk<VC_BF16>(s, C, c0, c1, P.unit, P.atol, P.rtol, rec); break;
  }
}

// Merges records recs[0 .. n) (n <= 256) in a fixed order: totals in r
// (thread 0), histogram bin t (t < 50) in hist.
__device__ void np_merge(NpLds &s, const NpRec *recs, uint32_t n, NpRec &r, uint64_t &hist) {
  const uint32_t t = threadIdx.x;
  const bool has = t < n;
  const NpRec *const x = recs + (has ? t : 0);
  s.c[0][t] = has ? x->n_pairs : 0;
  s.c[1][t] = has ? x->n_fail : 0;
  s.c[2][t] = has ? x->n_zero_tol : 0;
  s.mv[t] = has ? x->max_ratio : 0.0;
  s.mi[t] = has ? x->argmax_ratio : -1;
  s.mu[t] = has ? x->max_ulp_fail : 0u;
  np_reduce(s, r);
  const uint32_t bin = t & 63u, part = t >> 6;
  uint64_t h = 0;
  if (bin < (uint32_t)kRatioBins)
    h = strided_sum(recs, part, n, [&](const NpRec &x) { return x.ratio_hist[bin]; });
  else if (bin < (uint32_t)(kRatioBins + kUlpBins))
    h = strided_sum(recs, part, n, [&](const NpRec &x) { return x.ulp_hist[bin - kRatioBins]; });
  __syncthreads();
  s.c[0][t] = h;
  __syncthreads();
  hist = t < 64 ? s.c[0][t] + s.c[0][t + 64] + s.c[0][t + 128] + s.c[0][t + 192] : 0;
}

__device__ void np_write(vc_nearpass *o, const NpCase &C, const NpRec &r, uint64_t h) {
  const uint32_t t = threadIdx.x;
  if (t < (uint32_t)kRatioBins) o->ratio_hist[t] = h;
  else if (t < (uint32_t)(kRatioBins + kUlpBins)) o->ulp_hist[t - kRatioBins] = h;
  if (t == 0) {
    o->numel = C.numel;
    o->n_pairs = r.n_pairs;
    o->n_fail = r.n_fail;
    o->n_zero_tol = r.n_zero_tol;
    o->max_ratio = r.max_ratio;
    o->argmax_ratio = r.argmax_ratio;
    o->max_ulp_fail = r.max_ulp_fail;
    o->reserved = 0;
  }
}

__global__ __launch_bounds__(kPThreads) void nearpass_merge_kernel(const NpParams P) {
  __shared__ NpLds s;
  const uint64_t g = blockIdx.x;
  if (threadIdx.x < 64) {
    const uint32_t ci = find_first(P.group_first, (uint32_t)P.n_cases, g);
    if (threadIdx.x == 0) s.item = ci;
  }
  __syncthreads();
  const uint32_t ci = s.item;
  const NpCase C = P.cases[ci];
  const uint64_t first = C.chunk_begin + (g - P.group_first[ci]) * kProbeGroupChunks;
  const uint32_t n = (uint32_t)min((uint64_t)kProbeGroupChunks,
                                   C.chunk_begin + C.n_chunks - first);
  NpRec r;
  uint64_t h;
  np_merge(s, P.recs + first, n, r, h);
  if (C.n_chunks <= kProbeGroupChunks) {
    np_write(P.out + ci, C, r, h);
    return;
  }
  NpRec *const gr = P.grecs + g;
  if (threadIdx.x < (uint32_t)kRatioBins) gr->ratio_hist[threadIdx.x] = (uint32_t)h;
  else if (threadIdx.x < (uint32_t)(kRatioBins + kUlpBins))
    gr->ulp_hist[threadIdx.x - kRatioBins] = (uint32_t)h;
  if (threadIdx.x == 0) {
    gr->n_pairs = r.n_pairs;
    gr->n_fail = r.n_fail;
    gr->n_zero_tol = r.n_zero_tol;
    gr->max_ratio = r.max_ratio;
    gr->argmax_ratio = r.argmax_ratio;
    gr->max_ulp_fail = r.max_ulp_fail;
    gr->pad0 = 0;
  }
}

__global__ __launch_bounds__(kPThreads) void nearpass_final_kernel(const NpParams P) {
  __shared__ NpLds s;
  const uint32_t ci = blockIdx.x;
  const NpCase C = P.cases[ci];
  if (C.n_chunks <= kProbeGroupChunks) return;
  const uint32_t n_groups = (C.n_chunks + kProbeGroupChunks - 1) / kProbeGroupChunks;
  NpRec r;
  uint64_t h;
  np_merge(s, P.grecs + P.group_first[ci], n_groups, r, h);
  np_write(P.out + ci, C, r, h);
}

// ---------------------------------------------------------------- content hash
//
// H = M(0x243F6A8885A308D3 ^ (D << 56) ^ n) + sum_i M(w_i ^ i * G) mod 2^64,
// with M the SplitMix64 finalizer (Steele, Lea and Flood, 2014) and w_i the
// i-th 64-bit little-endian word of the tensor's storage (the last one
// zero-padded). A lane's 16 bytes of a step are two words; chunk and step
// boundaries fall on 1 KiB, so no word straddles them. The sum is order-free:
// every block adds its chunk's part to the tensor's sum with one 64-bit
// integer atomic, and the block holding the tensor's first chunk adds the
// length / type term.

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

template <int DT>
__device__ uint64_t hash_chunk(const ProbeTensor &T, uint64_t c0, uint64_t c1, uint32_t U) {
  constexpr int V = DT == VC_F32 ? 4 : 8;
  constexpr int ES = DT == VC_F32 ? 4 : 2;
  constexpr uint32_t ITER = 64 * V;
  constexpr uint64_t G = 0x9E3779B97F4A7C15ull;
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint64_t w0 = min(c0 + (uint64_t)wave * U, c1), w1 = min(w0 + U, c1);
  const bool vec = ((uintptr_t)T.data % 16) == 0;
  constexpr int EW = 8 / ES;  // elements per word
  uint64_t h = 0;
  // i * G for the lane's first word (its element offset times ES / 8; w0 is
  // a multiple of 1024 elements), advanced by a constant per step
  uint64_t ig = ((w0 + (uint64_t)lane * V) / EW) * G;
  for (uint64_t b = w0; b < w1; b += ITER, ig += (uint64_t)(ITER / EW) * G) {
    const uint64_t i0 = b + (uint64_t)lane * V;
    // elements past w1 load as zero: the zero padding of the last word
    const p32x4 q = (vec && b + ITER <= w1) ? pload16(T.data + i0 * ES)
                                            : pload_guarded<DT>(T.data, i0, w1);
    if (i0 < w1) h += mix64(((uint64_t)q[1] << 32 | q[0]) ^ ig);
    if (i0 + EW < w1) h += mix64(((uint64_t)q[3] << 32 | q[2]) ^ (ig + G));
  }
  return h;
}

__global__ __launch_bounds__(kPThreads) void hash_kernel(const HashParams P) {
  __shared__ uint64_t part[kPWaves];
  __shared__ uint32_t item;
  const uint64_t chunk = blockIdx.x;
  if (threadIdx.x < 64) {
    const uint32_t ti = find_first(P.chunk_first, (uint32_t)P.n_tensors, chunk);
    if (threadIdx.x == 0) item = ti;
  }
  __syncthreads();
  const uint32_t ti = item;
  const ProbeTensor T = P.tensors[ti];
  const uint64_t CH = 4ull * P.unit;
  const uint64_t c0 = (chunk - T.chunk_begin) * CH;
  const uint64_t c1 = max(c0, min(c0 + CH, T.numel));
  uint64_t h;
  switch (T.dtype) {
    case VC_F32: h = hash_chunk<VC_F32>(T, c0, c1, P.unit); break;
    case VC_F16: h = hash_chunk<VC_F16>(T, c0, c1, P.unit); break;
    default: h = hash_chunk<VC_BF16>(T, c0, c1, P.unit); break;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) h += __shfl_xor(h, m);
  if ((threadIdx.x & 63u) == 0) part[threadIdx.x >> 6] = h;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t s = part[0] + part[1] + part[2] + part[3];
    if (chunk == T.chunk_begin)
      s += mix64(0x243F6A8885A308D3ull ^ ((uint64_t)(uint32_t)T.dtype << 56) ^ T.numel);
    atomicAdd(P.out + ti, (unsigned long long)s);
  }
}

}  // namespace

hipError_t launch_hash(const HashParams &p, uint64_t n_chunks, hipStream_t s, hipEvent_t begin,
                       hipEvent_t end) {
  hipError_t e;
  if (begin != nullptr && (e = hipEventRecord(begin, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(hash_kernel, dim3((uint32_t)n_chunks), dim3(kPThreads), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (end != nullptr && (e = hipEventRecord(end, s)) != hipSuccess) return e;
  return hipSuccess;
}

hipError_t launch_nearpass(const NpParams &p, uint64_t n_chunks, uint64_t n_groups,
                           hipStream_t s, hipEvent_t begin, hipEvent_t end) {
  hipError_t e;
  if (begin != nullptr && (e = hipEventRecord(begin, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(nearpass_kernel, dim3((uint32_t)n_chunks), dim3(kPThreads), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (end != nullptr && (e = hipEventRecord(end, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(nearpass_merge_kernel, dim3((uint32_t)n_groups), dim3(kPThreads), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // (every case owns at least one group: as many groups as cases means no
  // case has group records to merge)
  if (n_groups == (uint64_t)p.n_cases) return hipSuccess;
  hipLaunchKernelGGL(nearpass_final_kernel, dim3((uint32_t)p.n_cases), dim3(kPThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_probe(const ProbeParams &p, uint64_t n_chunks, uint64_t n_groups,
                        hipStream_t s, hipEvent_t begin, hipEvent_t end) {
  hipError_t e;
  if (begin != nullptr && (e = hipEventRecord(begin, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(probe_kernel, dim3((uint32_t)n_chunks), dim3(kPThreads), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (end != nullptr && (e = hipEventRecord(end, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(probe_merge_kernel, dim3((uint32_t)n_groups), dim3(kPThreads), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // (every tensor owns at least one group: as many groups as tensors means
  // no tensor has group records to merge)
  if (n_groups == (uint64_t)p.n_tensors) return hipSuccess;
  hipLaunchKernelGGL(probe_final_kernel, dim3((uint32_t)p.n_tensors), dim3(kPThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace vck
