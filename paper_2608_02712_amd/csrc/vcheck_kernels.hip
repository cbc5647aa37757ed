// vcheck_kernels.hip -- gfx950 kernels of the validation library.
//
// One streaming pass over (cand, ref) computes, per case, everything the
// engine-owned validation and forensics need (Sec. 3.2 Validate and the
// numerical-deviation evidence; Sec. 4.2 localization; Sec. 4.3 integrity and
// full-coverage evidence): the tolerance gate for up to 8 pairs, NaN/Inf
// counts, exact max/argmax of |c-r| and |c-r|/|r|, binary64 error sums, the
// per-tile mismatch map, the ordered first-k mismatch indices and the
// degenerate-output detector counts. Each block of the main kernel writes
// one chunk record; separate launches then merge the records in a fixed
// order: a finalize kernel per group of up to 256 chunks (writing the case's
// results directly when the case has one group) and a second one for cases
// with several groups. Kernel boundaries order the launches, so the streaming
// kernel needs no device-scope fences; the block that writes the last case's
// results also writes the suite match rates, after one acquire-release
// increment of a completion count per case.
//
// Work decomposition: a case is cut into chunks of 4 * U elements; one block
// (4 waves) owns one chunk and streams it front to back: a step is 64 lanes x
// 16 bytes (one fully coalesced 1 KiB non-temporal load per tensor) and the
// four waves take steps round robin, so the block's loads always target one
// contiguous stretch of memory. Loads run two steps ahead of the evaluation.
//
// Exactness. The definition is binary64 on exactly decoded values. Each step
// is evaluated by the cheapest of three tiers that is exact for it:
//  1. binary32 tier. When every element of the step has |c - r| <= 0.998 |r|
//     (binary16/bfloat16 storage) or <= 0.49 |r| (binary32 storage), the
//     binary32 difference c - r is exact (the exponents of c and r differ by
//     at most 10; for binary32 by Sterbenz's lemma; binary16 values are
//     multiples of 2^-24, so their difference is also exact whenever it is
//     below 1), so |c - r| equals its binary64 value. The gate then compares it with binary64 thresholds
//     (several pairs) or, for a single pair, with binary32 bounds
//     fma(|r|, rlo, alo) <= atol + rtol |r| <= fma(|r|, rhi, ahi) (the host
//     shrinks / grows the pair by 2^-20 and only enables this when the
//     thresholds stay in the normal binary32 range); an element between the
//     bounds sends the step to tier 2. The running-maximum test of |c - r| is
//     an exact binary32 comparison against the threshold rounded down to
//     binary32; the quotient's test compares the binary32 estimate with the
//     threshold lowered by 2^-20 (more than the estimate's error), so it
//     never misses a larger quotient, and the update decides exactly.
//  2. binary64 tier: the same evaluation in binary64 for steps with finite
//     values and non-zero references.
//  3. exact tier: element by element with the class tests (NaN, Inf, r = 0,
//     partial tail steps).
// Each lane keeps its exact best (value, offset) of |c - r| and of the
// quotient; a wave-uniform threshold (the wave's best so far) filters
// elements, so only an element that strictly beats it reaches the update
// (ties never do, since later elements have larger indices). Only sum_rel
// uses quotient estimates (binary32 or binary64 reciprocals, relative error
// below 5e-7, within the 1e-6 contract). Counts come from wave ballots and
// popcounts; no floating-point atomics are used, so every result is
// bit-reproducible.
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

constexpr uint32_t kNone = 0xffffffffu;
constexpr int kDeferCap = 32;  // deferred steps listed per wave before they are evaluated
// a list entry keeps its list position and wave in bits 1..7 of the step's
// chunk offset (a multiple of 256)
static_assert(kDeferCap <= 32, "list entry layout");
// s_waitcnt immediates (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt in
// 6:4, lgkmcnt in 11:8): wait until at most 2 (or 0) vector memory
// operations are outstanding, other counters unconstrained
constexpr int kWaitVm2 = 0x0f72;
constexpr int kWaitVm0 = 0x0f70;
// outcome of a fast tier for one step
constexpr int kDone = 0;      // evaluated and committed
constexpr int kDefer = 1;     // to the exact tier, after streaming
constexpr int kNotTaken = 2;  // not this tier (nothing changed)
constexpr int kLocate = 3;    // committed; mismatch positions are recorded after streaming
constexpr int kUsual = 4;     // committed by the usual step: nothing else to record

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

// Tile geometry of one chunk, for the localization path. The chunk's first
// element is at row row0 = trow0 * tile_h + rrem0 and column col0 of the
// (rows, cols) view.
struct ChunkTiles {
  uint64_t tiles_c;    // tiles per tile row
  uint64_t trow0;      // tile row of row0
  uint64_t tcol0;      // col0 / tile_w (rows of 2^31 or more elements)
  uint64_t room;       // cols - col0: elements from the chunk start to the row end
  uint64_t tile_off;   // offset of the case's map in the tile-map output
  uint64_t win_base;   // first tile of the block's LDS window
  uint32_t *tile_maps;
  uint32_t col0;       // (rows shorter than 2^31 elements)
  uint32_t cols32;
  uint32_t rrem0;
  uint32_t crem0;      // col0 % tile_w (rows of 2^31 or more elements)
  DivMagic cdiv, hdiv, wdiv;
  uint32_t win_len, kq, do_tiles, wide;
};

// Tile (row-major index within the case's map) of the element at chunk
// offset o, with 32-bit divisions by the invariant divisors only (a chunk
// holds fewer than 2^18 elements).
__device__ __forceinline__ uint64_t tile_at(const ChunkTiles &g, uint32_t o, uint32_t &dr) {
  uint64_t tc;  // tile column (dr: rows past row0)
  if (!g.wide) {
    const uint32_t x = g.col0 + o;
    dr = div_by(x, g.cdiv.m, g.cdiv.shifts);
    tc = div_by(x - dr * g.cols32, g.wdiv.m, g.wdiv.shifts);
  } else {
    // rows of 2^31 elements or more: the chunk spans at most two rows
    dr = (uint64_t)o >= g.room ? 1u : 0u;
    tc = dr ? (uint64_t)div_by(o - (uint32_t)g.room, g.wdiv.m, g.wdiv.shifts)
            : g.tcol0 + div_by(g.crem0 + o, g.wdiv.m, g.wdiv.shifts);
  }
  return (g.trow0 + div_by(g.rrem0 + dr, g.hdiv.m, g.hdiv.shifts)) * g.tiles_c + tc;
}

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
  d.group_begin = t->group_begin;
  d.n_chunks = t->n_chunks;
  d.n_groups = t->n_groups;
  d.status = t->status;
  d.inp_mask = t->inp_mask;
  d.vec_ok = t->vec_ok;
  d.orig = t->orig;
  d.dtype = t->dtype;
  d.unit_elems = t->unit_elems;
  d.cols_div.m = t->cols_div.m;
  d.cols_div.shifts = t->cols_div.shifts;
  d.n_tiles = t->n_tiles;
  return d;
}

template <typename I>
__device__ __forceinline__ void max_merge(double &v, I &i, double ov, I oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}


__device__ __forceinline__ double readlane_f64(double x, uint32_t l) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)b, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(b >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// One step of a wave maximum: v and the value CTRL moves in (DPP; lanes with
// no source, or outside the rows ROWS enables, see -1).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_max(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)b, CTRL, ROWS, 0xf, false);
  const uint32_t hi =
      __builtin_amdgcn_update_dpp(0xbff00000u, (uint32_t)(b >> 32), CTRL, ROWS, 0xf, false);
  return __builtin_fmax(v, __longlong_as_double((long long)(((uint64_t)hi << 32) | lo)));
}

// Wave-wide maximum of v (values -1 or >= 0), wave-uniform: row shifts by
// 1, 2, 3, 4 and 8 leave each row's maximum in its last lane, two row
// broadcasts carry them to lane 63.
__device__ __forceinline__ double wave_max_val(double v) {
  v = dpp_max<0x111, 0xf>(v);  // row_shr:1
  v = dpp_max<0x112, 0xf>(v);  // row_shr:2
  v = dpp_max<0x113, 0xf>(v);  // row_shr:3
  v = dpp_max<0x114, 0xf>(v);  // row_shr:4
  v = dpp_max<0x118, 0xf>(v);  // row_shr:8
  v = dpp_max<0x142, 0xa>(v);  // row_bcast:15
  v = dpp_max<0x143, 0xc>(v);  // row_bcast:31
  return readlane_f64(v, kWaveSize - 1);
}

// One step of a wave sum: v plus the value CTRL moves in (lanes with no
// source, or outside the rows ROWS enables, add 0).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_add(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)b, CTRL, ROWS, 0xf, false);
  const uint32_t hi = __builtin_amdgcn_update_dpp(0u, (uint32_t)(b >> 32), CTRL, ROWS, 0xf, false);
  return v + __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Wave-wide sum of v, wave-uniform, in a fixed order: row shifts by 1, 2, 4
// and 8 leave each row's sum in its last lane, two row broadcasts add them
// up in lane 63.
__device__ __forceinline__ double wave_sum(double v) {
  v = dpp_add<0x111, 0xf>(v);  // row_shr:1
  v = dpp_add<0x112, 0xf>(v);  // row_shr:2
  v = dpp_add<0x114, 0xf>(v);  // row_shr:4
  v = dpp_add<0x118, 0xf>(v);  // row_shr:8
  v = dpp_add<0x142, 0xa>(v);  // row_bcast:15
  v = dpp_add<0x143, 0xc>(v);  // row_bcast:31
  return readlane_f64(v, kWaveSize - 1);
}

// Wave-wide minimum of i, wave-uniform (the pattern of wave_max_val).
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t i) {
  i = min(i, (uint32_t)__builtin_amdgcn_update_dpp(0xffffffffu, i, 0x111, 0xf, 0xf, false));
  i = min(i, (uint32_t)__builtin_amdgcn_update_dpp(0xffffffffu, i, 0x112, 0xf, 0xf, false));
  i = min(i, (uint32_t)__builtin_amdgcn_update_dpp(0xffffffffu, i, 0x113, 0xf, 0xf, false));
  i = min(i, (uint32_t)__builtin_amdgcn_update_dpp(0xffffffffu, i, 0x114, 0xf, 0xf, false));
  i = min(i, (uint32_t)__builtin_amdgcn_update_dpp(0xffffffffu, i, 0x118, 0xf, 0xf, false));
  i = min(i, (uint32_t)__builtin_amdgcn_update_dpp(0xffffffffu, i, 0x142, 0xa, 0xf, false));
  i = min(i, (uint32_t)__builtin_amdgcn_update_dpp(0xffffffffu, i, 0x143, 0xc, 0xf, false));
  return __builtin_amdgcn_readlane(i, kWaveSize - 1);
}

// Wave-wide (largest value, smallest index among the lanes holding it), as
// wave_max, through DPP: the maximum first, then the smallest index of the
// lanes that hold it.
__device__ __forceinline__ void wave_max_dpp(double &v, uint32_t &i) {
  const double m = wave_max_val(v);
  i = wave_min_u32(v == m ? i : kNone);
  v = m;
}

// c - r of element j of a step in binary32 (one rounding); binary16 pairs go
// through the mixed-precision FMA, which converts both operands exactly.
template <int DT>
__device__ __forceinline__ float diff32(const u32x4 &cq, const u32x4 &rq, int j) {
  if constexpr (DT == VC_F16) {
    const int w = j >> 1;
    const uint32_t cw = w == 0 ? cq[0] : w == 1 ? cq[1] : w == 2 ? cq[2] : cq[3];
    const uint32_t rw = w == 0 ? rq[0] : w == 1 ? rq[1] : w == 2 ? rq[2] : rq[3];
    float d;
    if (j & 1)
      asm("v_fma_mix_f32 %0, %1, 1.0, -%2 op_sel:[1,0,1] op_sel_hi:[1,0,1]" : "=v"(d) : "v"(cw), "v"(rw));
    else
      asm("v_fma_mix_f32 %0, %1, 1.0, -%2 op_sel_hi:[1,0,1]" : "=v"(d) : "v"(cw), "v"(rw));
    return d;
  } else {
    return dec32<DT>(elem<DT>(cq, j)) - dec32<DT>(elem<DT>(rq, j));
  }
}

// Binary16 operands of the mixed-precision FMA: the half SEL (0 low, 1 high)
// of a storage word enters v_fma_mix_f32 as an exactly converted binary32
// value, so these take no separate conversion.
// fma(|r|, |x|, y) with r the binary16 half SEL of rw.
template <int SEL>
__device__ __forceinline__ float h_fma_rx(uint32_t rw, float x, float y) {
  float g;
  if constexpr (SEL)
    asm("v_fma_mix_f32 %0, |%1|, |%2|, %3 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
        : "=v"(g) : "v"(rw), "v"(x), "v"(y));
  else
    asm("v_fma_mix_f32 %0, |%1|, |%2|, %3 op_sel_hi:[1,0,0]" : "=v"(g) : "v"(rw), "v"(x), "v"(y));
  return g;
}
// |r| * |x| with r the binary16 half SEL of rw.
template <int SEL>
__device__ __forceinline__ float h_mul_rx(uint32_t rw, float x) {
  float g;
  if constexpr (SEL)
    asm("v_fma_mix_f32 %0, |%1|, |%2|, 0 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
        : "=v"(g) : "v"(rw), "v"(x));
  else
    asm("v_fma_mix_f32 %0, |%1|, |%2|, 0 op_sel_hi:[1,0,0]" : "=v"(g) : "v"(rw), "v"(x));
  return g;
}
// |r_lo| * |r_hi| of the two binary16 halves of rw (exact: 22 significant bits).
__device__ __forceinline__ float h_prod(uint32_t rw) {
  float g;
  asm("v_fma_mix_f32 %0, |%1|, |%1|, 0 op_sel:[0,1,0] op_sel_hi:[1,1,0]" : "=v"(g) : "v"(rw));
  return g;
}

// Largest binary32 value <= x, for x = -1 or x >= 0 (the running-maximum
// thresholds); values above the binary32 range give FLT_MAX.
__device__ __forceinline__ float f32_down(double x) {
  if (x < 0.0) return -1.0f;
  float f = (float)x;
  if ((double)f > x) f = __uint_as_float(__float_as_uint(f) - 1u);
  return f;
}

// Smallest binary32 value > x, for finite x (x = -1 or x >= 0 here).
__device__ __forceinline__ float f32_next_up(float x) {
  const uint32_t b = __float_as_uint(x);
  return x >= 0.0f ? __uint_as_float((b & 0x7fffffffu) + 1u) : __uint_as_float(b - 1u);
}

// ------------------------------------------------------------ merge helpers

// The finalize runs blocks of kFinThreads threads. Its merge takes up to
// kFinThreads records per pass (a chunk group is one pass), one record per
// thread, held in registers (independent 16-byte loads). Each wave reduces
// its 64 records with DPP in a fixed order (row shifts by 1, 2, 4 and 8, then
// two row broadcasts: an inclusive scan, whose last lane holds the total),
// and the wave totals are combined in wave order, so the binary64 sums are
// reproducible. (One block of 1024 threads merging up to 4096 records in
// four passes took twice as long as 16 blocks of 256 records and a second
// level: the records' loads through one CU bound it.) The lanes of a wave hold ascending, disjoint element ranges:
// among records with the same maximum the first lane holding it has the
// smallest index.
static_assert(offsetof(ChunkRec, nfound) == 92 && offsetof(ChunkRec, eq_bits) == 96 &&
                  offsetof(ChunkRec, amax_abs) == 100 && offsetof(ChunkRec, max_abs) == 112 &&
                  offsetof(ChunkRec, max_rel) == 120 && offsetof(ChunkRec, sum_abs) == 128,
              "record word layout");
constexpr int kRecWords = (int)(sizeof(ChunkRec) / 4);
constexpr int kFinThreads = kBlockThreads;
constexpr int kFinWaves = kFinThreads / kWaveSize;
static_assert(kGroupChunks % kFinThreads == 0, "a chunk group is whole merge passes");

struct MergeScratch {
  // per-wave totals of the current pass
  uint32_t wcnt[kFinWaves][kRecCounts];
  uint32_t wnf[kFinWaves], weq[kFinWaves];
  double wsum[2][kFinWaves], wmax[2][kFinWaves];
  uint64_t widx[2][kFinWaves];
  uint32_t woff[kFinWaves];                  // first output position of each wave's entries
  uint32_t nfstart[kFinThreads];             // first output position of each record
  uint32_t pass_lo, pass_hi;                 // output positions of the pass's entries
  // running totals over the passes
  uint64_t cnt[kRecCounts];
  double sum_abs, sum_rel, max_abs, max_rel;
  uint64_t amax_abs, amax_rel;
  uint32_t eq_all, nf_total;
};

// Inclusive scan of a 32-bit value over the wave with one combining
// operation per step (lanes with no source combine with `id`).
template <typename Op>
__device__ __forceinline__ uint32_t wave_scan_u32(uint32_t x, uint32_t id, Op op) {
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, x, 0x111, 0xf, 0xf, false));  // row_shr:1
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, x, 0x112, 0xf, 0xf, false));  // row_shr:2
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, x, 0x114, 0xf, 0xf, false));  // row_shr:4
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, x, 0x118, 0xf, 0xf, false));  // row_shr:8
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, x, 0x142, 0xa, 0xf, false));  // row_bcast:15
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, x, 0x143, 0xc, 0xf, false));  // row_bcast:31
  return x;
}

// Merges records recs[0..n) into the totals in s; record i covers elements
// [i * span, (i + 1) * span) of the parent range. With
// k > 0 the staged
// first-k lists are concatenated in record order (entry e of record i is
// parent element i * span + e) into out64 (final: global indices) or out32
// (a group: offsets within the group), at most k entries; s.nf_total is
// their number. Called by the whole block; the totals are valid for every
// thread on return.
template <bool FINAL>
__device__ __forceinline__ void merge_all(MergeScratch &s, const ChunkRec *__restrict__ recs,
                                          uint32_t n, uint64_t span,
                                          const uint32_t *__restrict__ stage,
                                          uint64_t stage_stride, uint32_t k,
                                          uint32_t *__restrict__ out32,
                                          int64_t *__restrict__ out64) {
  const uint32_t t = threadIdx.x, lane = t % kWaveSize, wave = t / kWaveSize;
  if (t < (uint32_t)kRecCounts) s.cnt[t] = 0;
  if (t == 0) {
    s.sum_abs = s.sum_rel = 0.0;
    s.max_abs = s.max_rel = -1.0;
    s.amax_abs = s.amax_rel = UINT64_MAX;
    s.eq_all = 0xffffffffu;
    s.nf_total = 0;
  }
  for (uint32_t base = 0; base < n; base += kFinThreads) {
    const uint32_t m = min(n - base, (uint32_t)kFinThreads);
    // the record of this thread; past the pass's last record, the neutral
    // record (no counts, no entries, all equality bits, no maximum)
    u32x4 v[kRecWords / 4];
    if (t < m) {
      const u32x4 *src = (const u32x4 *)(recs + base + t);
#pragma unroll
      for (int i = 0; i < kRecWords / 4; ++i) v[i] = src[i];
    } else {
      const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < 6; ++i) v[i] = z;                // words 0..23
      v[6] = (u32x4){0xffffffffu, kNone, kNone, 0u};       // eq_bits, amax, pad
      v[7] = (u32x4){0u, 0xbff00000u, 0u, 0xbff00000u};    // max_abs = max_rel = -1
      v[8] = z;                                            // sums
    }
    auto word = [&](int i) __attribute__((always_inline)) -> uint32_t { return v[i / 4][i % 4]; };
    auto dword = [&](int i) __attribute__((always_inline)) -> double {
      const uint64_t lo = word(i), hi = word(i + 1);
      return __longlong_as_double((long long)(lo | hi << 32));
    };
    const auto add = [](uint32_t a, uint32_t b) { return a + b; };
    // counters: a record counts at most kGroupChunks * kMaxChunkElems
    // (a group record), so a wave's sum fits 32 bits
    static_assert((uint64_t)kGroupChunks * kMaxChunkElems * kWaveSize <= (1ull << 32),
                  "wave sums of record counts");
#pragma unroll
    for (int f = 0; f < kRecCounts; ++f) {
      const uint32_t c = wave_scan_u32(word(f), 0u, add);
      if (lane == kWaveSize - 1) s.wcnt[wave][f] = c;
    }
    const uint32_t nf = word(23);
    const uint32_t nf_incl = wave_scan_u32(nf, 0u, add);
    const uint32_t eq =
        wave_scan_u32(word(24), 0xffffffffu, [](uint32_t a, uint32_t b) { return a & b; });
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const double sm = wave_sum(dword(32 + 2 * f));
      const double x = dword(28 + 2 * f);
      const double mx = wave_max_val(x);
      // the first lane holding the maximum (-1: no lane has one)
      const uint64_t holders = ballot(x == mx);
      const uint32_t hl = holders != 0 ? (uint32_t)__builtin_ctzll(holders) : 0u;
      const uint32_t ai = __builtin_amdgcn_readlane(word(25 + f), hl);
      if (lane == kWaveSize - 1) {
        s.wsum[f][wave] = sm;
        s.wmax[f][wave] = mx;
        s.widx[f][wave] = mx > -1.0 ? (uint64_t)(base + wave * kWaveSize + hl) * span + ai
                                    : UINT64_MAX;
      }
    }
    if (lane == kWaveSize - 1) {
      s.wnf[wave] = nf_incl;
      s.weq[wave] = eq;
    }
    __syncthreads();
    // the wave totals, in wave order, one role per thread
    if (t < (uint32_t)kRecCounts) {
      uint64_t a = s.cnt[t];
#pragma unroll
      for (int w = 0; w < kFinWaves; ++w) a += s.wcnt[w][t];
      s.cnt[t] = a;
    } else if (t == 64 || t == 65) {
      const uint32_t f = t - 64;
      double a = f ? s.sum_rel : s.sum_abs;
#pragma unroll
      for (int w = 0; w < kFinWaves; ++w) a += s.wsum[f][w];
      if (f) s.sum_rel = a;
      else s.sum_abs = a;
    } else if (t == 128 || t == 129) {
      // (earlier records first: a strict comparison keeps them on ties)
      const uint32_t f = t - 128;
      double bv = f ? s.max_rel : s.max_abs;
      uint64_t bi = f ? s.amax_rel : s.amax_abs;
#pragma unroll
      for (int w = 0; w < kFinWaves; ++w) {
        const bool take = s.wmax[f][w] > bv;
        bv = take ? s.wmax[f][w] : bv;
        bi = take ? s.widx[f][w] : bi;
      }
      if (f) {
        s.max_rel = bv;
        s.amax_rel = bi;
      } else {
        s.max_abs = bv;
        s.amax_abs = bi;
      }
    } else if (t == 192) {
      uint32_t e = s.eq_all;
#pragma unroll
      for (int w = 0; w < kFinWaves; ++w) e &= s.weq[w];
      s.eq_all = e;
    } else if (t == 193) {
      // (a wave lists at most 64 k <= 2^16 entries: no overflow)
      uint32_t c = s.nf_total;
      s.pass_lo = c;
#pragma unroll
      for (int w = 0; w < kFinWaves; ++w) {
        s.woff[w] = c;
        c = min(c + s.wnf[w], k);
      }
      s.pass_hi = c;
      s.nf_total = c;
    }
    __syncthreads();
    if (k > 0) {
      // first output position of each record: its wave's offset plus the
      // entries of the records before it in the wave
      if (t < m) s.nfstart[t] = min(s.woff[wave] + (nf_incl - nf), k);
      __syncthreads();
      // one output entry per thread: entry e belongs to the last record whose
      // first position is <= e
      const uint32_t lo = s.pass_lo, hi = s.pass_hi;
      for (uint32_t e = lo + t; e < hi; e += kFinThreads) {
        uint32_t a = 0, b = m - 1;
        while (a < b) {
          const uint32_t mid = (a + b + 1) / 2;
          if (s.nfstart[mid] <= e) a = mid;
          else b = mid - 1;
        }
        const uint64_t r = base + a;
        const uint64_t gi = r * span + stage[r * stage_stride + (e - s.nfstart[a])];
        if constexpr (FINAL) out64[e] = (int64_t)gi;
        else out32[e] = (uint32_t)gi;
      }
      __syncthreads();
    }
  }
  __syncthreads();
}

// Output pointers and options of the completion path (copied field by field
// from the kernel argument: a reference to the by-value argument would force
// it into private memory).
struct FinArgs {
  vc_stats *stats;
  uint64_t *mismatches;
  uint8_t *pass_out;
  int64_t *first_k;
  vc_integrity *integ;
  double *match_rate;
  double *numeric_rate;
  Counters *ctr;
  int32_t n_cases, n_tols, primary, k, do_integ;
};

// Writes the results of a case from its records (chunk records when the case
// has one group, else group records) and, for the last case of the call, the
// suite match rates. Called by the whole block.
__device__ __forceinline__ void finalize_case(MergeScratch &s, const FinArgs &P, const DevCase &cs,
                              const ChunkRec *recs, uint32_t n, uint64_t span,
                              const uint32_t *stage, uint64_t stage_stride) {
  const bool ok = cs.status == 0;
  const uint32_t oi = cs.orig;
  const bool want_fk = P.first_k != nullptr && P.k > 0;
  const uint32_t k = want_fk ? (uint32_t)P.k : 0u;
  int64_t *const fk = want_fk ? P.first_k + (uint64_t)oi * k : nullptr;
  merge_all<true>(s, recs, n, span, stage, stage_stride, ok ? k : 0u, nullptr, fk);
  if (want_fk) {
    const uint32_t nf = ok ? s.nf_total : 0u;
    for (uint32_t pos = nf + threadIdx.x; pos < k; pos += kFinThreads) fk[pos] = -1;
  }
  if (threadIdx.x != 0) return;
  const int nt = P.n_tols;
  const int prim = P.primary;
  const uint64_t n_el = ok ? cs.numel : 0;
  auto cnt = [&](int w) -> uint64_t { return ok ? s.cnt[w] : 0; };
  vc_stats st;
  st.numel = cs.numel;
  st.mismatches = cnt(prim);
  st.nan_cand = cnt(8);
  st.inf_cand = cnt(9);
  st.nan_ref = cnt(10);
  st.inf_ref = cnt(11);
  st.n_finite = cnt(12);
  st.n_rel = cnt(13);
  st.n_rel_undef = cnt(14);
  const bool has_abs = ok && s.amax_abs != UINT64_MAX;
  const bool has_rel = ok && s.amax_rel != UINT64_MAX;
  st.max_abs = has_abs ? s.max_abs : 0.0;
  st.argmax_abs = has_abs ? (int64_t)s.amax_abs : -1;
  st.max_rel = has_rel ? s.max_rel : 0.0;
  st.argmax_rel = has_rel ? (int64_t)s.amax_rel : -1;
  st.sum_abs = ok ? s.sum_abs : 0.0;
  st.sum_rel = ok ? s.sum_rel : 0.0;
  st.case_status = cs.status;
  st.pass = (ok && cnt(prim) == 0) ? 1 : 0;
  if (P.stats != nullptr) P.stats[oi] = st;
  for (int p = 0; p < nt; ++p) {
    const uint8_t pass = (ok && cnt(p) == 0) ? 1 : 0;
    if (P.pass_out != nullptr) P.pass_out[(uint64_t)oi * nt + p] = pass;
    if (P.mismatches != nullptr) P.mismatches[(uint64_t)oi * nt + p] = cnt(p);
  }
  uint32_t flags = 0;
  if (P.do_integ) {
    const uint64_t zc = cnt(15), zr = cnt(16), efc = cnt(17), efr = cnt(18);
    const uint64_t bfc = cnt(19), bfr = cnt(20), hfc = cnt(21), hfr = cnt(22);
    vc_integrity g;
    g.zero_cand = zc;
    g.zero_ref = zr;
    g.eqfirst_cand = efc;
    g.eqfirst_ref = efr;
    g.bf16rep_cand = bfc;
    g.bf16rep_ref = bfr;
    g.fp16rep_cand = hfc;
    g.fp16rep_ref = hfr;
    const uint32_t eqb = ok ? s.eq_all : 0u;
    const uint32_t inp_mask = ok ? cs.inp_mask : 0u;
    const uint32_t eq_c = (eqb >> kEqCandInpShift) & 0xffu & inp_mask;
    const uint32_t eq_r = (eqb >> kEqRefInpShift) & 0xffu & inp_mask;
    g.cand_eq_input_mask = eq_c;
    g.ref_eq_input_mask = eq_r;
    g.cand_eq_ref = eqb & kEqCandRef;
    g.copy_input = -1;
    if (ok) {
      const bool f32 = cs.dtype == VC_F32;
      if (zc == n_el && n_el >= 1 && zr < n_el) flags |= VC_FLAG_ALL_ZERO;
      if (efc == n_el && n_el >= 2 && zc < n_el && efr < n_el) flags |= VC_FLAG_CONSTANT;
      const uint32_t copy = eq_c & ~eq_r;
      if (copy != 0) {
        flags |= VC_FLAG_INPUT_COPY;
        g.copy_input = __builtin_ctz(copy);
      }
      if (f32 && bfc == n_el && n_el >= 2 && zc < n_el && efc < n_el && bfr < n_el)
        flags |= VC_FLAG_LOWPREC_BF16;
      if (f32 && hfc == n_el && bfc < n_el && n_el >= 2 && zc < n_el && efc < n_el &&
          hfr < n_el)
        flags |= VC_FLAG_LOWPREC_FP16;
    }
    g.flags = flags;
    g.reserved = 0;
    if (P.integ != nullptr) P.integ[oi] = g;
  }
  if (P.match_rate == nullptr && P.numeric_rate == nullptr) return;
  // suite counters
  for (int p = 0; p < nt; ++p) {
    if (ok && cnt(p) == 0) {
      atomicAdd(&P.ctr->pass[p], 1u);
      if (flags == 0) atomicAdd(&P.ctr->cert[p], 1u);
    }
  }
  // The case written last writes the suite rates. Its increment of the
  // completion count acquires what every earlier case released with its
  // own increment (the counter updates above), so it reads final counters.
  const uint32_t done =
      __hip_atomic_fetch_add(&P.ctr->done, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
  if (done + 1 != (uint32_t)P.n_cases) return;
  const double nc = (double)P.n_cases;
  for (int p = 0; p < nt; ++p) {
    const uint32_t num = __hip_atomic_load(&P.ctr->pass[p], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t cert = __hip_atomic_load(&P.ctr->cert[p], __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    if (P.match_rate != nullptr) P.match_rate[p] = (double)cert / nc;
    if (P.numeric_rate != nullptr) P.numeric_rate[p] = (double)num / nc;
    // every other case has finished with the counters: clear them for the
    // next call of a prepared sweep
    P.ctr->pass[p] = 0;
    P.ctr->cert[p] = 0;
  }
  P.ctr->done = 0;
}

// Last table entry (in [lo, hi)) whose value in `first` is <= x; `first`
// ascends strictly and first[lo] <= x. A 64-way search: each lane tests one
// probe and the ballot counts the probes at or below x. Wave-uniform.
__device__ __forceinline__ uint64_t find_entry(const uint64_t *first, uint64_t lo, uint64_t hi,
                                               uint64_t x) {
  const VCK_GLOBAL uint64_t *f = (const VCK_GLOBAL uint64_t *)first;
  const uint64_t lane = threadIdx.x & (kWaveSize - 1);
  uint64_t n = hi - lo;
  while (n > (uint64_t)kWaveSize) {
    const uint64_t stride = (n + kWaveSize - 1) / kWaveSize;
    const uint64_t idx = lo + lane * stride;
    const bool le = idx < lo + n ? f[idx] <= x : false;
    const uint64_t kx = popc(ballot(le)) - 1u;
    lo += kx * stride;
    n = min(stride, n - kx * stride);
  }
  const bool le = lane < n ? f[lo + lane] <= x : false;
  return lo + popc(ballot(le)) - 1u;
}

// ------------------------------------------------------------ main kernel

// The register budget of 72 VGPRs (seven waves per SIMD) steers the
// scheduler toward that occupancy; a variant that needs more registers still
// gets them (none spills). Binary32 storage with up to four pairs must keep
// six waves per SIMD (80 VGPRs), which it does without spilling.
template <int DT, int NT, bool INTEG>
__global__ __launch_bounds__(kBlockThreads)
__attribute__((amdgpu_num_vgpr(72), amdgpu_waves_per_eu(DT == VC_F32 && NT <= 4 ? 6 : 1)))
void main_kernel(const Params P) {
  constexpr int V = Tr<DT>::V;
  constexpr int ES = Tr<DT>::ES;
  constexpr uint32_t ITER = kWaveSize * V;  // elements per wave step
  static_assert(ITER % 256 == 0, "list entry layout");
  // Single pair, 16-bit storage: a step the fast tiers find mismatching
  // while positions are recorded is committed, and its mismatch bits wait in
  // LDS for the localization after streaming. Binary32 storage defers such
  // a step whole to the exact tier instead: there the committing path costs
  // registers (and resident waves) across the streaming loop.
  constexpr bool kBitsInLds = NT == 1 && DT != VC_F32;
  constexpr uint32_t ALL = (1u << V) - 1u;
  // binary32 tier: bound on the estimate of |c - r| / |r| under which c - r
  // is exact in binary32 (with a margin for the estimate's error)
  constexpr float QT = ES == 4 ? 0.49f : 0.998f;
  // the tier-1 range of |r| as strict bounds: 2^-60 <= |r| <= 2^30
  constexpr float kRangeHiUp = 0x1.000002p30f, kRangeLoDown = 0x1.fffffep-61f;

  struct StreamLds {
    uint32_t win[kTileWindow];    // block tile-count window
  };
  __shared__ StreamLds sh_st;
  // localization parameters, read from LDS by the (rare) localization path
  // so that they do not occupy registers across the streaming loop
  __shared__ ChunkTiles sh_loc;
  // each wave's list of deferred steps (chunk offsets of the steps), the
  // lists' lengths and first-k counts, and their merged order
  __shared__ uint32_t s_defer[kWavesPerBlock][kDeferCap];
  __shared__ uint32_t s_coop[kWavesPerBlock][2];
  __shared__ uint32_t s_order[kWavesPerBlock * kDeferCap];
  // single pair: each lane's primary-pair mismatch bits of the listed steps
  // that the fast tiers committed (indexed by wave and list position)
  __shared__ uint8_t s_pb[kWavesPerBlock][kDeferCap][kWaveSize];
  // dynamic LDS (launched with 5 * k words): each wave's ordered first-k
  // list, then the merged list of the block
  extern __shared__ uint32_t dyn_lds[];
  __shared__ ChunkRec s_out[kWavesPerBlock];
  // counters touched only by the exact tier, per wave (kept out of scalar
  // registers): nan_c, inf_c, nan_r, inf_r, n_fin, n_rel, n_rel_undef
  __shared__ uint32_t s_rare[kWavesPerBlock][8];

  // The block's set-up runs at raised wave priority: it is a short serial
  // chain that otherwise waits behind the streaming waves of the other
  // blocks on the SIMD, keeping the block's slot from streaming; the
  // streaming loop runs at the base priority.
  __builtin_amdgcn_s_setprio(3);
  const uint32_t lane = threadIdx.x & (kWaveSize - 1);
  // wave index: uniform per wave (keeps every range bound in scalar registers)
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  const uint64_t chunk = P.chunk_lo + blockIdx.x;

  // Locate the case: the last table entry whose first chunk is <= chunk. A
  // 64-way search: each lane tests one probe, the ballot counts the probes at
  // or below the chunk (the first chunks ascend strictly).
  const VCK_CONST DevCase *table = (const VCK_CONST DevCase *)P.cases;
  uint64_t ci = 0;
  if (table != nullptr) ci = find_entry(P.case_chunk, P.case_lo, P.case_hi, chunk);
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
  const uint64_t CH = 4 * U;
  const uint64_t rel_chunk = chunk - chunk_begin;
  const uint64_t cstart = rel_chunk * CH;
  const uint64_t cend = dcs.status != 0 ? cstart : min(cstart + CH, numel);
  const int prim = P.primary;
  // The wave's first step (chunk step `wave`, when the chunk has it) is
  // loaded here, so that its latency overlaps the block set-up below.
  u32x4 pre_c = {0u, 0u, 0u, 0u}, pre_r = {0u, 0u, 0u, 0u};
  if (vec && (uint64_t)(wave + 1) * ITER <= cend - cstart) {
    const uint64_t i0 = cstart + (uint64_t)wave * ITER;
    pre_c = load16(cand + i0 * ES + lane * 16u);
    pre_r = load16(ref + i0 * ES + lane * 16u);
  }
  // Params fields used by the step lambdas, as locals: the lambdas capture by
  // reference, and a captured by-value argument would live in private memory.
  const int32_t kk = P.k;
  const bool do_tiles = P.do_tiles != 0;
  const uint32_t eqnan_mask = P.eqnan_mask;
  const bool t1ok = P.tier1 != 0;
  uint32_t *const tile_maps = P.tile_maps;
  // tolerance pairs in registers (constant indices only: a runtime index into
  // the kernel-argument struct would copy it to private memory)
  double atol[NT], rtol[NT];
#pragma unroll
  for (int p = 0; p < NT; ++p) {
    atol[p] = P.atol[p];
    rtol[p] = P.rtol[p];
  }
  const float rlo = P.rlo, alo = P.alo, rhi = P.rhi, ahi = P.ahi;
  const float alo_up = f32_next_up(alo);

  // Per-lane exact best (value, chunk offset) of d (k = 0) and of the
  // quotient (k = 1), kept in LDS: only the rare update paths touch them, so
  // the streaming loop carries no registers for them.
  __shared__ double s_bv[2][kWavesPerBlock][kWaveSize];
  __shared__ uint32_t s_bi[2][kWavesPerBlock][kWaveSize];
  s_bv[0][wave][lane] = -1.0;
  s_bv[1][wave][lane] = -1.0;
  s_bi[0][wave][lane] = kNone;
  s_bi[1][wave][lane] = kNone;
  // per-lane binary64 sums
  double acc_abs = 0.0, acc_rel = 0.0;
  // Wave-uniform running thresholds, kept in LDS: the rare update paths
  // (raise_abs, raise_rel) write them and every step reads a snapshot, so
  // the streaming loop carries no registers for them.
  //  T_abs, T_rel   the wave's best d and quotient so far (-1: none);
  //  thr_abs        T_abs rounded down to binary32, thr_abs_up the next float;
  //  b_rel          T_rel lowered by 2^-20 and rounded down (0 when T_rel = 0);
  //  rel_zero       T_rel == 0: any d > 0 beats it;
  //  b_mul, s_rel   the single-pair quotient screen: an element passes when
  //                 |d| - b_mul |r| < s_rel, b_mul = b_rel (binary32 /
  //                 bfloat16 storage: at most the exactness bound QT), or 0
  //                 with s_rel = 2^-149 while T_rel = 0 (any d > 0 is caught).
  struct WaveThr {
    double T_abs, T_rel;
    float thr_abs, thr_abs_up, b_rel, b_mul, s_rel;
    uint32_t rel_zero;
  };
  __shared__ WaveThr s_thr[kWavesPerBlock];
  // The quotient screen of every wave uses the largest quotient any wave of
  // the block has found so far: it is a value reached by some element, and
  // the screen (lowered by 2^-20) passes every quotient at or above it, ties
  // included, so it only drops elements that cannot hold the maximum. Kept
  // as the bits of the lowered binary32 bound b_rel (> 0; 0: none), raised by
  // an LDS atomic maximum. The exact tests and the zero-quotient screen stay
  // with the wave's own best: they skip ties, which only stream order within
  // the wave justifies.
  __shared__ uint32_t s_blk_rel;
  if (threadIdx.x == 0) s_blk_rel = 0u;
  {
    WaveThr t;
    t.T_abs = t.T_rel = -1.0;
    t.thr_abs = t.b_rel = t.b_mul = -1.0f;
    t.thr_abs_up = f32_next_up(-1.0f);
    t.s_rel = 0.0f;
    t.rel_zero = 0;
    s_thr[wave] = t;
  }
  // wave-uniform counters
  uint32_t mism[NT];
#pragma unroll
  for (int p = 0; p < NT; ++p) mism[p] = 0;
  uint32_t fast_steps = 0;  // steps committed by tiers 1 and 2
  if (lane < 8) s_rare[wave][lane] = 0;
  uint32_t zc = 0, zr = 0, efc = 0, efr = 0, bfc = 0, bfr = 0, hfc = 0, hfr = 0;
  uint64_t diff_cr = 0;
  uint32_t eqc = INTEG ? inp_mask : 0u, eqr = eqc;
  uint32_t nfound = 0;
  uint32_t first_c = 0, first_r = 0;
  if constexpr (INTEG) {
    if (numel > 0 && dcs.status == 0) {
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
  const uint32_t kq = kk > 0 ? (uint32_t)kk : 0u;
  if (threadIdx.x == 0) {
    ChunkTiles g = {};
    g.tile_maps = tile_maps;
    g.kq = kq;
    g.do_tiles = do_tiles ? 1u : 0u;
    if (do_tiles && cend > cstart) {
      const uint64_t th = (uint64_t)P.tile_h, tw = (uint64_t)P.tile_w;
      g.wide = cols >= (1ull << 31) ? 1u : 0u;
      // 32-bit magic-number divisions where the operands fit (the usual
      // case); 64-bit division otherwise
      constexpr uint64_t k32 = 1ull << 32;
      const uint64_t row0 = (!g.wide && cstart < k32)
                                ? div_by((uint32_t)cstart, dcs.cols_div.m, dcs.cols_div.shifts)
                                : cstart / cols;
      const uint64_t col0 = cstart - row0 * cols;
      g.tiles_c = tiles_c;
      g.trow0 = row0 < k32 ? div_by((uint32_t)row0, P.th_div.m, P.th_div.shifts) : row0 / th;
      g.rrem0 = (uint32_t)(row0 - g.trow0 * th);
      g.col0 = (uint32_t)col0;
      g.cols32 = (uint32_t)cols;
      g.room = cols - col0;
      g.tcol0 = col0 < k32 ? div_by((uint32_t)col0, P.tw_div.m, P.tw_div.shifts) : col0 / tw;
      g.crem0 = (uint32_t)(col0 - g.tcol0 * tw);
      g.cdiv = dcs.cols_div;
      g.hdiv = P.th_div;
      g.wdiv = P.tw_div;
      g.tile_off = tile_off;
      // tiles of the first and last element; a chunk spanning several rows
      // also covers the start (end) of its first (last) tile row when that
      // tile row holds another of its rows
      const uint32_t last = (uint32_t)(cend - cstart - 1);
      uint32_t dr_first;
      const uint64_t t_first = tile_at(g, 0, dr_first), t_last = tile_at(g, last, dr_first);
      const uint32_t dr_last =
          g.wide ? ((uint64_t)last >= g.room ? 1u : 0u) : div_by(g.col0 + last, g.cdiv.m, g.cdiv.shifts);
      const uint32_t rr_last = g.rrem0 + dr_last;  // below 2^31: a chunk spans < 2^18 rows
      const uint32_t rq_last = div_by(rr_last, P.th_div.m, P.th_div.shifts);
      const uint64_t tr_last = g.trow0 + rq_last;
      const bool multi = dr_last > 0;
      const uint64_t t_min = (multi && g.rrem0 + 1 < th) ? g.trow0 * tiles_c : t_first;
      const uint64_t t_max =
          (multi && rr_last != rq_last * (uint32_t)th) ? tr_last * tiles_c + tiles_c - 1 : t_last;
      if (t_max - t_min < (uint64_t)kTileWindow) {
        g.win_base = t_min;
        g.win_len = (uint32_t)(t_max - t_min + 1);
      }
    }
    sh_loc = g;
  }
  __syncthreads();
  {
    const uint32_t wl = sh_loc.win_len;
    for (uint32_t e = threadIdx.x; e < wl; e += kBlockThreads) sh_st.win[e] = 0;
  }
  __syncthreads();
  __builtin_amdgcn_s_setprio(0);

  // Localization of the primary-pair mismatches given by per-lane bit mask
  // pb (bit j = the element at chunk offset off0 + j): ordered first-k
  // staging and tile counts.
  auto localize = [&](uint32_t pb, uint32_t off0) __attribute__((always_inline)) {
    asm volatile("" ::: "memory");  // read the block's parameters from LDS here
    const ChunkTiles &g = sh_loc;
    if (nfound < kq) {
      uint32_t *const lstage = dyn_lds + wave * kq;  // this wave's list
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
        if (pos < kq) lstage[pos] = off0 + j;
        ++pos;
      }
      nfound = min(nfound + total, kq);
    }
    if (g.do_tiles != 0 && pb != 0) {
      // a lane's elements are consecutive: when its first and last
      // mismatches lie in one row and one tile, so do all of them (one
      // addition)
      uint32_t dr_lo, dr_hi;
      const uint64_t t_lo = tile_at(g, off0 + __builtin_ctz(pb), dr_lo);
      const uint64_t t_hi = tile_at(g, off0 + 31 - __builtin_clz(pb), dr_hi);
      const bool one = t_lo == t_hi && dr_lo == dr_hi;
      uint32_t bits = one ? 1u : pb;
      const uint32_t add = one ? popc(pb) : 1u;
      while (bits != 0) {
        const int j = __builtin_ctz(bits);
        bits &= bits - 1;
        uint32_t dr;
        const uint64_t t = one ? t_lo : tile_at(g, off0 + j, dr);
        if (t - g.win_base < (uint64_t)g.win_len)
          atomicAdd(&sh_st.win[t - g.win_base], add);
        else
          atomicAdd(&g.tile_maps[g.tile_off + t], add);
      }
    }
  };

  // Whether mismatch positions are still recorded: tile maps requested, or
  // the wave's first-k list not yet full (uniform).
  auto loc_on = [&]() __attribute__((always_inline)) {
    return do_tiles || nfound < kq;
  };

  // Raise the wave thresholds to the lanes' bests (after an update).
  auto raise_abs = [&](uint64_t lanes) __attribute__((always_inline)) {
    const double lb_abs = s_bv[0][wave][lane];
    const double v = popc(lanes) == 1 ? readlane_f64(lb_abs, (uint32_t)__builtin_ctzll(lanes))
                                      : wave_max_val(lb_abs);
    if (v > s_thr[wave].T_abs) {
      const float t = f32_down(v);
      s_thr[wave].T_abs = v;
      s_thr[wave].thr_abs = t;
      s_thr[wave].thr_abs_up = f32_next_up(t);
    }
  };
  auto raise_rel = [&](uint64_t lanes) __attribute__((always_inline)) {
    const double lb_rel = s_bv[1][wave][lane];
    const double v = popc(lanes) == 1 ? readlane_f64(lb_rel, (uint32_t)__builtin_ctzll(lanes))
                                      : wave_max_val(lb_rel);
    if (v > s_thr[wave].T_rel) {
      const bool zero = !(v > 0.0);
      const float b = zero ? 0.0f : f32_down(v * (1.0 - 0x1p-20));
      s_thr[wave].T_rel = v;
      s_thr[wave].b_rel = b;
      s_thr[wave].rel_zero = zero ? 1u : 0u;
      s_thr[wave].b_mul = zero ? 0.0f : (DT != VC_F16 ? __builtin_fminf(b, QT) : b);
      s_thr[wave].s_rel = zero ? 0x1p-149f : 0.0f;
      if (lane == 0 && b > 0.0f)
        __hip_atomic_fetch_max(&s_blk_rel, __float_as_uint(b), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  };
  // Tier-1 update of the lane bests for the lanes in absm | relm, given each
  // lane's largest |c - r| (md) and largest quotient estimate (mq) of the
  // step. Every |c - r| of the step is exact in binary32: a lane whose md
  // beats its best finds the first element holding md. For the quotient,
  // only elements whose estimate lies within 2^-19 of mq can hold the step's
  // largest quotient (the estimates are within 2^-21 of the quotients); each
  // of them (usually one) is divided exactly in binary64 and compared.
  auto t1_update = [&](const u32x4 &cq, const u32x4 &rq, uint64_t absm, uint64_t relm,
                       uint32_t off0, float md, float mq) __attribute__((always_inline)) {
    if (((absm >> lane) & 1ull) && (double)md > s_bv[0][wave][lane]) {
      uint32_t jb = 0;
#pragma unroll 1
      for (int j = V - 1; j >= 0; --j)
        if (__builtin_fabsf(diff32<DT>(cq, rq, j)) == md) jb = (uint32_t)j;
      s_bv[0][wave][lane] = md;
      s_bi[0][wave][lane] = off0 + jb;
    }
    if ((relm >> lane) & 1ull) {
      double lb_rel = s_bv[1][wave][lane];
      uint32_t li_rel = s_bi[1][wave][lane];
      const float band = mq * (1.0f - 0x1p-19f);
#pragma unroll 1
      for (int j = 0; j < V; ++j) {
        const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
        const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
        if (d * __builtin_amdgcn_rcpf(a) >= band) {
          const double q = (double)d / (double)a;
          if (q > lb_rel) {
            lb_rel = q;
            li_rel = off0 + (uint32_t)j;
          }
        }
      }
      s_bv[1][wave][lane] = lb_rel;
      s_bi[1][wave][lane] = li_rel;
    }
    if (absm != 0) raise_abs(absm);
    if (relm != 0) raise_rel(relm);
  };

  // Single-pair variant of t1_update (every |c - r| of the step exact in
  // binary32, every r finite and non-zero), with its element loops unrolled
  // and free of branches. A lane in absm whose md beats its best records the
  // first element holding md. A lane in relm forms its elements' quotient
  // estimates (largest mq, within 2^-21 of the quotients), then takes as
  // candidates the elements with |d| - b |r| >= 0 for b = mq (1 - 2^-19) (an
  // exact sign): they include every element that can hold the largest
  // quotient, and any other element's quotient lies more than 2^-20 below it,
  // so it cannot tie after rounding. A lane with one candidate (the rule)
  // divides it once in binary64; a lane with several evaluates them in
  // order, exactly.
  auto t1_update1 = [&](const u32x4 &cq, const u32x4 &rq, uint64_t absm, uint64_t relm,
                        uint32_t off0, float md) __attribute__((always_inline)) {
    if (((absm >> lane) & 1ull) && (double)md > s_bv[0][wave][lane]) {
      uint32_t jb = 0;
#pragma unroll
      for (int j = V - 1; j >= 0; --j)
        jb = __builtin_fabsf(diff32<DT>(cq, rq, j)) == md ? (uint32_t)j : jb;
      s_bv[0][wave][lane] = md;
      s_bi[0][wave][lane] = off0 + jb;
    }
    if (DT == VC_BF16 && ((relm >> lane) & 1ull)) {
      // (bfloat16: the unrolled form below costs registers, and with them
      // resident waves; the rolled form tests every element in the band)
      double lb_rel = s_bv[1][wave][lane];
      uint32_t li_rel = s_bi[1][wave][lane];
      float mq = 0.0f;
#pragma unroll 1
      for (int j = 0; j < V; ++j) {
        const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
        const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
        mq = __builtin_fmaxf(mq, d * __builtin_amdgcn_rcpf(a));
      }
      const float nb = -(mq * (1.0f - 0x1p-19f));
#pragma unroll 1
      for (int j = 0; j < V; ++j) {
        const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
        const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
        if (__builtin_fmaf(nb, a, d) >= 0.0f) {
          const double q = (double)d / (double)a;
          if (q > lb_rel) {
            lb_rel = q;
            li_rel = off0 + (uint32_t)j;
          }
        }
      }
      s_bv[1][wave][lane] = lb_rel;
      s_bi[1][wave][lane] = li_rel;
    }
    if (DT != VC_BF16 && relm != 0) {
      const bool mine = (relm >> lane) & 1ull;
      float mq = 0.0f;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
        const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
        mq = __builtin_fmaxf(mq, d * __builtin_amdgcn_rcpf(a));
      }
      const float nb = -(mq * (1.0f - 0x1p-19f));
      uint32_t ncand = 0, cj = 0;
      float cd = 0.0f, ca = 1.0f;
#pragma unroll
      for (int j = V - 1; j >= 0; --j) {
        const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
        const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
        const bool c = __builtin_fmaf(nb, a, d) >= 0.0f;
        ncand += c ? 1u : 0u;
        cj = c ? (uint32_t)j : cj;
        cd = c ? d : cd;
        ca = c ? a : ca;
      }
      double lb_rel = s_bv[1][wave][lane];
      uint32_t li_rel = s_bi[1][wave][lane];
      const double q1 = (double)cd / (double)ca;
      if (mine && q1 > lb_rel) {
        lb_rel = q1;
        li_rel = off0 + cj;
      }
      // (mq = 0: every quotient is 0 and the first element holds it, as taken)
      const bool several = mine && ncand > 1 && mq > 0.0f;
      if (ballot(several) != 0 && several) {
#pragma unroll 1
        for (int j = 0; j < V; ++j) {
          const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
          const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
          if (__builtin_fmaf(nb, a, d) >= 0.0f) {
            const double q = (double)d / (double)a;
            if (q > lb_rel) {
              lb_rel = q;
              li_rel = off0 + (uint32_t)j;
            }
          }
        }
      }
      if (mine) {
        s_bv[1][wave][lane] = lb_rel;
        s_bi[1][wave][lane] = li_rel;
      }
    }
    if (absm != 0) raise_abs(absm);
    if (relm != 0) raise_rel(relm);
  };

  // Exact updates of the lane bests for the lanes in `lanes` (every element
  // of those lanes is finite with r != 0: tiers 1 and 2 only, in stream
  // order, so an equal value never replaces the best).
  auto abs_update = [&](const u32x4 &cq, const u32x4 &rq, uint64_t lanes, uint32_t off0)
                        __attribute__((always_inline)) {
    if ((lanes >> lane) & 1ull) {
      double lb_abs = s_bv[0][wave][lane];
      uint32_t li_abs = s_bi[0][wave][lane];
#pragma unroll 1
      for (int j = 0; j < V; ++j) {
        const double d = __builtin_fabs(dec64<DT>(elem<DT>(cq, j)) - dec64<DT>(elem<DT>(rq, j)));
        const uint32_t o = off0 + j;
        if (d > lb_abs) {
          lb_abs = d;
          li_abs = o;
        }
      }
      s_bv[0][wave][lane] = lb_abs;
      s_bi[0][wave][lane] = li_abs;
    }
    raise_abs(lanes);
  };
  auto rel_update = [&](const u32x4 &cq, const u32x4 &rq, uint64_t lanes, uint32_t off0)
                        __attribute__((always_inline)) {
    if ((lanes >> lane) & 1ull) {
      double lb_rel = s_bv[1][wave][lane];
      uint32_t li_rel = s_bi[1][wave][lane];
#pragma unroll 1
      for (int j = 0; j < V; ++j) {
        const double r = dec64<DT>(elem<DT>(rq, j));
        const double d = __builtin_fabs(dec64<DT>(elem<DT>(cq, j)) - r);
        const double a = __builtin_fabs(r);
        const uint32_t o = off0 + j;
        // exact sign test: d / a > lb  <=>  d - lb * a > 0
        const double e = __builtin_fma(-lb_rel, a, d);
        if (a != 0.0 && e > 0.0) {
          const double q = d / a;
          if (q > lb_rel) {
            lb_rel = q;
            li_rel = o;
          }
        }
      }
      s_bv[1][wave][lane] = lb_rel;
      s_bi[1][wave][lane] = li_rel;
    }
    raise_rel(lanes);
  };

  // Exact binary64 evaluation of one step (element by element). Returns the
  // lane's primary-pair mismatch bits (bit j: element j) for the caller's
  // localization.
  auto exact_step = [&](const u32x4 &cq, const u32x4 &rq, uint32_t vmask, uint32_t off0)
                        __attribute__((always_inline)) -> uint32_t {
    uint32_t pb = 0;
    uint32_t nan_c_step = 0, nan_r_step = 0, inf_c_step = 0, inf_r_step = 0;
    uint32_t fin_step = 0, rel_step = 0, undef_step = 0;
    double lb_abs = s_bv[0][wave][lane], lb_rel = s_bv[1][wave][lane];
    uint32_t li_abs = s_bi[0][wave][lane], li_rel = s_bi[1][wave][lane];
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
      // deferred steps are evaluated after later steps of the stream: an
      // equal value wins when it comes first
      const uint32_t o = off0 + j;
      if (fin) {
        acc_abs += d;
        if (d > lb_abs || (d == lb_abs && o < li_abs)) {
          lb_abs = d;
          li_abs = o;
        }
      }
      if (relok) {
        const double q = d / a;
        acc_rel += q;
        if (q > lb_rel || (q == lb_rel && o < li_rel)) {
          lb_rel = q;
          li_rel = o;
        }
      }
    }
    s_bv[0][wave][lane] = lb_abs;
    s_bv[1][wave][lane] = lb_rel;
    s_bi[0][wave][lane] = li_abs;
    s_bi[1][wave][lane] = li_rel;
    raise_abs(~0ull);
    raise_rel(~0ull);
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
    return pb;
  };

  // Tier 1 (binary32) for a full step. Returns kNotTaken (and changes
  // nothing) when some element is not finite, has r = 0, is outside the
  // exactness bound, or (single pair) falls between the gate bounds, and
  // (single pair) kDefer, changing nothing, when some element fails the gate
  // while mismatch positions are recorded. One pass computes the sums, the
  // running-maximum tests and whether any element fails a gate; the common
  // step (valid, nothing failing, no new maximum) then commits with one
  // uniform branch, and the counts of failing elements are taken in a second
  // pass over the step only when some element failed.
  auto t1_step = [&](const u32x4 &cq, const u32x4 &rq, uint32_t off0, uint32_t &pbm,
                     const WaveThr &th, double &add_a, double &add_q)
                     __attribute__((always_inline)) -> int {
    float sa0 = 0.f, sa1 = 0.f, sq0 = 0.f, sq1 = 0.f;
    float md = 0.f, mq = 0.f, mr = 0.f;
    // single pair: whether some element fails; several pairs: the failures
    // of each pair are counted in this pass (binary64 gate on the exact
    // difference)
    uint64_t fany = 0;
    uint32_t fc1[NT];
#pragma unroll
    for (int p = 0; p < NT; ++p) fc1[p] = 0;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const float r = dec32<DT>(elem<DT>(rq, j));
      const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
      const float a = __builtin_fabsf(r);
      if constexpr (NT == 1) {
        fany |= ballot(d > __builtin_fmaf(a, rlo, alo));
      } else {
        const double d64 = d, a64 = a;
#pragma unroll
        for (int p = 0; p < NT; ++p) {
          fc1[p] += popc(ballot(d64 > atol[p] + rtol[p] * a64));
        }
      }
      const float ra = __builtin_amdgcn_rcpf(a);
      const float q = d * ra;
      if (j & 1) {
        sa1 += d;
        sq1 += q;
      } else {
        sa0 += d;
        sq0 += q;
      }
      md = __builtin_fmaxf(md, d);
      mq = __builtin_fmaxf(mq, q);

      // |r| in [2^-60, 2^30]: the reciprocal, every non-zero quotient and
      // the gate thresholds stay in the normal binary32 range (a non-zero
      // |c - r| <= 0.998 |r| is at least 2^-92 there)
      if constexpr (DT != VC_F16) mr = __builtin_fmaxf(mr, __builtin_fmaf(a, 0x1p30f, ra));
    }
    const float sa = sa0 + sa1, sq = sq0 + sq1;
    // exactness: |c - r| <= QT |r| bounds the exponent gap; binary16
    // values are multiples of 2^-24, so any |c - r| < 1 is exact as well
    bool ok = __builtin_isfinite(sa + sq) && (mq <= QT || (DT == VC_F16 && md < 1.0f));
    if constexpr (DT != VC_F16) ok = ok && mr <= 0x1p60f;
    const uint64_t bad = ballot(!ok);
    const uint64_t absm = ballot(md > th.thr_abs);
    const uint64_t relm = th.rel_zero ? ballot(md > 0.0f) : ballot(mq >= th.b_rel);
    // (binary32 storage, single pair: such a step is deferred whole)
    const bool defer_loc = !kBitsInLds && NT == 1 && fany != 0 && loc_on();
    if ((bad | absm | relm | fany) == 0 && !defer_loc) {
#pragma unroll
      for (int p = 0; p < NT; ++p) mism[p] += fc1[p];
      ++fast_steps;
      add_a = (double)sa;
      add_q = (double)sq;
      return kDone;
    }
    if (bad != 0) return kNotTaken;
    if (defer_loc) return kDefer;
    const u32x4 &cs = cq, &rs = rq;
#pragma unroll
    for (int p = 0; p < NT; ++p) mism[p] += fc1[p];
    int res = kDone;
    if (NT == 1 && fany != 0) {
      // exact counts, the lane's mismatch bits and the elements between
      // the bounds
      uint32_t fcnt = 0, bits = 0;
      uint64_t amb = 0;
#pragma unroll 1
      for (int j = 0; j < V; ++j) {
        const float c = dec32<DT>(elem<DT>(cs, j));
        const float r = dec32<DT>(elem<DT>(rs, j));
        const float d = __builtin_fabsf(c - r);
        const float a = __builtin_fabsf(r);
        const bool f = d > __builtin_fmaf(a, rlo, alo);
        fcnt += popc(ballot(f));
        amb |= ballot(f && !(d > __builtin_fmaf(a, rhi, ahi)));
        bits |= (f ? 1u : 0u) << j;
      }
      if (amb != 0) return kNotTaken;
      mism[0] += fcnt;
      if (kBitsInLds && loc_on()) {
        pbm = bits;
        res = kLocate;
      }
    }
    ++fast_steps;
    add_a = (double)sa;
    add_q = (double)sq;
    if ((absm | relm) != 0) t1_update(cs, rs, absm, relm, off0, md, mq);
    return res;
  };

  // Tier 1 for a full step, single tolerance pair. One pass over the step
  // computes, per lane, in binary32:
  //  - d = c - r, the sum of |d| and the largest |d| (md);
  //  - the gate screen g = |d| - rlo |r| (one rounding): every element with
  //    g <= alo passes the binary64 gate (rlo and alo are the pair shrunk by
  //    2^-20, more than the rounding of g);
  //  - the quotient screen e = |d| - b_mul |r| (its sign is exact): an
  //    element with e < s_rel has a quotient below the running threshold
  //    and, with binary32 / bfloat16 storage, below the exactness bound QT;
  //  - for each two consecutive elements the sum of their quotients
  //    |d| / |r| as (|r1| |d0| + |r0| |d1|) / (|r0| |r1|): one reciprocal
  //    per two elements, relative error below 6 * 2^-24 (the product of two
  //    16-bit values is exact); its sum, and for binary16 its maximum p;
  //  - for binary32 / bfloat16 storage the range of |r|.
  // One ballot of "finite sums and max(g - alo_up, md - thr_abs_up,
  // max e - s_rel, exactness and range terms) < 0" commits the usual step.
  // Any other step is sorted out below, with the outcomes of t1_step.
  auto t1_single = [&](const u32x4 &cq, const u32x4 &rq, uint32_t off0, uint32_t &pbm,
                       const WaveThr &th, double &add_a, double &add_q)
                       __attribute__((always_inline)) -> int {
    const float nrlo = -rlo, nb = -th.b_mul;
    float sa = 0.f, sq = 0.f, md = 0.f, gm = 0.f, em = 0.f, pm = 0.f;
    float rmx = 0.f, rmn = 0.f;
#pragma unroll
    for (int p = 0; p < V / 2; ++p) {
      float d0, d1, g0, g1, e0, e1, P, N;
      if constexpr (DT == VC_F16) {
        const uint32_t rw = rq[p];
        d0 = diff32<DT>(cq, rq, 2 * p);
        d1 = diff32<DT>(cq, rq, 2 * p + 1);
        // (binary32 arithmetic on converted halves, which the compiler maps
        // onto v_fma_mix_f32 with binary16 operands)
        const float a0 = __builtin_fabsf(dec32<DT>(rw & 0xffffu));
        const float a1 = __builtin_fabsf(dec32<DT>(rw >> 16));
        g0 = __builtin_fmaf(nrlo, a0, __builtin_fabsf(d0));
        g1 = __builtin_fmaf(nrlo, a1, __builtin_fabsf(d1));
        e0 = __builtin_fmaf(nb, a0, __builtin_fabsf(d0));
        e1 = __builtin_fmaf(nb, a1, __builtin_fabsf(d1));
        P = h_prod(rw);
        N = h_fma_rx<1>(rw, d0, h_mul_rx<0>(rw, d1));
      } else {
        const float r0 = dec32<DT>(elem<DT>(rq, 2 * p)), r1 = dec32<DT>(elem<DT>(rq, 2 * p + 1));
        d0 = dec32<DT>(elem<DT>(cq, 2 * p)) - r0;
        d1 = dec32<DT>(elem<DT>(cq, 2 * p + 1)) - r1;
        const float a0 = __builtin_fabsf(r0), a1 = __builtin_fabsf(r1);
        g0 = __builtin_fmaf(a0, nrlo, __builtin_fabsf(d0));
        g1 = __builtin_fmaf(a1, nrlo, __builtin_fabsf(d1));
        e0 = __builtin_fmaf(a0, nb, __builtin_fabsf(d0));
        e1 = __builtin_fmaf(a1, nb, __builtin_fabsf(d1));
        P = a0 * a1;
        N = __builtin_fmaf(a1, __builtin_fabsf(d0), a0 * __builtin_fabsf(d1));
        if (p == 0) {
          rmx = __builtin_fmaxf(a0, a1);
          rmn = __builtin_fminf(a0, a1);
        } else {
          rmx = __builtin_fmaxf(rmx, __builtin_fmaxf(a0, a1));
          rmn = __builtin_fminf(rmn, __builtin_fminf(a0, a1));
        }
      }
      const float ad0 = __builtin_fabsf(d0), ad1 = __builtin_fabsf(d1);
      const float q = N * __builtin_amdgcn_rcpf(P);
      if (p == 0) {
        gm = __builtin_fmaxf(g0, g1);
        em = __builtin_fmaxf(e0, e1);
        md = __builtin_fmaxf(ad0, ad1);
        sa = ad0 + ad1;
        sq = q;
        if constexpr (DT == VC_F16) pm = q;
      } else {
        gm = __builtin_fmaxf(gm, __builtin_fmaxf(g0, g1));
        em = __builtin_fmaxf(em, __builtin_fmaxf(e0, e1));
        md = __builtin_fmaxf(md, __builtin_fmaxf(ad0, ad1));
        sa += ad0 + ad1;
        sq += q;
        if constexpr (DT == VC_F16) pm = __builtin_fmaxf(pm, q);
      }
    }
    const bool fin = __builtin_isfinite(sa + sq);
    float x = __builtin_fmaxf(__builtin_fmaxf(gm - alo_up, md - th.thr_abs_up), em - th.s_rel);
    if constexpr (DT == VC_F16) {
      // inexact difference: |d| >= 1 and a quotient at or above QT
      x = __builtin_fmaxf(x, __builtin_fminf(md - 1.0f, pm - QT));
    } else {
      // |r| outside [2^-60, 2^30] (a quotient at or above QT is caught by e)
      x = __builtin_fmaxf(x, __builtin_fmaxf(rmx - kRangeHiUp, kRangeLoDown - rmn));
    }
    if (ballot(!(fin && x < 0.0f)) == 0) {
      ++fast_steps;
      add_a = (double)sa;
      add_q = (double)sq;
      return kUsual;
    }
    // not exact in binary32, not finite, r = 0 or |r| out of range: tier 2
    bool ok = fin;
    if constexpr (DT == VC_F16) {
      ok = ok && !(md >= 1.0f && pm >= QT);
    } else {
      // a quotient at or above QT has e >= 0 with b_mul <= QT, or (best
      // quotient 0) some d > 0: decided per element
      bool exq = true;
      if (em >= th.s_rel) {
#pragma unroll ES == 4 ? V : 1
        for (int j = 0; j < V; ++j) {
          const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
          const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
          exq = exq && __builtin_fmaf(a, -QT, d) < 0.0f;
        }
      }
      ok = ok && exq && rmx <= 0x1p30f && rmn >= 0x1p-60f;
    }
    if (ballot(!ok) != 0) return kNotTaken;
    const uint64_t fany = ballot(gm > alo);
    // (binary32 storage: such a step is deferred whole)
    if (!kBitsInLds && fany != 0 && loc_on()) return kDefer;
    int res = kDone;
    if (fany != 0) {
      // exact counts, the lane's mismatch bits and the elements between the
      // bounds
      uint32_t fcnt = 0, bits = 0;
      uint64_t amb = 0;
      // (binary32 storage unrolls the element loops of this path: its
      // element index then needs no selects; 16-bit storage keeps them rolled
      // for its register budget)
#pragma unroll ES == 4 ? V : 1
      for (int j = 0; j < V; ++j) {
        const float d = __builtin_fabsf(diff32<DT>(cq, rq, j));
        const float a = __builtin_fabsf(dec32<DT>(elem<DT>(rq, j)));
        const bool f = d > __builtin_fmaf(a, rlo, alo);
        fcnt += popc(ballot(f));
        amb |= ballot(f && !(d > __builtin_fmaf(a, rhi, ahi)));
        bits |= (f ? 1u : 0u) << j;
      }
      if (amb != 0) return kNotTaken;
      mism[0] += fcnt;
      if (kBitsInLds && loc_on()) {
        pbm = bits;
        res = kLocate;
      }
    }
    ++fast_steps;
    add_a = (double)sa;
    add_q = (double)sq;
    const uint64_t absm = ballot(md > th.thr_abs);
    const uint64_t relm = ballot(em >= th.s_rel);
    if ((absm | relm) != 0) t1_update1(cq, rq, absm, relm, off0, md);
    return res;
  };

  // Tier 2 (binary64) for a full step. Returns kNotTaken (changing nothing)
  // when the step holds a NaN, an infinity or a zero reference, and (single
  // pair) kLocate, with the lane's mismatch bits in pbm, when a mismatch
  // position must be recorded.
  auto t2_step = [&](const u32x4 &cq, const u32x4 &rq, uint32_t off0, uint32_t &pbm,
                     const WaveThr &th, double &add_a, double &add_q)
                     __attribute__((always_inline)) -> int {
    double sa = 0.0, sq = 0.0;
    uint32_t fcnt[NT];
#pragma unroll
    for (int p = 0; p < NT; ++p) fcnt[p] = 0;
    uint64_t absm = 0, relm = 0;
    uint32_t bits = 0;
#pragma unroll ES == 4 ? V : 1
    for (int j = 0; j < V; ++j) {
      const double c = dec64<DT>(elem<DT>(cq, j));
      const double r = dec64<DT>(elem<DT>(rq, j));
      const double d = __builtin_fabs(c - r);
      const double a = __builtin_fabs(r);
#pragma unroll
      for (int p = 0; p < NT; ++p) {
        const double t = atol[p] + rtol[p] * a;
        const bool f = !(d <= t);
        fcnt[p] += popc(ballot(f));
        if (kBitsInLds) bits |= (f ? 1u : 0u) << j;
      }
      sa += d;
      sq += d * __builtin_amdgcn_rcp(a);
      absm |= ballot(d > th.T_abs);
      relm |= ballot(__builtin_fma(-th.T_rel, a, d) > 0.0);
    }
    if (ballot(!__builtin_isfinite(sa + sq)) != 0) return kNotTaken;
    if (!kBitsInLds && NT == 1 && fcnt[0] != 0 && loc_on()) return kDefer;
#pragma unroll
    for (int p = 0; p < NT; ++p) mism[p] += fcnt[p];
    ++fast_steps;
    add_a = sa;
    add_q = sq;
    if (absm != 0) abs_update(cq, rq, absm, off0);
    if (relm != 0) rel_update(cq, rq, relm, off0);
    if (kBitsInLds && fcnt[0] != 0 && loc_on()) {
      pbm = bits;
      return kLocate;
    }
    return kDone;
  };

  // Primary-pair mismatch bits of a step that tier 1 or 2 committed (every
  // element finite): the gate in binary64.
  auto locate_step = [&](const u32x4 &cq, const u32x4 &rq) __attribute__((always_inline)) {
    double at = 0.0, rt = 0.0;
#pragma unroll
    for (int p = 0; p < NT; ++p)
      if (p == prim) {
        at = atol[p];
        rt = rtol[p];
      }
    uint32_t pb = 0;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const double c = dec64<DT>(elem<DT>(cq, j));
      const double r = dec64<DT>(elem<DT>(rq, j));
      if (!(__builtin_fabs(c - r) <= at + rt * __builtin_fabs(r))) pb |= 1u << j;
    }
    return pb;
  };

  // Degenerate-output detector counts of one side (cand or ref) of a step
  // (bitwise; NaN handling of the binary16 test is added by the exact tier).
  // Every predicate counted here implies that the element's low 13 bits are
  // zero (zero, bfloat16- and binary16-representable values) or that it
  // equals the case's first element bit for bit, so one cheap per-lane
  // summary rules out the usual step. A predicate that holds for every
  // element of the step, or for none, is counted from lane summaries; only a
  // mixed step counts element by element.
  auto integ_side = [&](const u32x4 &xq, uint32_t first, uint32_t &n_zero, uint32_t &n_first,
                        uint32_t &n_bf, uint32_t &n_hf, uint32_t vmask, bool full)
                        __attribute__((always_inline)) {
    constexpr uint32_t kStep = kWaveSize * V;
    // count of valid elements with pred, given lane summaries all_p / any_p
    auto count = [&](bool all_p, bool any_p, auto pred) __attribute__((always_inline)) {
      if (full && ballot(!all_p) == 0) return kStep;
      if (ballot(any_p) == 0) return 0u;
      uint32_t n = 0;
#pragma unroll
      for (int j = 0; j < V; ++j) n += popc(ballot(((vmask >> j) & 1u) && pred(elem<DT>(xq, j))));
      return n;
    };
    if constexpr (DT == VC_F32) {
      uint32_t pre = 0xffffffffu;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const uint32_t x = elem<DT>(xq, j);
        pre = min(pre, ((vmask >> j) & 1u) ? min(x & 0x1fffu, x ^ first) : ~0u);
      }
      if (ballot(pre == 0) == 0) return;
      uint32_t o = 0, of = 0, mz = ~0u, mf = ~0u, mb = ~0u, m13 = ~0u, amax = 0, mn = ~0u;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const uint32_t x = elem<DT>(xq, j), ax = x & 0x7fffffffu, xf = x ^ first;
        if ((vmask >> j) & 1u) {
          o |= x;
          of |= xf;
          mf = min(mf, xf);
          mz = min(mz, ax);
          mb = min(mb, x & 0xffffu);
          m13 = min(m13, x & 0x1fffu);
          amax = max(amax, ax);
          mn = min(mn, ax - 1u);
        }
      }
      n_zero += count((o & 0x7fffffffu) == 0, mz == 0,
                      [](uint32_t x) { return (x & 0x7fffffffu) == 0; });
      n_first += count(of == 0, mf == 0, [&](uint32_t x) { return x == first; });
      n_bf += count((o & 0xffffu) == 0, mb == 0, [](uint32_t x) { return (x & 0xffffu) == 0; });
      // binary16-representable: 0, or |x| in [2^-14, 65504] with the low 13
      // bits zero (the lane-wide test); subnormal binary16 values, infinities
      // and anything else are left to the element test
      n_hf += count((o & 0x1fffu) == 0 && amax <= 0x477fe000u && mn >= 0x387fffffu, m13 == 0,
                    [](uint32_t x) {
                      const float f = __uint_as_float(x);
                      return (float)(_Float16)f == f;
                    });
    } else {
      // two elements per word: a zero half word is detected by the borrow of
      // (v - 0x00010001) into a bit that is clear in v (a conservative test)
      const uint32_t ff = first | (first << 16);
      uint32_t hit = 0, o = 0, of = 0;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t wm = (vmask >> (2 * w)) & 3u;
        const uint32_t keep = (wm & 1u ? 0x0000ffffu : 0u) | (wm & 2u ? 0xffff0000u : 0u);
        const uint32_t z = (xq[w] & 0x7fff7fffu) | ~keep, e = (xq[w] ^ ff) | ~keep;
        hit |= ((z - 0x00010001u) & ~z & 0x80008000u) | ((e - 0x00010001u) & ~e & 0x80008000u);
        o |= xq[w] & keep;
        of |= (xq[w] ^ ff) & keep;
      }
      if (ballot(hit != 0) == 0) return;
      n_zero += count((o & 0x7fff7fffu) == 0, true,
                      [](uint32_t x) { return (x & 0x7fffu) == 0; });
      n_first += count(of == 0, true, [&](uint32_t x) { return x == first; });
    }
  };

  // Detector counts and bit-equality evidence of one step.
  auto integ_step = [&](const u32x4 &cq, const u32x4 &rq, uint32_t vmask, bool full,
                        uint32_t off0) __attribute__((always_inline)) {
    const uint64_t i0 = cstart + off0;
    integ_side(cq, first_c, zc, efc, bfc, hfc, vmask, full);
    integ_side(rq, first_r, zr, efr, bfr, hfr, vmask, full);
    // cand bit-equal to ref: tested only while no difference has been seen
    if (diff_cr == 0) {
      uint32_t dx = 0;
#pragma unroll
      for (int j = 0; j < V; ++j)
        dx |= ((vmask >> j) & 1u) ? (elem<DT>(cq, j) ^ elem<DT>(rq, j)) : 0u;
      diff_cr = ballot(dx != 0);
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

  // Steps that tiers 1 and 2 do not complete (non-finite values, zero
  // references, ambiguous gate decisions and, with one tolerance pair,
  // mismatches whose positions are recorded) are deferred: the wave lists
  // them (in stream order) and later evaluates them with the exact tier,
  // reloading their data. With several pairs, a step the fast tiers
  // committed with primary-pair mismatches is listed for its positions only
  // (bit 0 of its listed offset set; offsets of steps are multiples of 256):
  // there the exact tier would evaluate every pair again. Neither the exact
  // tier's code nor the localization then runs inside the streaming loop,
  // which keeps the loop's register footprint, and with it the number of
  // resident waves, set by tiers 1 and 2 alone.
  uint32_t nd = 0;  // deferred steps of the wave (uniform)
  auto defer = [&](uint32_t off0) __attribute__((always_inline)) {
    if (lane == 0) s_defer[wave][nd] = off0;
    ++nd;
  };

  // Back-off of tier 1: after a step it cannot take, the wave skips it for
  // 1, then 3, then 7 steps while the failures go on (data that is not tame
  // tends to stay so); a step it takes resets the back-off.
  uint32_t t1_hold = 0, t1_next = 0;
  // primary-pair mismatch count of the wave (uniform)
  auto prim_count = [&]() __attribute__((always_inline)) {
    uint32_t m = 0;
#pragma unroll
    for (int p = 0; p < NT; ++p)
      if (p == prim) m = mism[p];
    return m;
  };
  auto step = [&](const u32x4 &cq, const u32x4 &rq, uint32_t off0)
                  __attribute__((always_inline)) {
    const uint32_t m0 = prim_count();
    const bool tried = t1ok && t1_hold == 0;
    uint32_t pbm = 0;
    WaveThr th = s_thr[wave];
    {
      const float bb = __uint_as_float(s_blk_rel);
      if (bb > 0.0f && bb > th.b_rel) {
        th.b_rel = bb;
        th.b_mul = DT != VC_F16 ? __builtin_fminf(bb, QT) : bb;
        th.s_rel = 0.0f;
        th.rel_zero = 0u;
      }
    }
    // the step's contributions to the binary64 sums (one update below)
    double add_a = 0.0, add_q = 0.0;
    int res = kNotTaken;
    if (tried) {
      if constexpr (NT == 1) res = t1_single(cq, rq, off0, pbm, th, add_a, add_q);
      else res = t1_step(cq, rq, off0, pbm, th, add_a, add_q);
    }
    if (res == kUsual) {
      // the usual step: nothing else to decide or record
      t1_next = 0u;  // (t1_hold is 0)
    } else {
      if (tried) {
        const bool tame = res != kNotTaken;
        t1_next = tame ? 0u : min(2u * t1_next + 1u, 7u);
        t1_hold = tame ? 0u : t1_next;
      } else if (t1_hold > 0) {
        --t1_hold;
      }
      if (res == kNotTaken) res = t2_step(cq, rq, off0, pbm, th, add_a, add_q);
      if (res == kLocate) {
        if (nd == 0) {
          // nothing of the wave is listed: its positions are recorded now, in
          // stream order, while the loads of the next steps are in flight
          localize(pbm, off0);
        } else {
          // single pair: the lane's mismatch bits wait in LDS; the entry
          // holds the offset, bit 0, the list position and the wave
          s_pb[wave][nd][lane] = (uint8_t)pbm;
          defer(off0 | 1u | (nd << 1) | (wave << 6));
        }
      } else if (res != kDone) {
        defer(off0);
      } else if (NT > 1 && prim_count() != m0 && loc_on()) {
        defer(off0 | 1u);
      }
    }
    acc_abs += add_a;
    acc_rel += add_q;
    if constexpr (INTEG) integ_step(cq, rq, ALL, true, off0);
  };

  // Steps of ITER elements (one KiB per wave and tensor), taken by the four
  // waves in rounds of four consecutive steps, so the block streams its
  // chunk front to back. With binary32 storage wave w takes position w of
  // every round; with 16-bit storage the positions rotate by one per round
  // (wave w takes position (w + round) mod 4): a faulty tile repeats at the
  // same column of every row, and rows of 16-bit data are often exactly four
  // steps long, so without the rotation all of its steps would fall to one
  // wave. The partial tail step goes to the wave owning its position. (32-bit
  // counters: a chunk holds fewer than 2^18 elements, and uniform 32-bit
  // arithmetic stays on the scalar unit.)
  const uint32_t n_steps = (uint32_t)((cend - cstart) / ITER);  // full steps in the chunk
  // binary32 storage: round robin; 16-bit storage: rotated rounds
  constexpr bool rot = ES == 2;
  const uint32_t n_rounds = n_steps / 4, n_part = n_steps % 4;
  const uint32_t n_full = rot ? n_rounds + (((wave + n_rounds) & 3u) < n_part ? 1u : 0u)
                              : (n_steps > wave ? (n_steps - wave + 3) / 4 : 0u);
  const bool tail_here = rot ? ((n_part - n_rounds) & 3u) == wave : n_part == wave;
  const uint32_t lane_off = lane * V;
  // chunk step index of the wave's step st
  auto step_idx = [&](uint32_t st) __attribute__((always_inline)) {
    return rot ? 4u * st + ((wave + st) & 3u) : wave + 4u * st;
  };
  // chunk offset of this lane's first element in the wave's step st
  auto step_off = [&](uint32_t st) __attribute__((always_inline)) {
    return step_idx(st) * ITER + lane_off;
  };
  // Evaluation of one listed step given its list entry: the mismatch
  // positions only (several pairs, bit 0 set), else the exact tier.
  auto deferred_step = [&](uint32_t entry) __attribute__((always_inline)) {
    const uint32_t e = __builtin_amdgcn_readfirstlane(entry);
    const uint32_t o0 = (e & ~0xffu) + lane_off;
    uint32_t pb;
    if (kBitsInLds && (e & 1u)) {
      pb = s_pb[(e >> 6) & 3u][(e >> 1) & 31u][lane];
    } else {
      const uint64_t i0 = cstart + o0;
      const u32x4 cq = vec ? load16(cand + i0 * ES) : load_guarded<DT>(cand, i0, cend);
      const u32x4 rq = vec ? load16(ref + i0 * ES) : load_guarded<DT>(ref, i0, cend);
      pb = (NT > 1 && (e & 1u)) ? locate_step(cq, rq) : exact_step(cq, rq, ALL, o0);
    }
    if (loc_on() && ballot(pb != 0) != 0) localize(pb, o0);
  };
  // the wave's deferred steps, in stream order
  auto flush = [&]() __attribute__((always_inline)) {
    for (uint32_t e = 0; e < nd; ++e) deferred_step(s_defer[wave][e]);
    nd = 0;
  };
  if (vec) {
    // Two steps per trip: while a step is evaluated the loads of the next
    // step are in flight. The loads are unconditional (past the end they
    // re-read the last step, a cache hit) and a trip has no exit between its
    // steps, so every step is preceded by an explicit wait for its own loads
    // only and the evaluation never waits for the prefetch, whatever path it
    // takes. The inner loop ends when the deferral list could overflow; the
    // list is then evaluated and streaming resumes.
    const uint8_t *const cb = cand + cstart * ES;  // block-uniform bases
    const uint8_t *const rb = ref + cstart * ES;
    const uint32_t lane_b = lane * 16u;
    const uint32_t last = n_full > 0 ? n_full - 1 : 0;
    auto off = [&](uint32_t st) __attribute__((always_inline)) {
      return step_idx(min(st, last)) * ITER * ES + lane_b;
    };
    auto ld = [&](const uint8_t *base, uint32_t st) __attribute__((always_inline)) {
      return load16(base + off(st));
    };
    uint32_t st = 0;
    u32x4 ca = pre_c, ra = pre_r;  // step 0 (loaded before the set-up)
    while (st < n_full) {
      while (st + 1 < n_full && nd + 2 <= (uint32_t)kDeferCap) {
        const u32x4 cn = ld(cb, st + 1), rn = ld(rb, st + 1);
        __builtin_amdgcn_s_waitcnt(kWaitVm2);
        step(ca, ra, step_off(st));
        ca = ld(cb, st + 2);
        ra = ld(rb, st + 2);
        __builtin_amdgcn_s_waitcnt(kWaitVm2);
        step(cn, rn, step_off(st + 1));
        st += 2;
      }
      if (st + 1 == n_full && nd < (uint32_t)kDeferCap) {
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        step(ca, ra, step_off(st));
        st += 1;
      }
      if (st < n_full) {  // the list is full and steps remain
        flush();
        ca = ld(cb, st);
        ra = ld(rb, st);
      }
    }
  } else {
    for (uint32_t st = 0; st < n_full; ++st) {
      const uint32_t o0 = step_off(st);
      const u32x4 cq = load_guarded<DT>(cand, cstart + o0, cend);
      const u32x4 rq = load_guarded<DT>(ref, cstart + o0, cend);
      step(cq, rq, o0);
      if (nd == (uint32_t)kDeferCap && st + 1 < n_full) flush();
    }
  }
  // The steps still listed are evaluated by the four waves together, in the
  // chunk's stream order (wave w takes every fourth), when no wave has
  // recorded a mismatch position yet: each wave then records positions in
  // increasing order, as the final merge of the four lists requires. A
  // concentrated failure (many listed steps in one wave) is thus spread over
  // the block. Otherwise each wave evaluates its own list.
  if (lane == 0) {
    s_coop[wave][0] = nd;
    s_coop[wave][1] = nfound;
  }
  __syncthreads();
  const uint32_t nd0 = s_coop[0][0], nd1 = s_coop[1][0], nd2 = s_coop[2][0], nd3 = s_coop[3][0];
  const uint32_t n_listed = nd0 + nd1 + nd2 + nd3;
  if ((s_coop[0][1] | s_coop[1][1] | s_coop[2][1] | s_coop[3][1]) == 0 && n_listed != 0) {
    // rank of every listed step among all listed steps (the lists ascend)
    for (uint32_t e = threadIdx.x; e < kWavesPerBlock * kDeferCap; e += kBlockThreads) {
      const uint32_t w = e / kDeferCap, i = e % kDeferCap;
      if (i >= s_coop[w][0]) continue;
      const uint32_t x = s_defer[w][i];
      uint32_t rank = i;
      for (uint32_t v = 0; v < (uint32_t)kWavesPerBlock; ++v) {
        if (v == w) continue;
        uint32_t lo = 0, hi = s_coop[v][0];
        while (lo < hi) {
          const uint32_t mid = (lo + hi) / 2;
          if (s_defer[v][mid] < x) lo = mid + 1;
          else hi = mid;
        }
        rank += lo;
      }
      s_order[rank] = x;
    }
    __syncthreads();
    for (uint32_t r = wave; r < n_listed; r += kWavesPerBlock) deferred_step(s_order[r]);
    nd = 0;
  } else {
    flush();
  }
  if ((cend - cstart) % ITER != 0 && tail_here) {
    const uint32_t o0 = n_steps * ITER + lane_off;
    const uint64_t i0 = cstart + o0;
    const u32x4 ct = load_guarded<DT>(cand, i0, cend);
    const u32x4 rt = load_guarded<DT>(ref, i0, cend);
    uint32_t vmask = 0;
#pragma unroll
    for (int j = 0; j < V; ++j) vmask |= (i0 + j < cend ? 1u : 0u) << j;
    const uint32_t pb = exact_step(ct, rt, vmask, o0);
    if (loc_on() && ballot(pb != 0) != 0) localize(pb, o0);
    if constexpr (INTEG) integ_step(ct, rt, vmask, false, o0);
  }

  // wave reductions (fixed order)
  double lb_abs = s_bv[0][wave][lane], lb_rel = s_bv[1][wave][lane];
  uint32_t li_abs = s_bi[0][wave][lane], li_rel = s_bi[1][wave][lane];
  wave_max_dpp(lb_abs, li_abs);
  wave_max_dpp(lb_rel, li_rel);
  acc_abs = wave_sum(acc_abs);
  acc_rel = wave_sum(acc_rel);
  if (lane == 0) {
    ChunkRec &o = s_out[wave];
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
    o.zero_c = zc;
    o.zero_r = zr;
    o.eqf_c = efc;
    o.eqf_r = efr;
    o.bf_c = bfc;
    o.bf_r = bfr;
    o.f16_c = hfc;
    o.f16_r = hfr;
    o.nfound = nfound;
    o.eq_bits = (diff_cr == 0 ? kEqCandRef : 0u) | (eqc << kEqCandInpShift) |
                (eqr << kEqRefInpShift);
    o.amax_abs = li_abs;
    o.amax_rel = li_rel;
    o.pad = 0;
    o.max_abs = li_abs == kNone ? -1.0 : lb_abs;
    o.max_rel = li_rel == kNone ? -1.0 : lb_rel;
    o.sum_abs = acc_abs;
    o.sum_rel = acc_rel;
  }
  __syncthreads();
  // flush the tile window (all four waves are done with it)
  const uint32_t f_len = sh_loc.win_len;
  for (uint32_t e = threadIdx.x; e < f_len; e += kBlockThreads) {
    const uint32_t v = sh_st.win[e];
    if (v != 0) atomicAdd(&tile_maps[tile_off + sh_loc.win_base + e], v);
  }
  // Merge the four waves' ascending first-k lists (disjoint index sets) into
  // the k smallest: an entry's rank is its position in its own list plus the
  // number of smaller entries in the other three.
  uint32_t merged = 0;
  const uint32_t *const stage0 = dyn_lds;
  uint32_t *const lmerged = dyn_lds + kWavesPerBlock * kq;
  if (kk > 0) {
    const uint32_t k = (uint32_t)kk;
    const uint32_t total =
        s_out[0].nfound + s_out[1].nfound + s_out[2].nfound + s_out[3].nfound;
    if (total > 0) {
      for (uint32_t e = threadIdx.x; e < kWavesPerBlock * k; e += kBlockThreads) {
        const uint32_t w = e / k, i = e % k;
        if (i >= s_out[w].nfound) continue;
        const uint32_t x = stage0[w * k + i];
        uint32_t rank = i;
        for (uint32_t v = 0; v < (uint32_t)kWavesPerBlock; ++v) {
          if (v == w) continue;
          uint32_t lo = 0, hi = s_out[v].nfound;  // count of list v below x
          while (lo < hi) {
            const uint32_t mid = (lo + hi) / 2;
            if (stage0[v * k + mid] < x) lo = mid + 1;
            else hi = mid;
          }
          rank += lo;
        }
        if (rank < k) lmerged[rank] = x;
      }
      merged = min(total, k);
      __syncthreads();
      for (uint32_t e = threadIdx.x; e < merged; e += kBlockThreads)
        P.stage[(uint64_t)chunk * k + e] = lmerged[e];
    }
  }
  // the chunk record: counter word q by thread q, the rest by thread 32
  {
    ChunkRec *const rec = P.recs + chunk;
    const uint32_t q = threadIdx.x;
    if (q < (uint32_t)kRecCounts) {
      uint32_t a = 0;
      for (int w = 0; w < kWavesPerBlock; ++w) a += ((const uint32_t *)&s_out[w])[q];
      ((uint32_t *)rec)[q] = a;
    } else if (q == 32) {
      uint32_t eqb = s_out[0].eq_bits;
      double ma = s_out[0].max_abs, mr = s_out[0].max_rel;
      uint32_t ia = s_out[0].amax_abs, ir = s_out[0].amax_rel;
      double sa = s_out[0].sum_abs, sr = s_out[0].sum_rel;
      for (int w = 1; w < kWavesPerBlock; ++w) {
        eqb &= s_out[w].eq_bits;
        max_merge(ma, ia, s_out[w].max_abs, s_out[w].amax_abs);
        max_merge(mr, ir, s_out[w].max_rel, s_out[w].amax_rel);
        sa += s_out[w].sum_abs;
        sr += s_out[w].sum_rel;
      }
      rec->nfound = merged;
      rec->eq_bits = eqb;
      rec->amax_abs = ia;
      rec->amax_rel = ir;
      rec->pad = 0;
      rec->max_abs = ma;
      rec->max_rel = mr;
      rec->sum_abs = sa;
      rec->sum_rel = sr;
    }
  }

}

// ------------------------------------------------------------ finalize

// Tile blocks of the finalize launch (the blocks past the group blocks):
// copy the accumulated tile counts of the whole call to the tile-map output
// and clear the accumulators for the next call. Each thread moves
// kTileRun counts per round, all loaded before any is stored.
constexpr int kTileRun = 8;

__device__ __forceinline__ void publish_tiles(const Params &P) {
  uint32_t *__restrict__ acc = P.tile_maps;
  uint32_t *__restrict__ out = P.tile_out;
  const uint64_t n = P.tiles_total;
  const uint64_t nb = gridDim.x - P.n_groups, b = blockIdx.x - P.n_groups;
  constexpr uint64_t kPer = (uint64_t)kFinThreads * kTileRun;
  for (uint64_t base = b * kPer + threadIdx.x; base < n; base += nb * kPer) {
    uint32_t v[kTileRun];
#pragma unroll
    for (int q = 0; q < kTileRun; ++q) {
      const uint64_t i = base + (uint64_t)q * kFinThreads;
      v[q] = i < n ? acc[i] : 0u;
    }
#pragma unroll
    for (int q = 0; q < kTileRun; ++q) {
      const uint64_t i = base + (uint64_t)q * kFinThreads;
      if (i < n) {
        out[i] = v[q];
        acc[i] = 0;
      }
    }
  }
}

// One finalize launch, one block per chunk group of the call (a group is up
// to kGroupChunks consecutive chunks of one case). A case with one group is
// written directly from its chunk records. For a larger case each group
// block merges its chunks into a group record; the group block that arrives
// last (an acquire-release count per case) then merges the case's group
// records in group order and writes the results, so the merge order, and
// with it every output bit, does not depend on which block arrives last.
// The blocks past the group blocks publish the tile counts. Kernel
// boundaries order the chunk records and tile counts before this launch.
__global__ __launch_bounds__(kFinThreads) void finalize_kernel(const Params P) {
  __shared__ MergeScratch M;
  __shared__ uint32_t s_last;
  const uint64_t g = blockIdx.x;
  if (g >= P.n_groups) {
    publish_tiles(P);
    return;
  }
  const VCK_CONST DevCase *table = (const VCK_CONST DevCase *)P.cases;
  uint64_t ci = 0;
  DevCase cs;
  if (table != nullptr) {
    ci = P.group_case != nullptr ? (uint64_t)((const VCK_GLOBAL uint32_t *)P.group_case)[g] : g;
    cs = load_case(table + ci);
  } else {
    cs = P.single;
  }
  FinArgs F;
  F.stats = P.stats;
  F.mismatches = P.mismatches;
  F.pass_out = P.pass_out;
  F.first_k = P.first_k;
  F.integ = P.integ;
  F.match_rate = P.match_rate;
  F.numeric_rate = P.numeric_rate;
  F.ctr = P.ctr;
  F.n_cases = P.n_cases;
  F.n_tols = P.n_tols;
  F.primary = P.primary;
  F.k = P.k;
  F.do_integ = P.do_integ;
  const uint64_t CH = 4ull * cs.unit_elems;
  const uint32_t k = P.k > 0 ? (uint32_t)P.k : 0u;
  const uint64_t cstride = k;
  const uint32_t g_local = (uint32_t)(g - cs.group_begin);
  if (cs.n_groups == 1) {
    finalize_case(M, F, cs, P.recs + cs.chunk_begin, cs.n_chunks, CH,
                  P.stage + cs.chunk_begin * cstride, cstride);
    return;
  }
  const uint32_t gc0 = g_local * kGroupChunks;
  const uint32_t gchunks = min((uint32_t)kGroupChunks, cs.n_chunks - gc0);
  const ChunkRec *const grp = P.recs + cs.chunk_begin + gc0;
  merge_all<false>(M, grp, gchunks, CH, P.stage + (cs.chunk_begin + gc0) * cstride, cstride, k,
                   P.gstage + g * k, nullptr);
  const uint32_t gnf = M.nf_total;
  if (threadIdx.x == 0) {
    ChunkRec r;
#pragma unroll
    for (int q = 0; q < kRecCounts; ++q) ((uint32_t *)&r)[q] = (uint32_t)M.cnt[q];
    r.nfound = gnf;
    r.eq_bits = M.eq_all;
    r.amax_abs = M.amax_abs == UINT64_MAX ? kNone : (uint32_t)M.amax_abs;
    r.amax_rel = M.amax_rel == UINT64_MAX ? kNone : (uint32_t)M.amax_rel;
    r.pad = 0;
    r.max_abs = M.max_abs;
    r.max_rel = M.max_rel;
    r.sum_abs = M.sum_abs;
    r.sum_rel = M.sum_rel;
    P.grecs[g] = r;
  }
  // Publish the group record and first-k list (written by several waves):
  // each wave releases its own stores, then one count per group.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev =
        __hip_atomic_fetch_add(&P.gdone[ci], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = prev + 1 == cs.n_groups ? 1u : 0u;
  }
  __syncthreads();
  if (s_last == 0) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  if (threadIdx.x == 0) P.gdone[ci] = 0;  // (cleared for the next call)
  finalize_case(M, F, cs, P.grecs + cs.group_begin, cs.n_groups, CH * kGroupChunks,
                P.gstage + cs.group_begin * k, k);
}

// Copies the descriptor blob from pinned host memory, clears the counter
// area and the tile maps; writes zero rates for a sweep without cases.
__global__ __launch_bounds__(256) void prologue_kernel(const Prologue Q) {
  const uint64_t tid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t nth = (uint64_t)gridDim.x * blockDim.x;
  if (Q.blob_src != nullptr) {
    const u32x4 *src = (const u32x4 *)Q.blob_src;
    u32x4 *dst = (u32x4 *)Q.blob_dst;
    for (uint64_t i = tid; i < Q.blob_bytes / 16; i += nth) dst[i] = src[i];
  }
  for (uint64_t i = tid; i < Q.zero_words; i += nth) Q.zero[i] = 0;
  for (uint64_t i = tid; i < Q.n_tiles; i += nth) Q.tiles[i] = 0;
  if (Q.n_cases == 0 && tid < (uint64_t)Q.n_tols) {
    if (Q.match_rate != nullptr) Q.match_rate[tid] = 0.0;
    if (Q.numeric_rate != nullptr) Q.numeric_rate[tid] = 0.0;
  }
}

template <int DT, int NT, bool INTEG>
hipError_t launch_main_t(const Params &p, uint64_t n_chunks, hipStream_t s) {
  const size_t lds = (size_t)(kWavesPerBlock + 1) * (size_t)(p.k > 0 ? p.k : 0) * sizeof(uint32_t);
  hipLaunchKernelGGL((main_kernel<DT, NT, INTEG>), dim3((uint32_t)n_chunks), dim3(kBlockThreads),
                     lds, s, p);
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

hipError_t launch_prologue(const Prologue &p, hipStream_t s) {
  uint64_t work = p.blob_bytes / 16;
  if (p.zero_words > work) work = p.zero_words;
  if (p.n_tiles > work) work = p.n_tiles;
  uint64_t blocks = (work + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 2048) blocks = 2048;
  hipLaunchKernelGGL(prologue_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_finalize(const Params &p, hipStream_t s) {
  constexpr uint64_t kPer = (uint64_t)kFinThreads * kTileRun;
  uint64_t tile_blocks = 0;
  if (p.tile_out != nullptr && p.tile_maps != nullptr && p.tiles_total > 0)
    tile_blocks = min((p.tiles_total + kPer - 1) / kPer, (uint64_t)1024);
  const uint64_t blocks = p.n_groups + tile_blocks;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(finalize_kernel, dim3((uint32_t)blocks), dim3(kFinThreads), 0, s, p);
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

}  // namespace vck
