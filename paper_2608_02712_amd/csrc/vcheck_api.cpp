// vcheck_api.cpp -- host side of the C ABI declared in include/vcheck.h:
// argument validation (before anything is enqueued), work planning, workspace
// layout, descriptor upload and kernel launches.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "vcheck_internal.h"

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_prof_begin = nullptr, g_prof_end = nullptr;

vc_status fail(vc_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t elem_size(int32_t dtype) { return dtype == VC_F32 ? 4 : 2; }
bool dtype_ok(int32_t dtype) { return dtype == VC_F32 || dtype == VC_F16 || dtype == VC_BF16; }

// numel of a descriptor; -1 on an invalid shape or overflow past 2^62.
int64_t numel_of(const vc_tensor &t) {
  if (t.ndim < 0 || t.ndim > VC_MAX_NDIM) return -1;
  int64_t n = 1;
  for (int i = 0; i < t.ndim; ++i) {
    if (t.shape[i] < 0) return -1;
    if (t.shape[i] == 0) n = 0;
    else if (n != 0 && n > (int64_t(1) << 62) / t.shape[i]) return -1;
    else n *= t.shape[i];
  }
  return n;
}

// C of the (R, C) view: last dimension, 1 for a 0-d tensor.
uint64_t cols_of(const vc_tensor &t) { return t.ndim == 0 ? 1 : (uint64_t)t.shape[t.ndim - 1]; }

bool same_shape(const vc_tensor &a, const vc_tensor &b) {
  if (a.ndim != b.ndim) return false;
  for (int i = 0; i < a.ndim; ++i)
    if (a.shape[i] != b.shape[i]) return false;
  return true;
}

// Checks one descriptor on its own. Returns VC_OK or an error status.
// Status of a tensor descriptor without formatting a message (the per-case
// loop of a large sweep calls this; check_tensor formats on failure only).
vc_status tensor_status(const vc_tensor *t) {
  if (t == nullptr) return VC_ERR_NULL;
  if (!dtype_ok(t->dtype)) return VC_ERR_DTYPE;
  if (t->ndim < 0 || t->ndim > VC_MAX_NDIM) return VC_ERR_SHAPE;
  const int64_t n = numel_of(*t);
  if (n < 0) return VC_ERR_SHAPE;
  if (n > 0 && t->data == nullptr) return VC_ERR_NULL;
  if ((uintptr_t)t->data % elem_size(t->dtype) != 0) return VC_ERR_ALIGN;
  return VC_OK;
}

vc_status check_tensor(const vc_tensor *t, const char *what) {
  if (t == nullptr) return fail(VC_ERR_NULL, "%s descriptor is NULL", what);
  if (!dtype_ok(t->dtype)) return fail(VC_ERR_DTYPE, "%s has unknown dtype %d", what, t->dtype);
  if (t->ndim < 0 || t->ndim > VC_MAX_NDIM)
    return fail(VC_ERR_SHAPE, "%s has ndim %d outside 0..%d", what, t->ndim, VC_MAX_NDIM);
  const int64_t n = numel_of(*t);
  if (n < 0) return fail(VC_ERR_SHAPE, "%s has a negative or too large shape", what);
  if (n > 0 && t->data == nullptr) return fail(VC_ERR_NULL, "%s data is NULL", what);
  if ((uintptr_t)t->data % elem_size(t->dtype) != 0)
    return fail(VC_ERR_ALIGN, "%s data is not aligned to its element size", what);
  return VC_OK;
}

vc_status check_tols(const vc_tol *tols, int32_t n_tols) {
  if (n_tols < 1 || n_tols > VC_MAX_TOLS)
    return fail(VC_ERR_LIMIT, "n_tols %d outside 1..%d", n_tols, VC_MAX_TOLS);
  if (tols == nullptr) return fail(VC_ERR_NULL, "tolerance array is NULL");
  for (int p = 0; p < n_tols; ++p) {
    const vc_tol &t = tols[p];
    if (!std::isfinite(t.atol) || !std::isfinite(t.rtol) || t.atol < 0 || t.rtol < 0)
      return fail(VC_ERR_TOL, "tolerance pair %d: atol and rtol must be finite and >= 0", p);
    if (t.equal_nan != 0 && t.equal_nan != 1)
      return fail(VC_ERR_TOL, "tolerance pair %d: equal_nan must be 0 or 1", p);
  }
  return VC_OK;
}

struct Group {
  int32_t dtype;
  uint64_t case_lo, case_hi;    // table range
  uint64_t chunk_lo, n_chunks;  // global chunk range
  uint32_t unit;
};

struct Plan {
  std::vector<vck::DevCase> table;
  std::vector<uint64_t> case_chunk;  // chunk_begin per table entry
  std::vector<uint64_t> case_group;  // group_begin per table entry
  std::vector<uint32_t> multi;       // table indices of cases with more than one group
  std::vector<Group> groups;
  uint64_t total_chunks = 0;
  uint64_t total_groups = 0;
  uint64_t tiles_total = 0;
  int32_t n_cases = 0, n_tols = 1, nt_class = 1, k = 0, primary = 0, tile_h = 1, tile_w = 1;
  bool do_tiles = false, do_firstk = false, do_integ = false;
  // workspace layout: [table | case_chunk | case_group | multi] (the blob
  // the prologue copies), chunk records, chunk first-k lists, group records,
  // group first-k lists, then the Counters the prologue clears
  size_t off_table = 0, off_cc = 0, off_cg = 0, off_multi = 0, blob_bytes = 0;
  size_t off_recs = 0, off_stage = 0, off_grecs = 0, off_gstage = 0;
  size_t off_ctr = 0, ctr_bytes = 0;
  size_t bytes = 0;
};

// Elements per wave (a chunk is four of them): about 16K waves over the
// group, between 1 Ki elements and 64 KiB of each tensor per wave, a power of
// two (so every step is 16-byte aligned). Many short chunks keep every CU
// streaming until the end of the launch; longer ones amortize the per-block
// setup and the running-maximum records.
#ifndef VCK_WAVE_TARGET
#define VCK_WAVE_TARGET 16384
#endif
// How the four waves of a block share its chunk: with 16-bit storage each
// wave streams one contiguous quarter, so that the steps of a faulty tile
// (the same columns of consecutive rows) spread over the four waves; with
// binary32 storage (rows of 4 KiB and more, where a tile's rows already fall
// on several waves) they take steps round robin, which streams a little
// faster there.
#ifndef VCK_SPLIT
#define VCK_SPLIT 2
#endif
uint32_t split_for(int32_t dtype) {
  if (VCK_SPLIT == 2) return dtype == VC_F32 ? 0u : 1u;
  if (VCK_SPLIT == 3) return 2u;
  if (VCK_SPLIT == 4) return dtype == VC_F32 ? 0u : 2u;
  return (uint32_t)VCK_SPLIT;
}

uint32_t unit_for(uint64_t group_elems, int32_t dtype) {
  const uint64_t lo = 1024, hi = 65536 / elem_size(dtype);
  uint64_t u = lo;
  while (u < hi && u * 2 * VCK_WAVE_TARGET <= group_elems) u *= 2;
  return (uint32_t)u;
}

// Builds the plan. `single` requests the API-error behaviour of the
// single-case entry points for dtype/shape mismatches.
vc_status make_plan(const vc_case *cases, int32_t n_cases, const vc_tol *tols, int32_t n_tols,
                    const vc_sweep_opts &opts, bool want_tiles, bool want_firstk, bool single,
                    Plan &plan) {
  if (n_cases < 0 || n_cases > (1 << 24))
    return fail(VC_ERR_LIMIT, "n_cases %d outside 0..2^24", n_cases);
  if (n_cases > 0 && cases == nullptr) return fail(VC_ERR_NULL, "case array is NULL");
  {
    const vc_status st = check_tols(tols, n_tols);
    if (st != VC_OK) return st;
  }
  if (opts.primary_tol < 0 || opts.primary_tol >= n_tols)
    return fail(VC_ERR_TOL, "primary_tol %d outside 0..%d", opts.primary_tol, n_tols - 1);
  if (want_tiles && (opts.tile_h < 1 || opts.tile_w < 1))
    return fail(VC_ERR_TILE, "tile_h and tile_w must be >= 1 (got %d x %d)", opts.tile_h,
                opts.tile_w);
  if (opts.k < 0 || opts.k > VC_MAX_K) return fail(VC_ERR_K, "k %d outside 0..%d", opts.k, VC_MAX_K);
  if (opts.do_integrity != 0 && opts.do_integrity != 1)
    return fail(VC_ERR_LIMIT, "do_integrity must be 0 or 1");

  plan.n_cases = n_cases;
  plan.n_tols = n_tols;
  plan.nt_class = n_tols <= 1 ? 1 : n_tols <= 2 ? 2 : n_tols <= 4 ? 4 : 8;
  plan.primary = opts.primary_tol;
  plan.do_tiles = want_tiles;
  plan.do_firstk = want_firstk && opts.k > 0;
  plan.k = plan.do_firstk ? opts.k : 0;
  plan.tile_h = want_tiles ? opts.tile_h : 1;
  plan.tile_w = want_tiles ? opts.tile_w : 1;
  plan.do_integ = opts.do_integrity == 1;

  // per-case descriptors in caller order first
  std::vector<vck::DevCase> dc(n_cases);
  std::vector<uint64_t> tile_count(n_cases, 0);
  for (int32_t i = 0; i < n_cases; ++i) {
    const vc_case &c = cases[i];
    char what[64];
    // A malformed descriptor (NULL data, unknown dtype, bad shape) is an API
    // error. A misaligned pointer or a cand/ref dtype or shape difference is
    // a per-case outcome in a sweep and an API error for a single case.
    vc_status st = tensor_status(&c.cand);
    if (st != VC_OK) {
      snprintf(what, sizeof what, "case %d cand", i);
      st = check_tensor(&c.cand, what);
      if (st != VC_ERR_ALIGN) return st;
    }
    vc_status st_r = tensor_status(&c.ref);
    if (st_r != VC_OK) {
      snprintf(what, sizeof what, "case %d ref", i);
      st_r = check_tensor(&c.ref, what);
      if (st_r != VC_ERR_ALIGN) return st_r;
    }
    if (st == VC_OK) st = st_r;
    if (c.n_inputs < 0 || c.n_inputs > VC_MAX_INPUTS)
      return fail(VC_ERR_LIMIT, "case %d: n_inputs %d outside 0..%d", i, c.n_inputs,
                  VC_MAX_INPUTS);
    if (c.n_inputs > 0 && c.inputs == nullptr)
      return fail(VC_ERR_NULL, "case %d: inputs array is NULL", i);
    if (plan.do_integ) {
      for (int32_t j = 0; j < c.n_inputs; ++j) {
        if (tensor_status(&c.inputs[j]) == VC_OK) continue;
        snprintf(what, sizeof what, "case %d input %d", i, j);
        const vc_status sx = check_tensor(&c.inputs[j], what);
        if (sx != VC_ERR_ALIGN) return sx;
      }
    }
    if (st == VC_OK && c.cand.dtype != c.ref.dtype)
      st = fail(VC_ERR_DTYPE, "case %d: cand and ref dtypes differ", i);
    if (st == VC_OK && !same_shape(c.cand, c.ref))
      st = fail(VC_ERR_SHAPE, "case %d: cand and ref shapes differ", i);
    if (st != VC_OK && single) return st;

    vck::DevCase &d = dc[i];
    memset(&d, 0, sizeof d);
    d.orig = (uint32_t)i;
    d.dtype = (uint32_t)c.ref.dtype;
    const int64_t n = numel_of(c.ref);
    d.numel = (uint64_t)n;
    // every case, evaluated or not, owns vcheck_tile_count(ref) tile slots
    if (want_tiles && n > 0) {
      const uint64_t cols = cols_of(c.ref), rows = (uint64_t)n / cols;
      tile_count[i] = ((rows + opts.tile_h - 1) / opts.tile_h) *
                      ((cols + opts.tile_w - 1) / opts.tile_w);
    }
    if (st != VC_OK) {
      d.status = st;
      continue;
    }
    d.cand = (const uint8_t *)c.cand.data;
    d.ref = (const uint8_t *)c.ref.data;
    d.cols = cols_of(c.ref);
    bool vec = ((uintptr_t)c.cand.data % 16 == 0) && ((uintptr_t)c.ref.data % 16 == 0);
    if (plan.do_integ) {
      for (int32_t j = 0; j < c.n_inputs; ++j) {
        const vc_tensor &x = c.inputs[j];
        if (x.dtype == c.ref.dtype && numel_of(x) == n &&
            (uintptr_t)x.data % elem_size(x.dtype) == 0) {
          d.inp_mask |= 1u << j;
          d.inp[j] = (const uint8_t *)x.data;
          vec = vec && ((uintptr_t)x.data % 16 == 0);
        }
      }
    }
    d.vec_ok = vec ? 1u : 0u;
    if (want_tiles && n > 0) d.tiles_c = (d.cols + opts.tile_w - 1) / opts.tile_w;
    if (d.cols < (1ull << 31)) d.cols_div = vck::div_magic((uint32_t)d.cols);
  }
  // tile-map offsets follow the caller's case order
  if (want_tiles) {
    uint64_t acc = 0;
    for (int32_t i = 0; i < n_cases; ++i) {
      dc[i].tile_off = acc;
      acc += tile_count[i];
    }
    plan.tiles_total = acc;
  }
  // group by dtype (stable): F32, F16, BF16; chunks numbered in table order
  uint64_t chunk = 0, group = 0;
  for (int32_t dt : {VC_F32, VC_F16, VC_BF16}) {
    Group g{};
    g.dtype = dt;
    g.case_lo = plan.table.size();
    uint64_t elems = 0;
    for (int32_t i = 0; i < n_cases; ++i)
      if ((int32_t)dc[i].dtype == dt && dc[i].status == 0) elems += dc[i].numel;
    g.unit = unit_for(elems, dt);
    g.chunk_lo = chunk;
    for (int32_t i = 0; i < n_cases; ++i) {
      if ((int32_t)dc[i].dtype != dt) continue;
      vck::DevCase d = dc[i];
      d.unit_elems = g.unit;
      d.chunk_begin = chunk;
      d.group_begin = group;
      const uint64_t ch = 4ull * g.unit;
      // a case that is not evaluated, or is empty, still owns one (empty)
      // chunk: its results are written by the same completion path
      uint64_t nc = d.status == 0 ? (d.numel + ch - 1) / ch : 0;
      if (nc == 0) nc = 1;
      if (nc > 0xffffffffull) return fail(VC_ERR_LIMIT, "case %d is too large", (int)d.orig);
      d.n_chunks = (uint32_t)nc;
      d.n_groups = (uint32_t)((nc + vck::kGroupChunks - 1) / vck::kGroupChunks);
      chunk += nc;
      group += d.n_groups;
      plan.table.push_back(d);
      plan.case_chunk.push_back(d.chunk_begin);
      plan.case_group.push_back(d.group_begin);
      if (d.n_groups > 1) plan.multi.push_back((uint32_t)(plan.table.size() - 1));
    }
    g.case_hi = plan.table.size();
    g.n_chunks = chunk - g.chunk_lo;
    if (g.n_chunks > 0x7fffffffull)
      return fail(VC_ERR_LIMIT, "the cases of one dtype need more than 2^31 - 1 blocks");
    if (g.case_hi > g.case_lo) plan.groups.push_back(g);
  }
  plan.total_chunks = chunk;
  plan.total_groups = group;

  // workspace layout
  const size_t nc = (size_t)n_cases;
  size_t off = 0;
  plan.off_table = off;
  plan.off_cc = off + sizeof(vck::DevCase) * nc;  // 176 * n: 16-byte aligned
  plan.off_cg = plan.off_cc + sizeof(uint64_t) * nc;
  plan.off_multi = plan.off_cg + sizeof(uint64_t) * nc;
  plan.blob_bytes =
      (plan.off_multi - off + sizeof(uint32_t) * plan.multi.size() + 15) / 16 * 16;
  off += align_up(plan.blob_bytes);
  plan.off_recs = off;
  off += align_up(sizeof(vck::ChunkRec) * (size_t)plan.total_chunks);
  plan.off_stage = off;
  off += align_up(sizeof(uint32_t) * (size_t)plan.total_chunks * (size_t)plan.k);
  plan.off_grecs = off;
  off += align_up(sizeof(vck::ChunkRec) * (size_t)plan.total_groups);
  plan.off_gstage = off;
  off += align_up(sizeof(uint32_t) * (size_t)plan.total_groups * (size_t)plan.k);
  plan.off_ctr = off;
  plan.ctr_bytes = sizeof(vck::Counters);
  off += align_up(plan.ctr_bytes);
  plan.bytes = off + kAlign;  // slack for aligning the caller's base pointer
  return VC_OK;
}

// ---- pinned staging for descriptor uploads ---------------------------------
// A small ring of pinned host buffers per device. The prologue kernel reads
// the descriptor blob straight from the pinned buffer; a slot is reused only
// after the event recorded behind that kernel has completed.
struct Slot {
  void *host = nullptr;
  void *dev = nullptr;  // device-visible address of `host`
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};
struct DeviceStaging {
  std::mutex mu;
  Slot slots[8];
  int next = 0;
};
constexpr int kMaxDevices = 64;
DeviceStaging g_staging[kMaxDevices];

vc_status hip_check(hipError_t e, const char *what) {
  if (e == hipSuccess) return VC_OK;
  return fail(VC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Takes the next slot of the current device (waiting for its previous use)
// and fills it with `bytes` bytes of `src`. The caller holds `lock` until it
// has recorded the slot's event behind the kernel that reads it.
vc_status stage_blob(const void *src, size_t bytes, std::unique_lock<std::mutex> &lock,
                     Slot *&slot) {
  int dev = 0;
  vc_status st = hip_check(hipGetDevice(&dev), "hipGetDevice");
  if (st != VC_OK) return st;
  if (dev < 0 || dev >= kMaxDevices) return fail(VC_ERR_HIP, "device id %d out of range", dev);
  DeviceStaging &ds = g_staging[dev];
  lock = std::unique_lock<std::mutex>(ds.mu);
  Slot &sl = ds.slots[ds.next];
  ds.next = (ds.next + 1) % 8;
  if (sl.pending) {
    st = hip_check(hipEventSynchronize(sl.ev), "hipEventSynchronize");
    if (st != VC_OK) return st;
    sl.pending = false;
  }
  if (sl.ev == nullptr) {
    st = hip_check(hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming), "hipEventCreate");
    if (st != VC_OK) return st;
  }
  if (sl.cap < bytes) {
    if (sl.host != nullptr) (void)hipHostFree(sl.host);
    sl.host = sl.dev = nullptr;
    sl.cap = 0;
    const size_t cap = std::max<size_t>(bytes, 64 * 1024);
    st = hip_check(hipHostMalloc(&sl.host, cap, hipHostMallocDefault), "hipHostMalloc");
    if (st != VC_OK) return st;
    st = hip_check(hipHostGetDevicePointer(&sl.dev, sl.host, 0), "hipHostGetDevicePointer");
    if (st != VC_OK) {
      (void)hipHostFree(sl.host);
      sl.host = nullptr;
      return st;
    }
    sl.cap = cap;
  }
  memcpy(sl.host, src, bytes);
  slot = &sl;
  return VC_OK;
}

struct Outputs {
  vc_stats *stats = nullptr;
  uint64_t *mismatches = nullptr;
  uint8_t *pass = nullptr;
  double *match_rate = nullptr;
  double *numeric_rate = nullptr;
  uint32_t *tile_maps = nullptr;
  int64_t *first_k = nullptr;
  vc_integrity *integ = nullptr;
};

// Binary32 bounds of a binary64 value x >= 0: largest float <= x, smallest
// float >= x (FLT_MAX / +Inf beyond the binary32 range).
float f32_below(double x) {
  if (x >= (double)FLT_MAX) return FLT_MAX;
  float f = (float)x;
  if ((double)f > x) f = std::nextafter(f, 0.0f);
  return f;
}
float f32_above(double x) {
  if (x > (double)FLT_MAX) return INFINITY;
  float f = (float)x;
  if ((double)f < x) f = std::nextafter(f, INFINITY);
  return f;
}

// Enqueues the planned work. `single` passes the one descriptor by value
// (no table).
vc_status run(const Plan &plan, const vc_tol *tols, const Outputs &out, void *ws, size_t ws_bytes,
              hipStream_t stream, bool single) {
  if (ws == nullptr) return fail(VC_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < plan.bytes)
    return fail(VC_ERR_WORKSPACE, "workspace has %zu bytes, %zu required", ws_bytes, plan.bytes);
  uint8_t *base = (uint8_t *)(((uintptr_t)ws + kAlign - 1) / kAlign * kAlign);

  vck::Params P;
  memset(&P, 0, sizeof P);
  P.n_cases = plan.n_cases;
  P.n_tols = plan.n_tols;
  P.primary = plan.primary;
  P.tile_h = plan.tile_h;
  P.tile_w = plan.tile_w;
  P.th_div = vck::div_magic((uint32_t)plan.tile_h);
  P.tw_div = vck::div_magic((uint32_t)plan.tile_w);
  P.k = plan.k;
  P.do_tiles = plan.do_tiles ? 1 : 0;
  P.do_integ = plan.do_integ ? 1 : 0;
  for (int p = 0; p < VC_MAX_TOLS; ++p) {
    const vc_tol &t = tols[p < plan.n_tols ? p : plan.n_tols - 1];
    P.atol[p] = t.atol;
    P.rtol[p] = t.rtol;
    if (t.equal_nan) P.eqnan_mask |= 1u << p;
  }
  // The binary32 tier evaluates several pairs in binary64; a single pair
  // uses binary32 bounds shrunk / grown by 2^-20, valid while the thresholds
  // stay in the normal binary32 range: atol = 0 or >= 2^-100, rtol = 0 or
  // >= 2^-60 (the kernel requires |r| >= 2^-60 for this tier).
  P.tier1 = 1;
  if (plan.n_tols == 1) {
    const double a = tols[0].atol, r = tols[0].rtol;
    const bool a_ok = a == 0.0 || a >= 0x1p-100, r_ok = r == 0.0 || r >= 0x1p-60;
    P.tier1 = (a_ok && r_ok) ? 1 : 0;
    P.rlo = f32_below(r - r * 0x1p-20);
    P.alo = f32_below(a - a * 0x1p-20);
    P.rhi = f32_above(r + r * 0x1p-20);
    P.ahi = f32_above(a + a * 0x1p-20);
  }
  P.recs = (vck::ChunkRec *)(base + plan.off_recs);
  P.stage = (uint32_t *)(base + plan.off_stage);
  P.grecs = (vck::ChunkRec *)(base + plan.off_grecs);
  P.gstage = (uint32_t *)(base + plan.off_gstage);
  P.ctr = (vck::Counters *)(base + plan.off_ctr);
  P.tile_maps = plan.do_tiles ? out.tile_maps : nullptr;
  P.stats = out.stats;
  P.mismatches = out.mismatches;
  P.pass_out = out.pass;
  P.first_k = plan.do_firstk ? out.first_k : nullptr;
  P.integ = out.integ;
  P.match_rate = out.match_rate;
  P.numeric_rate = out.numeric_rate;

  vck::Prologue Q;
  memset(&Q, 0, sizeof Q);
  Q.zero = (uint32_t *)(base + plan.off_ctr);
  Q.zero_words = plan.ctr_bytes / sizeof(uint32_t);
  Q.tiles = P.tile_maps;
  Q.n_tiles = P.tile_maps != nullptr ? plan.tiles_total : 0;
  Q.match_rate = out.match_rate;
  Q.numeric_rate = out.numeric_rate;
  Q.n_cases = plan.n_cases;
  Q.n_tols = plan.n_tols;

  std::unique_lock<std::mutex> lock;
  Slot *slot = nullptr;
  std::vector<uint8_t> blob;
  if (single) {
    P.cases = nullptr;
    P.single = plan.table[0];
  } else if (plan.n_cases > 0) {
    P.cases = (const vck::DevCase *)(base + plan.off_table);
    P.case_chunk = (const uint64_t *)(base + plan.off_cc);
    P.case_group = (const uint64_t *)(base + plan.off_cg);
    P.multi = (const uint32_t *)(base + plan.off_multi);
    blob.assign(plan.blob_bytes, 0);
    memcpy(blob.data(), plan.table.data(), sizeof(vck::DevCase) * plan.table.size());
    memcpy(blob.data() + (plan.off_cc - plan.off_table), plan.case_chunk.data(),
           sizeof(uint64_t) * plan.case_chunk.size());
    memcpy(blob.data() + (plan.off_cg - plan.off_table), plan.case_group.data(),
           sizeof(uint64_t) * plan.case_group.size());
    if (!plan.multi.empty())
      memcpy(blob.data() + (plan.off_multi - plan.off_table), plan.multi.data(),
             sizeof(uint32_t) * plan.multi.size());
    const vc_status st = stage_blob(blob.data(), blob.size(), lock, slot);
    if (st != VC_OK) return st;
    Q.blob_src = (const uint8_t *)slot->dev;
    Q.blob_dst = base + plan.off_table;
    Q.blob_bytes = plan.blob_bytes;
  }
  // The launches of the call, back to back: no host work or event sits
  // between them, so the GPU never waits for the host inside a call.
  auto launch_all = [&]() -> vc_status {
    vc_status st = hip_check(vck::launch_prologue(Q, stream), "prologue launch");
    if (st != VC_OK) return st;
    hipEvent_t prof_begin = g_prof_begin, prof_end = g_prof_end;
    g_prof_begin = g_prof_end = nullptr;
    if (prof_begin != nullptr) {
      st = hip_check(hipEventRecord(prof_begin, stream), "profile begin event");
      if (st != VC_OK) return st;
    }
    for (const Group &g : plan.groups) {
      vck::Params G = P;
      G.chunk_lo = g.chunk_lo;
      G.case_lo = g.case_lo;
      G.case_hi = g.case_hi;
      G.unit_elems = g.unit;
      G.split = split_for(g.dtype);
      st = hip_check(vck::launch_main(g.dtype, plan.nt_class, plan.do_integ ? 1 : 0, G,
                                      g.n_chunks, stream),
                     "main kernel launch");
      if (st != VC_OK) return st;
    }
    if (prof_end != nullptr) {
      st = hip_check(hipEventRecord(prof_end, stream), "profile end event");
      if (st != VC_OK) return st;
    }
    const uint64_t n_multi = single ? (plan.table[0].n_groups > 1 ? 1 : 0) : plan.multi.size();
    return hip_check(vck::launch_finalize(P, plan.total_groups, n_multi, stream),
                     "finalize launch");
  };
  vc_status st = launch_all();
  if (slot != nullptr) {
    // The staging slot may be refilled once the prologue has read it; an
    // event behind the call's last kernel (recorded also after a failed
    // launch, in case the prologue was enqueued) guards that. The slot's
    // lock is held until then.
    const vc_status se = hip_check(hipEventRecord(slot->ev, stream), "hipEventRecord");
    if (se == VC_OK) slot->pending = true;
    if (st == VC_OK) st = se;
  }
  return st;
}

vc_case one_case(const vc_tensor *cand, const vc_tensor *ref, const vc_tensor *inputs,
                 int32_t n_inputs) {
  vc_case c;
  memset(&c, 0, sizeof c);
  c.cand = *cand;
  c.ref = *ref;
  c.inputs = inputs;
  c.n_inputs = n_inputs;
  return c;
}

vc_status check_pair(const vc_tensor *cand, const vc_tensor *ref) {
  vc_status st = check_tensor(cand, "cand");
  if (st != VC_OK) return st;
  st = check_tensor(ref, "ref");
  if (st != VC_OK) return st;
  if (cand->dtype != ref->dtype) return fail(VC_ERR_DTYPE, "cand and ref dtypes differ");
  if (!same_shape(*cand, *ref)) return fail(VC_ERR_SHAPE, "cand and ref shapes differ");
  return VC_OK;
}

// ---- tensor-statistics probe ---------------------------------------------

struct ProbePlan {
  std::vector<vck::ProbeTensor> tensors;
  std::vector<uint64_t> chunk_first, group_first;
  uint32_t unit = 1024;
  uint64_t total_chunks = 0, total_groups = 0;
  size_t off_recs = 0, off_grecs = 0, blob_bytes = 0, bytes = 0;
};

// Elements per wave of the probe: a power of two between 1 Ki and 8 Ki
// (8-bit histogram counters per lane), about 16K waves over the batch, and
// at least what keeps every tensor within 256 groups of 256 chunks.
uint32_t probe_unit(uint64_t total, uint64_t largest) {
  uint64_t u = 1024;
  while (u < 8192 && u * 2 * VCK_WAVE_TARGET <= total) u *= 2;
  while (u < 8192 && 4 * u * vck::kProbeGroupChunks * vck::kProbeGroupChunks < largest) u *= 2;
  return (uint32_t)u;
}

vc_status make_probe_plan(const vc_tensor *tensors, int32_t n, ProbePlan &plan) {
  if (n < 0 || n > (1 << 20)) return fail(VC_ERR_LIMIT, "n_tensors %d outside 0..2^20", n);
  if (n > 0 && tensors == nullptr) return fail(VC_ERR_NULL, "tensors is NULL");
  uint64_t total = 0, largest = 0;
  char what[48];
  for (int32_t i = 0; i < n; ++i) {
    if (tensor_status(&tensors[i]) != VC_OK) {
      snprintf(what, sizeof what, "tensor %d", i);
      return check_tensor(&tensors[i], what);
    }
    const uint64_t m = (uint64_t)numel_of(tensors[i]);
    if (m >= (1ull << 31)) return fail(VC_ERR_LIMIT, "tensor %d has 2^31 elements or more", i);
    total += m;
    largest = std::max(largest, m);
  }
  plan.unit = probe_unit(total, largest);
  const uint64_t ch = 4ull * plan.unit;
  plan.tensors.resize(n);
  plan.chunk_first.resize(n);
  plan.group_first.resize(n);
  for (int32_t i = 0; i < n; ++i) {
    vck::ProbeTensor &t = plan.tensors[i];
    t.data = (const uint8_t *)tensors[i].data;
    t.numel = (uint64_t)numel_of(tensors[i]);
    t.dtype = tensors[i].dtype;
    t.chunk_begin = plan.total_chunks;
    const uint64_t nc = std::max<uint64_t>(1, (t.numel + ch - 1) / ch);
    t.n_chunks = (uint32_t)nc;
    plan.chunk_first[i] = plan.total_chunks;
    plan.group_first[i] = plan.total_groups;
    plan.total_chunks += nc;
    plan.total_groups += (nc + vck::kProbeGroupChunks - 1) / vck::kProbeGroupChunks;
  }
  if (plan.total_chunks > 0x7fffffffull)
    return fail(VC_ERR_LIMIT, "the batch needs more than 2^31 - 1 blocks");
  plan.blob_bytes = (sizeof(vck::ProbeTensor) + 2 * sizeof(uint64_t)) * (size_t)n;
  size_t off = align_up(plan.blob_bytes);
  plan.off_recs = off;
  off += align_up(sizeof(vck::ProbeRec) * (size_t)plan.total_chunks);
  plan.off_grecs = off;
  off += align_up(sizeof(vck::ProbeRec) * (size_t)plan.total_groups);
  plan.bytes = off + kAlign;  // room to align the caller's pointer
  return VC_OK;
}

// Runs one diagnostic call: stages the descriptor blob (`parts`, copied
// back to back) in a pinned slot, enqueues the prologue (copying it to
// `base`, clearing `zero_words` words at `zero`) and then `launch` (which
// receives the profiling events), and records the slot's event behind them.
template <typename F>
vc_status run_diagnostic(const std::vector<std::pair<const void *, size_t>> &parts, uint8_t *base,
                         uint32_t *zero, uint64_t zero_words, hipStream_t stream,
                         const char *what, F launch) {
  size_t total = 0;
  for (const auto &p : parts) total += p.second;
  std::vector<uint8_t> blob(total);
  size_t at = 0;
  for (const auto &p : parts) {
    memcpy(blob.data() + at, p.first, p.second);
    at += p.second;
  }
  std::unique_lock<std::mutex> lock;
  Slot *slot = nullptr;
  vc_status st = stage_blob(blob.data(), blob.size(), lock, slot);
  if (st != VC_OK) return st;
  vck::Prologue Q;
  memset(&Q, 0, sizeof Q);
  Q.blob_src = (const uint8_t *)slot->dev;
  Q.blob_dst = base;
  Q.blob_bytes = total;
  Q.zero = zero;
  Q.zero_words = zero_words;
  Q.n_cases = 1;  // (no suite rates to clear)
  hipEvent_t prof_begin = g_prof_begin, prof_end = g_prof_end;
  g_prof_begin = g_prof_end = nullptr;
  st = hip_check(vck::launch_prologue(Q, stream), "prologue launch");
  if (st == VC_OK) st = hip_check(launch(prof_begin, prof_end), what);
  // the staging slot is reused once the prologue has read it
  const vc_status se = hip_check(hipEventRecord(slot->ev, stream), "hipEventRecord");
  if (se == VC_OK) slot->pending = true;
  return st != VC_OK ? st : se;
}

// ---- near-pass statistics -------------------------------------------------

struct NpPlan {
  std::vector<vck::NpCase> cases;
  std::vector<uint64_t> chunk_first, group_first;
  uint32_t unit = 1024;
  uint64_t total_chunks = 0, total_groups = 0;
  size_t off_recs = 0, off_grecs = 0, blob_bytes = 0, bytes = 0;
};

vc_status make_np_plan(const vc_case *cases, int32_t n, NpPlan &plan) {
  if (n < 0 || n > (1 << 20)) return fail(VC_ERR_LIMIT, "n_cases %d outside 0..2^20", n);
  if (n > 0 && cases == nullptr) return fail(VC_ERR_NULL, "cases is NULL");
  uint64_t total = 0, largest = 0;
  char what[48];
  for (int32_t i = 0; i < n; ++i) {
    const vc_case &c = cases[i];
    if (tensor_status(&c.cand) != VC_OK) {
      snprintf(what, sizeof what, "case %d cand", i);
      return check_tensor(&c.cand, what);
    }
    if (tensor_status(&c.ref) != VC_OK) {
      snprintf(what, sizeof what, "case %d ref", i);
      return check_tensor(&c.ref, what);
    }
    if (c.cand.dtype != c.ref.dtype)
      return fail(VC_ERR_DTYPE, "case %d: cand and ref dtypes differ", i);
    if (!same_shape(c.cand, c.ref))
      return fail(VC_ERR_SHAPE, "case %d: cand and ref shapes differ", i);
    const uint64_t m = (uint64_t)numel_of(c.ref);
    if (m >= (1ull << 31)) return fail(VC_ERR_LIMIT, "case %d has 2^31 elements or more", i);
    total += m;
    largest = std::max(largest, m);
  }
  plan.unit = probe_unit(total, largest);
  const uint64_t ch = 4ull * plan.unit;
  plan.cases.resize(n);
  plan.chunk_first.resize(n);
  plan.group_first.resize(n);
  for (int32_t i = 0; i < n; ++i) {
    vck::NpCase &d = plan.cases[i];
    memset(&d, 0, sizeof d);
    d.cand = (const uint8_t *)cases[i].cand.data;
    d.ref = (const uint8_t *)cases[i].ref.data;
    d.numel = (uint64_t)numel_of(cases[i].ref);
    d.dtype = cases[i].ref.dtype;
    d.chunk_begin = plan.total_chunks;
    const uint64_t nc = std::max<uint64_t>(1, (d.numel + ch - 1) / ch);
    d.n_chunks = (uint32_t)nc;
    plan.chunk_first[i] = plan.total_chunks;
    plan.group_first[i] = plan.total_groups;
    plan.total_chunks += nc;
    plan.total_groups += (nc + vck::kProbeGroupChunks - 1) / vck::kProbeGroupChunks;
  }
  if (plan.total_chunks > 0x7fffffffull)
    return fail(VC_ERR_LIMIT, "the batch needs more than 2^31 - 1 blocks");
  plan.blob_bytes = (sizeof(vck::NpCase) + 2 * sizeof(uint64_t)) * (size_t)n;
  size_t off = align_up(plan.blob_bytes);
  plan.off_recs = off;
  off += align_up(sizeof(vck::NpRec) * (size_t)plan.total_chunks);
  plan.off_grecs = off;
  off += align_up(sizeof(vck::NpRec) * (size_t)plan.total_groups);
  plan.bytes = off + kAlign;
  return VC_OK;
}

}  // namespace

extern "C" {

vc_status vcheck_compare(const vc_tensor *cand, const vc_tensor *ref, const vc_tol *tol,
                         vc_stats *out, void *ws, size_t ws_bytes, void *stream) {
  g_last_error.clear();
  vc_status st = check_pair(cand, ref);
  if (st != VC_OK) return st;
  if (tol == nullptr) return fail(VC_ERR_NULL, "tolerance is NULL");
  if (out == nullptr) return fail(VC_ERR_NULL, "output stats pointer is NULL");
  const vc_case c = one_case(cand, ref, nullptr, 0);
  vc_sweep_opts opts{};
  Plan plan;
  st = make_plan(&c, 1, tol, 1, opts, false, false, true, plan);
  if (st != VC_OK) return st;
  Outputs o;
  o.stats = out;
  return run(plan, tol, o, ws, ws_bytes, (hipStream_t)stream, true);
}

vc_status vcheck_localize(const vc_tensor *cand, const vc_tensor *ref, const vc_tol *tol,
                          int32_t tile_h, int32_t tile_w, uint32_t *tile_map, int32_t k,
                          int64_t *first_k, vc_stats *out, void *ws, size_t ws_bytes,
                          void *stream) {
  g_last_error.clear();
  vc_status st = check_pair(cand, ref);
  if (st != VC_OK) return st;
  if (tol == nullptr) return fail(VC_ERR_NULL, "tolerance is NULL");
  if (tile_h < 1 || tile_w < 1)
    return fail(VC_ERR_TILE, "tile_h and tile_w must be >= 1 (got %d x %d)", tile_h, tile_w);
  if (k < 0 || k > VC_MAX_K) return fail(VC_ERR_K, "k %d outside 0..%d", k, VC_MAX_K);
  if (k > 0 && first_k == nullptr) return fail(VC_ERR_K, "first_k is NULL with k = %d", k);
  const int64_t tiles = vcheck_tile_count(cand, tile_h, tile_w);
  if (tiles > 0 && tile_map == nullptr) return fail(VC_ERR_NULL, "tile_map is NULL");
  const vc_case c = one_case(cand, ref, nullptr, 0);
  vc_sweep_opts opts{};
  opts.tile_h = tile_h;
  opts.tile_w = tile_w;
  opts.k = k;
  Plan plan;
  st = make_plan(&c, 1, tol, 1, opts, true, true, true, plan);
  if (st != VC_OK) return st;
  Outputs o;
  o.stats = out;
  o.tile_maps = tile_map;
  o.first_k = first_k;
  return run(plan, tol, o, ws, ws_bytes, (hipStream_t)stream, true);
}

vc_status vcheck_integrity(const vc_tensor *cand, const vc_tensor *ref, const vc_tensor *inputs,
                           int32_t n_inputs, const vc_tol *tol, vc_integrity *out,
                           vc_stats *stats, void *ws, size_t ws_bytes, void *stream) {
  g_last_error.clear();
  vc_status st = check_pair(cand, ref);
  if (st != VC_OK) return st;
  if (tol == nullptr) return fail(VC_ERR_NULL, "tolerance is NULL");
  if (out == nullptr) return fail(VC_ERR_NULL, "output integrity pointer is NULL");
  if (n_inputs < 0 || n_inputs > VC_MAX_INPUTS)
    return fail(VC_ERR_LIMIT, "n_inputs %d outside 0..%d", n_inputs, VC_MAX_INPUTS);
  if (n_inputs > 0 && inputs == nullptr) return fail(VC_ERR_NULL, "inputs array is NULL");
  const vc_case c = one_case(cand, ref, inputs, n_inputs);
  vc_sweep_opts opts{};
  opts.do_integrity = 1;
  Plan plan;
  st = make_plan(&c, 1, tol, 1, opts, false, false, true, plan);
  if (st != VC_OK) return st;
  Outputs o;
  o.stats = stats;
  o.integ = out;
  return run(plan, tol, o, ws, ws_bytes, (hipStream_t)stream, true);
}

vc_status vcheck_sweep(const vc_case *cases, int32_t n_cases, const vc_tol *tols, int32_t n_tols,
                       const vc_sweep_opts *opts, const vc_sweep_out *out, void *ws,
                       size_t ws_bytes, void *stream) {
  g_last_error.clear();
  if (out == nullptr) return fail(VC_ERR_NULL, "output descriptor is NULL");
  if (out->stats == nullptr && n_cases > 0) return fail(VC_ERR_NULL, "out->stats is NULL");
  vc_sweep_opts o{};
  if (opts != nullptr) o = *opts;
  if (o.do_integrity == 1 && out->integ == nullptr && n_cases > 0)
    return fail(VC_ERR_NULL, "do_integrity is set but out->integ is NULL");
  const bool want_tiles = out->tile_maps != nullptr;
  const bool want_firstk = out->first_k != nullptr;
  if (o.k > 0 && !want_firstk) o.k = 0;
  Plan plan;
  vc_status st = make_plan(cases, n_cases, tols, n_tols, o, want_tiles, want_firstk, false, plan);
  if (st != VC_OK) return st;
  Outputs oo;
  oo.stats = out->stats;
  oo.mismatches = out->mismatches;
  oo.pass = out->pass;
  oo.match_rate = out->match_rate;
  oo.numeric_rate = out->numeric_rate;
  oo.tile_maps = out->tile_maps;
  oo.first_k = out->first_k;
  oo.integ = out->integ;
  return run(plan, tols, oo, ws, ws_bytes, (hipStream_t)stream, false);
}

vc_status vcheck_workspace_bytes(const vc_case *cases, int32_t n_cases, int32_t n_tols,
                                 const vc_sweep_opts *opts, size_t *bytes) {
  g_last_error.clear();
  if (bytes == nullptr) return fail(VC_ERR_NULL, "bytes is NULL");
  vc_sweep_opts o{};
  if (opts != nullptr) o = *opts;
  if (n_tols < 1 || n_tols > VC_MAX_TOLS)
    return fail(VC_ERR_LIMIT, "n_tols %d outside 1..%d", n_tols, VC_MAX_TOLS);
  // sizing does not depend on tolerance values or tile geometry
  vc_tol dummy[VC_MAX_TOLS];
  for (auto &t : dummy) t = vc_tol{0.0, 0.0, 0, 0};
  o.tile_h = o.tile_h < 1 ? 1 : o.tile_h;
  o.tile_w = o.tile_w < 1 ? 1 : o.tile_w;
  if (o.primary_tol < 0 || o.primary_tol >= n_tols) o.primary_tol = 0;
  Plan plan;
  const vc_status st = make_plan(cases, n_cases, dummy, n_tols, o, false, o.k > 0, false, plan);
  if (st != VC_OK) return st;
  *bytes = plan.bytes;
  return VC_OK;
}

int64_t vcheck_tile_count(const vc_tensor *t, int32_t tile_h, int32_t tile_w) {
  if (t == nullptr || tile_h < 1 || tile_w < 1) return -1;
  const int64_t n = numel_of(*t);
  if (n < 0) return -1;
  if (n == 0) return 0;
  const uint64_t cols = cols_of(*t);
  const uint64_t rows = (uint64_t)n / cols;
  return (int64_t)(((rows + tile_h - 1) / tile_h) * ((cols + tile_w - 1) / tile_w));
}

const char *vcheck_status_str(vc_status status) {
  switch (status) {
    case VC_OK: return "ok";
    case VC_ERR_NULL: return "a required pointer is NULL";
    case VC_ERR_DTYPE: return "unknown dtype or cand/ref dtypes differ";
    case VC_ERR_SHAPE: return "bad shape or cand/ref shapes differ";
    case VC_ERR_TOL: return "invalid tolerance";
    case VC_ERR_TILE: return "invalid tile size";
    case VC_ERR_K: return "invalid first-k length";
    case VC_ERR_WORKSPACE: return "workspace missing or too small";
    case VC_ERR_LIMIT: return "a count is outside its supported range";
    case VC_ERR_HIP: return "HIP runtime error";
    case VC_ERR_ALIGN: return "data pointer not aligned to its element size";
    default: return "unknown status";
  }
}

const char *vcheck_last_error(void) { return g_last_error.c_str(); }

int32_t vcheck_abi_version(void) { return VCHECK_ABI_VERSION; }

vc_status vcheck_profile_events(void *begin_event, void *end_event) {
  g_last_error.clear();
  if ((begin_event == nullptr) != (end_event == nullptr))
    return fail(VC_ERR_NULL, "profile events must both be set or both be NULL");
  g_prof_begin = (hipEvent_t)begin_event;
  g_prof_end = (hipEvent_t)end_event;
  return VC_OK;
}

}  // extern "C"

vc_status vcheck_tensor_stats_workspace(const vc_tensor *tensors, int32_t n_tensors,
                                        size_t *bytes) {
  g_last_error.clear();
  if (bytes == nullptr) return fail(VC_ERR_NULL, "bytes is NULL");
  ProbePlan plan;
  const vc_status st = make_probe_plan(tensors, n_tensors, plan);
  if (st != VC_OK) return st;
  *bytes = plan.bytes;
  return VC_OK;
}

vc_status vcheck_tensor_stats(const vc_tensor *tensors, int32_t n_tensors, vc_tstats *out,
                              void *ws, size_t ws_bytes, void *stream_) {
  g_last_error.clear();
  ProbePlan plan;
  vc_status st = make_probe_plan(tensors, n_tensors, plan);
  if (st != VC_OK) return st;
  if (n_tensors == 0) return VC_OK;
  if (out == nullptr) return fail(VC_ERR_NULL, "out is NULL");
  if (ws == nullptr) return fail(VC_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < plan.bytes)
    return fail(VC_ERR_WORKSPACE, "workspace has %zu bytes, %zu required", ws_bytes, plan.bytes);
  uint8_t *base = (uint8_t *)(((uintptr_t)ws + kAlign - 1) / kAlign * kAlign);
  const size_t n = (size_t)n_tensors;
  vck::ProbeParams P;
  memset(&P, 0, sizeof P);
  P.tensors = (const vck::ProbeTensor *)base;
  P.chunk_first = (const uint64_t *)(base + sizeof(vck::ProbeTensor) * n);
  P.group_first = (const uint64_t *)(base + (sizeof(vck::ProbeTensor) + 8) * n);
  P.n_tensors = n_tensors;
  P.unit = plan.unit;
  P.recs = (vck::ProbeRec *)(base + plan.off_recs);
  P.grecs = (vck::ProbeRec *)(base + plan.off_grecs);
  P.out = out;
  const hipStream_t stream = (hipStream_t)stream_;
  return run_diagnostic({{plan.tensors.data(), sizeof(vck::ProbeTensor) * n},
                         {plan.chunk_first.data(), 8 * n},
                         {plan.group_first.data(), 8 * n}},
                        base, nullptr, 0, stream, "probe launch",
                        [&](hipEvent_t b, hipEvent_t e) {
                          return vck::launch_probe(P, plan.total_chunks, plan.total_groups,
                                                   stream, b, e);
                        });
}

vc_status vcheck_nearpass_workspace(const vc_case *cases, int32_t n_cases, size_t *bytes) {
  g_last_error.clear();
  if (bytes == nullptr) return fail(VC_ERR_NULL, "bytes is NULL");
  NpPlan plan;
  const vc_status st = make_np_plan(cases, n_cases, plan);
  if (st != VC_OK) return st;
  *bytes = plan.bytes;
  return VC_OK;
}

vc_status vcheck_nearpass(const vc_case *cases, int32_t n_cases, const vc_tol *tol,
                          vc_nearpass *out, void *ws, size_t ws_bytes, void *stream_) {
  g_last_error.clear();
  NpPlan plan;
  vc_status st = make_np_plan(cases, n_cases, plan);
  if (st != VC_OK) return st;
  st = check_tols(tol, 1);
  if (st != VC_OK) return st;
  if (n_cases == 0) return VC_OK;
  if (out == nullptr) return fail(VC_ERR_NULL, "out is NULL");
  if (ws == nullptr) return fail(VC_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < plan.bytes)
    return fail(VC_ERR_WORKSPACE, "workspace has %zu bytes, %zu required", ws_bytes, plan.bytes);
  uint8_t *base = (uint8_t *)(((uintptr_t)ws + kAlign - 1) / kAlign * kAlign);
  const size_t n = (size_t)n_cases;
  vck::NpParams P;
  memset(&P, 0, sizeof P);
  P.cases = (const vck::NpCase *)base;
  P.chunk_first = (const uint64_t *)(base + sizeof(vck::NpCase) * n);
  P.group_first = (const uint64_t *)(base + (sizeof(vck::NpCase) + 8) * n);
  P.n_cases = n_cases;
  P.unit = plan.unit;
  P.atol = tol->atol;
  P.rtol = tol->rtol;
  P.recs = (vck::NpRec *)(base + plan.off_recs);
  P.grecs = (vck::NpRec *)(base + plan.off_grecs);
  P.out = out;
  const hipStream_t stream = (hipStream_t)stream_;
  return run_diagnostic({{plan.cases.data(), sizeof(vck::NpCase) * n},
                         {plan.chunk_first.data(), 8 * n},
                         {plan.group_first.data(), 8 * n}},
                        base, nullptr, 0, stream, "near-pass launch",
                        [&](hipEvent_t b, hipEvent_t e) {
                          return vck::launch_nearpass(P, plan.total_chunks, plan.total_groups,
                                                      stream, b, e);
                        });
}

vc_status vcheck_content_hash_workspace(const vc_tensor *tensors, int32_t n_tensors,
                                        size_t *bytes) {
  g_last_error.clear();
  if (bytes == nullptr) return fail(VC_ERR_NULL, "bytes is NULL");
  ProbePlan plan;
  const vc_status st = make_probe_plan(tensors, n_tensors, plan);
  if (st != VC_OK) return st;
  *bytes = align_up(plan.blob_bytes) + kAlign;  // the tensor table only
  return VC_OK;
}

vc_status vcheck_content_hash(const vc_tensor *tensors, int32_t n_tensors, uint64_t *out,
                              void *ws, size_t ws_bytes, void *stream_) {
  g_last_error.clear();
  ProbePlan plan;
  vc_status st = make_probe_plan(tensors, n_tensors, plan);
  if (st != VC_OK) return st;
  if (n_tensors == 0) return VC_OK;
  if (out == nullptr) return fail(VC_ERR_NULL, "out is NULL");
  const size_t need = align_up(plan.blob_bytes) + kAlign;
  if (ws == nullptr) return fail(VC_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < need)
    return fail(VC_ERR_WORKSPACE, "workspace has %zu bytes, %zu required", ws_bytes, need);
  uint8_t *base = (uint8_t *)(((uintptr_t)ws + kAlign - 1) / kAlign * kAlign);
  const size_t n = (size_t)n_tensors;
  vck::HashParams P;
  memset(&P, 0, sizeof P);
  P.tensors = (const vck::ProbeTensor *)base;
  P.chunk_first = (const uint64_t *)(base + sizeof(vck::ProbeTensor) * n);
  P.n_tensors = n_tensors;
  P.unit = plan.unit;
  P.out = (unsigned long long *)out;
  const hipStream_t stream = (hipStream_t)stream_;
  // the prologue clears the sums
  return run_diagnostic({{plan.tensors.data(), sizeof(vck::ProbeTensor) * n},
                         {plan.chunk_first.data(), 8 * n},
                         {plan.group_first.data(), 8 * n}},
                        base, (uint32_t *)out, 2 * n, stream, "hash launch",
                        [&](hipEvent_t b, hipEvent_t e) {
                          return vck::launch_hash(P, plan.total_chunks, stream, b, e);
                        });
}
