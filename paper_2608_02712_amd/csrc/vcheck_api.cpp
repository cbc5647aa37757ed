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
  std::vector<uint32_t> group_case;  // table index per chunk group (empty: group = table index)
  std::vector<Group> groups;
  uint64_t total_chunks = 0;
  uint64_t total_groups = 0;
  uint64_t tiles_total = 0;
  int32_t n_cases = 0, n_tols = 1, nt_class = 1, k = 0, primary = 0, tile_h = 1, tile_w = 1;
  bool do_tiles = false, do_firstk = false, do_integ = false;
  // Workspace layout (each part 256-byte aligned): the descriptor blob
  // [table | case_chunk | group_case], chunk records, chunk first-k lists,
  // group records, group first-k lists, then the parts that are zero on
  // entry: the Counters, the per-case merged-group counts and the tile-count
  // accumulators.
  size_t off_table = 0, off_cc = 0, off_gc = 0, blob_bytes = 0;
  size_t off_recs = 0, off_stage = 0, off_grecs = 0, off_gstage = 0;
  size_t off_zero = 0, zero_bytes = 0, off_ctr = 0, off_gdone = 0, off_tacc = 0;
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

static_assert(4 * (65536 / 2) <= vck::kMaxChunkElems, "chunk size bound of the merge");
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
    d.n_tiles = tile_count[i];
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
  bool multi = false;
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
      if (d.n_groups > 1) multi = true;
      chunk += nc;
      group += d.n_groups;
      plan.table.push_back(d);
      plan.case_chunk.push_back(d.chunk_begin);
    }
    g.case_hi = plan.table.size();
    g.n_chunks = chunk - g.chunk_lo;
    if (g.n_chunks > 0x7fffffffull)
      return fail(VC_ERR_LIMIT, "the cases of one dtype need more than 2^31 - 1 blocks");
    if (g.case_hi > g.case_lo) plan.groups.push_back(g);
  }
  plan.total_chunks = chunk;
  plan.total_groups = group;
  if (group > 0x7fffffffull) return fail(VC_ERR_LIMIT, "the sweep needs more than 2^31 - 1 groups");
  // group -> table index, needed only when some case has several groups
  if (multi) {
    plan.group_case.reserve(group);
    for (size_t t = 0; t < plan.table.size(); ++t)
      for (uint32_t q = 0; q < plan.table[t].n_groups; ++q) plan.group_case.push_back((uint32_t)t);
  }

  // workspace layout
  const size_t nc = (size_t)n_cases;
  plan.off_table = 0;
  plan.off_cc = sizeof(vck::DevCase) * nc;  // 176 * n: 16-byte aligned
  plan.off_gc = plan.off_cc + sizeof(uint64_t) * nc;
  plan.blob_bytes = (plan.off_gc + sizeof(uint32_t) * plan.group_case.size() + 15) / 16 * 16;
  size_t off = align_up(plan.blob_bytes);
  plan.off_recs = off;
  off += align_up(sizeof(vck::ChunkRec) * (size_t)plan.total_chunks);
  plan.off_stage = off;
  off += align_up(sizeof(uint32_t) * (size_t)plan.total_chunks * (size_t)plan.k);
  plan.off_grecs = off;
  off += align_up(sizeof(vck::ChunkRec) * (size_t)plan.total_groups);
  plan.off_gstage = off;
  off += align_up(sizeof(uint32_t) * (size_t)plan.total_groups * (size_t)plan.k);
  plan.off_zero = off;
  plan.off_ctr = off;
  off += align_up(sizeof(vck::Counters));
  plan.off_gdone = off;
  off += align_up(sizeof(uint32_t) * std::max<size_t>(nc, 1));
  plan.off_tacc = off;
  off += align_up(sizeof(uint32_t) * (size_t)(want_tiles ? plan.tiles_total : 0));
  plan.zero_bytes = off - plan.off_zero;
  plan.bytes = off + kAlign;  // slack for aligning the caller's base pointer
  return VC_OK;
}

// The descriptor blob of a plan, as it is laid out at the workspace base.
std::vector<uint8_t> plan_blob(const Plan &plan) {
  std::vector<uint8_t> blob(plan.blob_bytes, 0);
  if (!plan.table.empty())
    memcpy(blob.data() + plan.off_table, plan.table.data(),
           sizeof(vck::DevCase) * plan.table.size());
  if (!plan.case_chunk.empty())
    memcpy(blob.data() + plan.off_cc, plan.case_chunk.data(),
           sizeof(uint64_t) * plan.case_chunk.size());
  if (!plan.group_case.empty())
    memcpy(blob.data() + plan.off_gc, plan.group_case.data(),
           sizeof(uint32_t) * plan.group_case.size());
  return blob;
}

vc_status hip_check(hipError_t e, const char *what) {
  if (e == hipSuccess) return VC_OK;
  return fail(VC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---- per-device state --------------------------------------------------------
// Per device the library keeps, allocated once and held until the process
// ends: a ring of kSlots pinned host buffers of kSlotBytes each, from which
// the prologue kernel of a one-shot call copies the call's descriptor blob
// (a slot is reused only after the event recorded behind the kernels that
// read it has completed), and the device address of the allocation-free
// entry point's scratch array. A blob larger than a slot is uploaded with a
// pageable hipMemcpyAsync instead, which returns only once the runtime has
// taken the bytes (waiting for the stream's earlier work).
constexpr int kSlots = 8;
constexpr size_t kSlotBytes = 256 * 1024;
constexpr int kMaxDevices = 64;

struct DeviceState {
  std::mutex mu;
  bool ring = false;  // the slots are allocated
  void *host[kSlots] = {};
  void *dev[kSlots] = {};  // device-visible addresses of host[]
  hipEvent_t ev[kSlots] = {};
  bool pending[kSlots] = {};
  int next = 0;
  uint8_t *scratch = nullptr;  // device address of the scratch array (vcheck_init)
};
DeviceState g_dev[kMaxDevices];

vc_status current_device(int &dev) {
  vc_status st = hip_check(hipGetDevice(&dev), "hipGetDevice");
  if (st != VC_OK) return st;
  if (dev < 0 || dev >= kMaxDevices) return fail(VC_ERR_HIP, "device id %d out of range", dev);
  return VC_OK;
}

// Allocates the staging ring of a device once (caller holds ds.mu).
vc_status ensure_ring(DeviceState &ds) {
  if (ds.ring) return VC_OK;
  for (int i = 0; i < kSlots; ++i) {
    vc_status st = hip_check(hipHostMalloc(&ds.host[i], kSlotBytes, hipHostMallocDefault),
                             "hipHostMalloc");
    if (st == VC_OK)
      st = hip_check(hipHostGetDevicePointer(&ds.dev[i], ds.host[i], 0), "hipHostGetDevicePointer");
    if (st == VC_OK)
      st = hip_check(hipEventCreateWithFlags(&ds.ev[i], hipEventDisableTiming), "hipEventCreate");
    if (st != VC_OK) return st;  // (partial allocations are kept for the next attempt)
  }
  ds.ring = true;
  return VC_OK;
}

// Takes the next slot of the current device (waiting for its previous use
// to complete) and fills it with `bytes` (<= kSlotBytes) bytes of `src`. The
// caller holds `lock` until it has recorded ev[slot] behind the kernels that
// read the slot. `allocate` = false: the ring must already exist.
vc_status stage_blob(const void *src, size_t bytes, bool allocate,
                     std::unique_lock<std::mutex> &lock, DeviceState *&dsp, int &slot) {
  int dev = 0;
  vc_status st = current_device(dev);
  if (st != VC_OK) return st;
  DeviceState &ds = g_dev[dev];
  lock = std::unique_lock<std::mutex>(ds.mu);
  if (!ds.ring) {
    if (!allocate) return fail(VC_ERR_STATE, "vcheck_init has not run on device %d", dev);
    st = ensure_ring(ds);
    if (st != VC_OK) return st;
  }
  const int i = ds.next;
  ds.next = (ds.next + 1) % kSlots;
  if (ds.pending[i]) {
    st = hip_check(hipEventSynchronize(ds.ev[i]), "hipEventSynchronize");
    if (st != VC_OK) return st;
    ds.pending[i] = false;
  }
  memcpy(ds.host[i], src, bytes);
  dsp = &ds;
  slot = i;
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

// Kernel parameters of a planned call whose workspace starts at `base`.
vck::Params make_params(const Plan &plan, const vc_tol *tols, const Outputs &out, uint8_t *base,
                        bool single) {
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
  P.gdone = (uint32_t *)(base + plan.off_gdone);
  P.tile_maps = plan.do_tiles && out.tile_maps != nullptr ? (uint32_t *)(base + plan.off_tacc)
                                                          : nullptr;
  P.tile_out = P.tile_maps != nullptr ? out.tile_maps : nullptr;
  P.tiles_total = P.tile_maps != nullptr ? plan.tiles_total : 0;
  P.n_groups = plan.total_groups;
  P.stats = out.stats;
  P.mismatches = out.mismatches;
  P.pass_out = out.pass;
  P.first_k = plan.do_firstk ? out.first_k : nullptr;
  P.integ = out.integ;
  P.match_rate = out.match_rate;
  P.numeric_rate = out.numeric_rate;
  if (single) {
    P.cases = nullptr;
    P.single = plan.table[0];
  } else if (plan.n_cases > 0) {
    P.cases = (const vck::DevCase *)(base + plan.off_table);
    P.case_chunk = (const uint64_t *)(base + plan.off_cc);
    P.group_case = plan.group_case.empty() ? nullptr : (const uint32_t *)(base + plan.off_gc);
  }
  return P;
}

// The prologue of a call: copies the blob from `blob_src` (a pinned slot,
// or nullptr when it is already in place) and clears the parts of the
// workspace that must be zero on entry; with no cases, writes zero rates.
vck::Prologue make_prologue(const Plan &plan, const vck::Params &P, uint8_t *base,
                            const void *blob_src) {
  vck::Prologue Q;
  memset(&Q, 0, sizeof Q);
  if (blob_src != nullptr) {
    Q.blob_src = (const uint8_t *)blob_src;
    Q.blob_dst = base + plan.off_table;
    Q.blob_bytes = plan.blob_bytes;
  }
  Q.zero = (uint32_t *)(base + plan.off_zero);
  Q.zero_words = plan.zero_bytes / sizeof(uint32_t);
  Q.match_rate = P.match_rate;
  Q.numeric_rate = P.numeric_rate;
  Q.n_cases = plan.n_cases;
  Q.n_tols = plan.n_tols;
  return Q;
}

// The streaming and finalize launches of a planned call, back to back: no
// host work or event sits between them (except the optional profiling
// events), so the GPU never waits for the host inside a call.
vc_status launch_streaming(const Plan &plan, const vck::Params &P, hipStream_t stream) {
  hipEvent_t prof_begin = g_prof_begin, prof_end = g_prof_end;
  g_prof_begin = g_prof_end = nullptr;
  vc_status st = VC_OK;
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
    st = hip_check(vck::launch_main(g.dtype, plan.nt_class, plan.do_integ ? 1 : 0, G,
                                    g.n_chunks, stream),
                   "main kernel launch");
    if (st != VC_OK) return st;
  }
  if (prof_end != nullptr) {
    st = hip_check(hipEventRecord(prof_end, stream), "profile end event");
    if (st != VC_OK) return st;
  }
  return hip_check(vck::launch_finalize(P, stream), "finalize launch");
}

// A one-shot call: uploads the blob (a pinned slot read by the prologue, or
// a pageable copy for a blob larger than a slot), clears the zero-on-entry
// parts, then launches. `single` passes the one descriptor by value (no
// table). `allocate` = false (the allocation-free entry point): the blob
// must fit a slot of an existing ring.
vc_status run(const Plan &plan, const vc_tol *tols, const Outputs &out, void *ws, size_t ws_bytes,
              hipStream_t stream, bool single, bool allocate = true) {
  if (ws == nullptr) return fail(VC_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < plan.bytes)
    return fail(VC_ERR_WORKSPACE, "workspace has %zu bytes, %zu required", ws_bytes, plan.bytes);
  uint8_t *base = (uint8_t *)(((uintptr_t)ws + kAlign - 1) / kAlign * kAlign);
  const vck::Params P = make_params(plan, tols, out, base, single);

  std::unique_lock<std::mutex> lock;
  DeviceState *ds = nullptr;
  int slot = -1;
  const void *src = nullptr;
  vc_status st = VC_OK;
  if (!single && plan.n_cases > 0) {
    const std::vector<uint8_t> blob = plan_blob(plan);
    if (blob.size() <= kSlotBytes) {
      st = stage_blob(blob.data(), blob.size(), allocate, lock, ds, slot);
      if (st != VC_OK) return st;
      src = ds->dev[slot];
    } else {
      if (!allocate)
        return fail(VC_ERR_LIMIT, "the case table (%zu bytes) exceeds the %zu-byte staging slot",
                    blob.size(), kSlotBytes);
      st = hip_check(hipMemcpyAsync(base + plan.off_table, blob.data(), blob.size(),
                                    hipMemcpyHostToDevice, stream),
                     "descriptor upload");
      if (st != VC_OK) return st;
    }
  }
  const vck::Prologue Q = make_prologue(plan, P, base, src);
  st = hip_check(vck::launch_prologue(Q, stream), "prologue launch");
  if (st == VC_OK) st = launch_streaming(plan, P, stream);
  if (ds != nullptr) {
    // The slot may be refilled once the prologue has read it; an event
    // behind the call's last kernel (recorded also after a failed launch, in
    // case the prologue was enqueued) guards that. The lock is held until then.
    const vc_status se = hip_check(hipEventRecord(ds->ev[slot], stream), "hipEventRecord");
    if (se == VC_OK) ds->pending[slot] = true;
    if (st == VC_OK) st = se;
  }
  return st;
}

// Argument checks and plan of a sweep (vcheck_sweep, vcheck_sweep_noalloc,
// vcheck_plan_sweep).
vc_status plan_sweep(const vc_case *cases, int32_t n_cases, const vc_tol *tols, int32_t n_tols,
                     const vc_sweep_opts *opts, const vc_sweep_out *out, Plan &plan,
                     Outputs &oo) {
  if (out == nullptr) return fail(VC_ERR_NULL, "output descriptor is NULL");
  if (out->stats == nullptr && n_cases > 0) return fail(VC_ERR_NULL, "out->stats is NULL");
  vc_sweep_opts o{};
  if (opts != nullptr) o = *opts;
  if (o.do_integrity == 1 && out->integ == nullptr && n_cases > 0)
    return fail(VC_ERR_NULL, "do_integrity is set but out->integ is NULL");
  const bool want_tiles = out->tile_maps != nullptr;
  const bool want_firstk = out->first_k != nullptr;
  if (o.k > 0 && !want_firstk) o.k = 0;
  const vc_status st =
      make_plan(cases, n_cases, tols, n_tols, o, want_tiles, want_firstk, false, plan);
  if (st != VC_OK) return st;
  oo.stats = out->stats;
  oo.mismatches = out->mismatches;
  oo.pass = out->pass;
  oo.match_rate = out->match_rate;
  oo.numeric_rate = out->numeric_rate;
  oo.tile_maps = out->tile_maps;
  oo.first_k = out->first_k;
  oo.integ = out->integ;
  return VC_OK;
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

// Elements per wave of the probe, the content hash and the near-pass
// statistics: a power of two between 1 Ki and 32 Ki (a wave's range stays
// within 128 KiB: 32-bit offsets; the histogram counters are 32-bit), about
// 16K waves over the batch, and at least what keeps every tensor within 256
// groups of 256 chunks.
uint32_t probe_unit(uint64_t total, uint64_t largest) {
  constexpr uint64_t kCap = 32768;
  uint64_t u = 1024;
  while (u < kCap && u * 2 * VCK_WAVE_TARGET <= total) u *= 2;
  while (u < kCap && 4 * u * vck::kProbeGroupChunks * vck::kProbeGroupChunks < largest) u *= 2;
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

// Runs one diagnostic call: uploads the descriptor blob (`parts`, copied
// back to back, a multiple of 16 bytes) to `base` (staged in a pinned slot
// that the prologue reads, or a pageable copy when larger than a slot),
// enqueues the prologue (clearing `zero_words` words at `zero`) and then
// `launch` (which receives the profiling events), and records the slot's
// event behind them.
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
  DeviceState *ds = nullptr;
  int slot = -1;
  vck::Prologue Q;
  memset(&Q, 0, sizeof Q);
  vc_status st = VC_OK;
  if (total <= kSlotBytes) {
    st = stage_blob(blob.data(), blob.size(), true, lock, ds, slot);
    if (st != VC_OK) return st;
    Q.blob_src = (const uint8_t *)ds->dev[slot];
    Q.blob_dst = base;
    Q.blob_bytes = total;
  } else {
    st = hip_check(hipMemcpyAsync(base, blob.data(), total, hipMemcpyHostToDevice, stream),
                   "descriptor upload");
    if (st != VC_OK) return st;
  }
  Q.zero = zero;
  Q.zero_words = zero_words;
  Q.n_cases = 1;  // (no suite rates to clear)
  hipEvent_t prof_begin = g_prof_begin, prof_end = g_prof_end;
  g_prof_begin = g_prof_end = nullptr;
  st = hip_check(vck::launch_prologue(Q, stream), "prologue launch");
  if (st == VC_OK) st = hip_check(launch(prof_begin, prof_end), what);
  if (ds != nullptr) {
    // the staging slot is reused once the prologue has read it
    const vc_status se = hip_check(hipEventRecord(ds->ev[slot], stream), "hipEventRecord");
    if (se == VC_OK) ds->pending[slot] = true;
    if (st == VC_OK) st = se;
  }
  return st;
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

// A prepared sweep: its plan and kernel parameters (pointing into the
// caller's workspace, which holds the uploaded case table).
struct vc_plan {
  Plan plan;
  vck::Params P;
  int device;
};

// Scratch of the allocation-free entry point (vcheck_sweep_noalloc): the
// workspace of its calls, one copy per device. Host code reaches it only
// through the device address that vcheck_init takes with
// hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[VC_NOALLOC_SCRATCH_BYTES];

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
  Plan plan;
  Outputs oo;
  const vc_status st = plan_sweep(cases, n_cases, tols, n_tols, opts, out, plan, oo);
  if (st != VC_OK) return st;
  return run(plan, tols, oo, ws, ws_bytes, (hipStream_t)stream, false);
}

vc_status vcheck_init(void) {
  g_last_error.clear();
  int dev = 0;
  vc_status st = current_device(dev);
  if (st != VC_OK) return st;
  DeviceState &ds = g_dev[dev];
  std::lock_guard<std::mutex> lock(ds.mu);
  st = ensure_ring(ds);
  if (st != VC_OK) return st;
  if (ds.scratch == nullptr) {
    void *p = nullptr;
    st = hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress");
    if (st != VC_OK) return st;
    ds.scratch = (uint8_t *)p;
  }
  return VC_OK;
}

vc_status vcheck_sweep_noalloc(const vc_case *cases, int32_t n_cases, const vc_tol *tols,
                               int32_t n_tols, const vc_sweep_opts *opts,
                               const vc_sweep_out *out, void *stream) {
  g_last_error.clear();
  Plan plan;
  Outputs oo;
  vc_status st = plan_sweep(cases, n_cases, tols, n_tols, opts, out, plan, oo);
  if (st != VC_OK) return st;
  if (plan.bytes > (size_t)VC_NOALLOC_SCRATCH_BYTES)
    return fail(VC_ERR_LIMIT, "the sweep needs %zu bytes of scratch; the maximum is %zu",
                plan.bytes, (size_t)VC_NOALLOC_SCRATCH_BYTES);
  int dev = 0;
  st = current_device(dev);
  if (st != VC_OK) return st;
  uint8_t *ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_dev[dev].mu);
    ws = g_dev[dev].scratch;
  }
  if (ws == nullptr) return fail(VC_ERR_STATE, "vcheck_init has not run on device %d", dev);
  return run(plan, tols, oo, ws, (size_t)VC_NOALLOC_SCRATCH_BYTES, (hipStream_t)stream, false,
             false);
}

vc_status vcheck_plan_sweep(const vc_case *cases, int32_t n_cases, const vc_tol *tols,
                            int32_t n_tols, const vc_sweep_opts *opts, const vc_sweep_out *out,
                            void *ws, size_t ws_bytes, void *stream_, vc_plan **plan_out) {
  g_last_error.clear();
  if (plan_out == nullptr) return fail(VC_ERR_NULL, "plan pointer is NULL");
  Plan plan;
  Outputs oo;
  vc_status st = plan_sweep(cases, n_cases, tols, n_tols, opts, out, plan, oo);
  if (st != VC_OK) return st;
  if (ws == nullptr) return fail(VC_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < plan.bytes)
    return fail(VC_ERR_WORKSPACE, "workspace has %zu bytes, %zu required", ws_bytes, plan.bytes);
  int dev = 0;
  st = current_device(dev);
  if (st != VC_OK) return st;
  const hipStream_t stream = (hipStream_t)stream_;
  uint8_t *base = (uint8_t *)(((uintptr_t)ws + kAlign - 1) / kAlign * kAlign);
  const vck::Params P = make_params(plan, tols, oo, base, false);
  // the case table stays in the workspace; the zero-on-entry parts are
  // cleared once here and by every launch's finalize afterwards
  if (plan.n_cases > 0) {
    const std::vector<uint8_t> blob = plan_blob(plan);
    st = hip_check(hipMemcpyAsync(base + plan.off_table, blob.data(), blob.size(),
                                  hipMemcpyHostToDevice, stream),
                   "descriptor upload");
    if (st != VC_OK) return st;
  }
  const vck::Prologue Q = make_prologue(plan, P, base, nullptr);
  st = hip_check(vck::launch_prologue(Q, stream), "prologue launch");
  if (st == VC_OK) st = hip_check(hipStreamSynchronize(stream), "hipStreamSynchronize");
  if (st != VC_OK) return st;
  vc_plan *p = new (std::nothrow) vc_plan;
  if (p == nullptr) return fail(VC_ERR_LIMIT, "out of host memory");
  p->plan = std::move(plan);
  p->P = P;
  p->device = dev;
  *plan_out = p;
  return VC_OK;
}

vc_status vcheck_plan_launch(vc_plan *plan, void *stream_) {
  g_last_error.clear();
  if (plan == nullptr) return fail(VC_ERR_NULL, "plan is NULL");
  int dev = 0;
  vc_status st = current_device(dev);
  if (st != VC_OK) return st;
  if (dev != plan->device)
    return fail(VC_ERR_STATE, "the plan was made on device %d, the current device is %d",
                plan->device, dev);
  const hipStream_t stream = (hipStream_t)stream_;
  if (plan->plan.n_cases == 0) {
    vck::Prologue Q;  // zero rates only
    memset(&Q, 0, sizeof Q);
    Q.match_rate = plan->P.match_rate;
    Q.numeric_rate = plan->P.numeric_rate;
    Q.n_tols = plan->plan.n_tols;
    return hip_check(vck::launch_prologue(Q, stream), "prologue launch");
  }
  return launch_streaming(plan->plan, plan->P, stream);
}

vc_status vcheck_plan_free(vc_plan *plan) {
  g_last_error.clear();
  delete plan;
  return VC_OK;
}

vc_status vcheck_workspace_bytes(const vc_case *cases, int32_t n_cases, int32_t n_tols,
                                 const vc_sweep_opts *opts, size_t *bytes) {
  g_last_error.clear();
  if (bytes == nullptr) return fail(VC_ERR_NULL, "bytes is NULL");
  vc_sweep_opts o{};
  if (opts != nullptr) o = *opts;
  if (n_tols < 1 || n_tols > VC_MAX_TOLS)
    return fail(VC_ERR_LIMIT, "n_tols %d outside 1..%d", n_tols, VC_MAX_TOLS);
  // sizing does not depend on tolerance values; tile geometry >= 1 x 1
  // means tile maps (4 bytes of accumulator per tile)
  vc_tol dummy[VC_MAX_TOLS];
  for (auto &t : dummy) t = vc_tol{0.0, 0.0, 0, 0};
  const bool tiles = o.tile_h >= 1 && o.tile_w >= 1;
  if (o.primary_tol < 0 || o.primary_tol >= n_tols) o.primary_tol = 0;
  Plan plan;
  const vc_status st = make_plan(cases, n_cases, dummy, n_tols, o, tiles, o.k > 0, false, plan);
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
    case VC_ERR_STATE: return "library state does not allow the call (see vcheck_last_error)";
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
