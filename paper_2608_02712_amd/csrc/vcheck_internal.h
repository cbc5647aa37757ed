// vcheck_internal.h -- layouts shared by the host C-ABI layer and the gfx950
// kernels of the validation library. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "vcheck.h"

namespace vck {

constexpr int kWaveSize = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlockThreads = kWaveSize * kWavesPerBlock;
constexpr int kTileWindow = 1024;  // LDS tile counters per block
constexpr int kGroupChunks = 256;  // chunks merged by one group record
constexpr uint32_t kMaxChunkElems = 1u << 17;  // 4 units of at most 64 KiB of 16-bit data

// Unsigned division of a 32-bit numerator by an invariant divisor d
// (1 <= d < 2^32) as a multiply-high, an add and two shifts (Granlund and
// Montgomery, Division by invariant integers using multiplication, PLDI 1994,
// Sec. 4, Fig. 4.1): with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1,
// t = mulhi(m, n) and n / d = (t + ((n - t) >> min(l, 1))) >> max(l - 1, 0).
struct DivMagic {
  uint32_t m;
  uint32_t shifts;  // min(l, 1) | max(l - 1, 0) << 8
};
inline DivMagic div_magic(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  DivMagic r;
  r.m = (uint32_t)((((1ull << 32) * ((1ull << l) - d)) / d) + 1);
  r.shifts = (l < 1 ? l : 1u) | ((l > 1 ? l - 1 : 0u) << 8);
  return r;
}
__device__ __forceinline__ uint32_t div_by(uint32_t n, uint32_t m, uint32_t shifts) {
  const uint32_t t = __umulhi(m, n);
  return (t + ((n - t) >> (shifts & 0xffu))) >> (shifts >> 8);
}

// Device-side case descriptor. The host builds one per case, in launch
// order (grouped by dtype), and uploads the table into the workspace (once
// for a prepared sweep). Every case owns at least one chunk: a case that is not
// evaluated (status != 0) or is empty gets one chunk with no elements, so
// its results are written by the same completion path as every other case.
struct DevCase {
  const uint8_t *cand;
  const uint8_t *ref;
  const uint8_t *inp[VC_MAX_INPUTS];
  uint64_t numel;
  uint64_t cols;         // C of the (R, C) view (1 for a 0-d tensor)
  uint64_t chunk_begin;  // global index of the case's first chunk
  uint64_t tile_off;     // offset of the case's tile map in the output
  uint64_t tiles_c;      // tiles per tile row: ceil(C / tile_w)
  uint64_t group_begin;  // global index of the case's first chunk group
  uint32_t n_chunks;     // >= 1
  uint32_t n_groups;     // ceil(n_chunks / kGroupChunks)
  int32_t status;        // 0, or a negative vc_status (case not evaluated)
  uint32_t inp_mask;     // bit j: input j takes part in the copy detector
  uint32_t vec_ok;       // 1: every pointer of the case is 16-byte aligned
  uint32_t orig;         // index of the case in the caller's arrays
  uint32_t dtype;
  uint32_t unit_elems;   // elements per wave range; a chunk is 4 of them
  DivMagic cols_div;     // division by cols (when cols < 2^31)
  uint64_t n_tiles;      // tiles of the case's map (0 without tile maps)
};
static_assert(sizeof(DevCase) == 176, "DevCase layout");

// Partial result of one chunk (one block of the main kernel; its four waves
// interleave over the chunk), or of one group of up to kGroupChunks chunks.
// Offsets are element offsets within the record's own range. The first
// kRecCounts words are counters that merge by addition.
struct ChunkRec {
  uint32_t mism[VC_MAX_TOLS];              // words 0..7
  uint32_t nan_c, inf_c, nan_r, inf_r;     // 8..11
  uint32_t n_fin, n_rel, n_rel_undef;      // 12..14
  uint32_t zero_c, zero_r, eqf_c, eqf_r;   // 15..18
  uint32_t bf_c, bf_r, f16_c, f16_r;       // 19..22
  uint32_t nfound;                         // staged first-k entries (<= k)
  uint32_t eq_bits;                        // see kEq* below; merges by AND
  uint32_t amax_abs, amax_rel;             // 0xffffffff when none
  uint32_t pad;
  double max_abs, max_rel;                 // -1.0 when none
  double sum_abs, sum_rel;
};
static_assert(sizeof(ChunkRec) == 144, "ChunkRec layout");
constexpr int kRecCounts = 23;

constexpr uint32_t kEqCandRef = 1u;        // bit 0: cand bit-equal to ref
constexpr int kEqCandInpShift = 8;         // bits 8..15: cand bit-equal to input j
constexpr int kEqRefInpShift = 16;         // bits 16..23: ref bit-equal to input j

// Suite counters in the workspace (zero on entry: cleared by the prologue of
// a one-shot call, and by the block that completes the last case, which
// reads them, for the next call of a prepared sweep).
struct Counters {
  uint32_t pass[VC_MAX_TOLS];       // cases passing pair p numerically
  uint32_t cert[VC_MAX_TOLS];       // ... and with no integrity flag
  uint32_t done;                    // cases whose results are written
  uint32_t pad[15];
};
static_assert(sizeof(Counters) == 128, "Counters layout");

// Kernel parameters (passed by value).
struct Params {
  const DevCase *cases;        // device table, or nullptr: use `single`
  const uint64_t *case_chunk;  // [table entries] chunk_begin, for the case lookup
  const uint32_t *group_case;  // [groups] table index of each chunk group, or nullptr
                               // when every case has one group (group = table index)
  int32_t n_cases;             // table entries (= caller cases)
  int32_t n_tols;              // 1 .. 8 (the kernel evaluates NT >= n_tols pairs)
  int32_t primary;
  int32_t tile_h, tile_w;
  DivMagic th_div, tw_div;     // division by tile_h, tile_w
  int32_t k;                   // first-k length (0: none)
  int32_t do_tiles;            // 1: tile maps requested
  int32_t do_integ;
  int32_t tier1;               // 1: the binary32 fast path is valid for these pairs
  uint32_t unit_elems;         // elements per wave range (one quarter of a chunk)
  uint32_t eqnan_mask;         // bit p: equal_nan of pair p
  uint64_t chunk_lo;           // first global chunk of this launch
  uint64_t case_lo;            // first table index of this launch's cases
  uint64_t case_hi;
  double atol[VC_MAX_TOLS];
  double rtol[VC_MAX_TOLS];
  // binary32 gate bounds of pair 0 (used when n_tols == 1):
  // fma(|r|, rlo, alo) <= atol + rtol |r| <= fma(|r|, rhi, ahi)
  float rlo, alo, rhi, ahi;

  ChunkRec *recs;              // [total chunks]
  uint32_t *stage;             // [total chunks * k] first-k lists (chunk offsets)
  ChunkRec *grecs;             // [total groups]
  uint32_t *gstage;            // [total groups * k]
  Counters *ctr;
  uint32_t *gdone;             // [table entries] groups merged (zero on entry)
  uint32_t *tile_maps;         // tile-count accumulators in the workspace (zero on
                               // entry), nullable
  uint32_t *tile_out;          // user tile maps, written by the finalize (nullable)
  uint64_t tiles_total;        // tiles of all maps of the call
  uint64_t n_groups;           // chunk groups of the call (finalize blocks that merge)
  // outputs
  vc_stats *stats;
  uint64_t *mismatches;
  uint8_t *pass_out;
  int64_t *first_k;
  vc_integrity *integ;
  double *match_rate;
  double *numeric_rate;
  DevCase single;
};

// Work of the prologue kernel of a one-shot call: copy the descriptor blob
// from pinned host memory (when staged there), clear the counters and the
// tile-count accumulators.
struct Prologue {
  const uint8_t *blob_src;  // device-visible pinned host pointer (or nullptr)
  uint8_t *blob_dst;
  uint64_t blob_bytes;      // multiple of 16
  uint32_t *zero;           // counter area
  uint64_t zero_words;
  uint32_t *tiles;
  uint64_t n_tiles;
  double *match_rate;       // written (0) when the sweep has no cases
  double *numeric_rate;
  int32_t n_cases;
  int32_t n_tols;
};

// ---- tensor-statistics probe (vcheck_probe.hip) ---------------------------

constexpr int kHistBins = 64;
constexpr int kHistEmin = -40;
constexpr uint32_t kProbeGroupChunks = 256;  // chunk records merged per group block

// One probed tensor (32 bytes). Its chunks are [chunk_begin, chunk_begin +
// n_chunks) (an empty tensor owns one empty chunk), its groups of up to
// kProbeGroupChunks chunks start at group_begin.
struct ProbeTensor {
  const uint8_t *data;
  uint64_t numel;
  uint64_t chunk_begin;
  uint32_t n_chunks;
  int32_t dtype;
};
static_assert(sizeof(ProbeTensor) == 32, "ProbeTensor layout");

// Partial statistics of one chunk or group (element indices within the
// tensor; -1 when no finite value).
struct ProbeRec {
  uint64_t nan, inf, zero, fin;
  int64_t argmin, argmax;
  double min, max, sum, sum_sq, sum_abs;
  uint32_t hist[kHistBins];
  uint64_t pad[1];
};
static_assert(sizeof(ProbeRec) == 352, "ProbeRec layout");
static_assert(sizeof(vc_tstats) == 608, "vc_tstats layout");

struct ProbeParams {
  const ProbeTensor *tensors;    // [n] in the workspace
  const uint64_t *chunk_first;   // [n] first chunk of each tensor (ascending)
  const uint64_t *group_first;   // [n] first group of each tensor (ascending)
  int32_t n_tensors;
  uint32_t unit;                 // elements per wave (a chunk is four)
  ProbeRec *recs;                // [total chunks]
  ProbeRec *grecs;               // [total groups]
  vc_tstats *out;                // [n]
};

// ---- near-pass statistics (vcheck_probe.hip) -------------------------------

constexpr int kRatioBins = 32;
constexpr int kUlpBins = 18;

// One case of the near-pass statistics (48 bytes); chunks and groups as for
// the probe.
struct NpCase {
  const uint8_t *cand;
  const uint8_t *ref;
  uint64_t numel;
  uint64_t chunk_begin;
  uint32_t n_chunks;
  int32_t dtype;
  uint64_t pad;
};
static_assert(sizeof(NpCase) == 48, "NpCase layout");

struct NpRec {
  uint64_t n_pairs, n_fail, n_zero_tol;
  double max_ratio;
  int64_t argmax_ratio;  // index within the case; -1 when none
  uint32_t max_ulp_fail, pad0;
  uint32_t ratio_hist[kRatioBins];
  uint32_t ulp_hist[kUlpBins];
  uint32_t pad1[2];
};
static_assert(sizeof(NpRec) == 256, "NpRec layout");
static_assert(sizeof(vc_nearpass) == 56 + 8 * (kRatioBins + kUlpBins), "vc_nearpass layout");

struct NpParams {
  const NpCase *cases;
  const uint64_t *chunk_first;
  const uint64_t *group_first;
  int32_t n_cases;
  uint32_t unit;
  double atol, rtol;
  NpRec *recs;
  NpRec *grecs;
  vc_nearpass *out;
};

hipError_t launch_nearpass(const NpParams &p, uint64_t n_chunks, uint64_t n_groups,
                           hipStream_t s, hipEvent_t begin, hipEvent_t end);

// Content hash: the probe's tensor table; out[t] is cleared by the prologue
// and receives one 64-bit atomic addition per chunk.
struct HashParams {
  const ProbeTensor *tensors;
  const uint64_t *chunk_first;
  int32_t n_tensors;
  uint32_t unit;
  unsigned long long *out;
};

hipError_t launch_hash(const HashParams &p, uint64_t n_chunks, hipStream_t s, hipEvent_t begin,
                       hipEvent_t end);

// Launches the probe's streaming and merge kernels; `begin` / `end`
// (nullable) are recorded around the streaming kernel.
hipError_t launch_probe(const ProbeParams &p, uint64_t n_chunks, uint64_t n_groups,
                        hipStream_t s, hipEvent_t begin, hipEvent_t end);

// Launchers (vcheck_kernels.hip). Each returns the HIP error of its launch.
hipError_t launch_prologue(const Prologue &p, hipStream_t s);
hipError_t launch_main(int dtype, int nt_class, int integ, const Params &p, uint64_t n_chunks,
                       hipStream_t s);
hipError_t launch_finalize(const Params &p, hipStream_t s);

}  // namespace vck
