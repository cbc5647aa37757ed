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
constexpr int kTileWindow = 2048;  // LDS tile counters per block

// Device-side case descriptor. The host builds one per case, in launch
// order (grouped by dtype), and uploads the table into the workspace.
struct DevCase {
  const uint8_t *cand;
  const uint8_t *ref;
  const uint8_t *inp[VC_MAX_INPUTS];
  uint64_t numel;
  uint64_t cols;         // C of the (R, C) view (1 for a 0-d tensor)
  uint64_t chunk_begin;  // global index of the case's first chunk
  uint64_t tile_off;     // offset of the case's tile map in the output
  uint64_t tiles_c;      // tiles per tile row: ceil(C / tile_w)
  uint32_t n_chunks;
  int32_t status;        // 0, or a negative vc_status (case not evaluated)
  uint32_t inp_mask;     // bit j: input j takes part in the copy detector
  uint32_t vec_ok;       // 1: every pointer of the case is 16-byte aligned
  uint32_t orig;         // index of the case in the caller's arrays
  uint32_t dtype;
  uint32_t unit_elems;   // elements per wave range; a chunk is 4 of them
  uint32_t reserved;
};
static_assert(sizeof(DevCase) == 152, "DevCase layout");

// Partial result of one chunk (one block of the main kernel; its four waves
// interleave over the chunk). Offsets are element offsets within the chunk.
struct ChunkRec {
  uint32_t mism[VC_MAX_TOLS];
  uint32_t nan_c, inf_c, nan_r, inf_r;
  uint32_t n_fin, n_rel, n_rel_undef, eq_bits;  // eq_bits: see kEq* below
  uint32_t nfound[kWavesPerBlock];              // staged first-k entries (all in slot 0)
  uint32_t zero_c, zero_r, eqf_c, eqf_r;
  uint32_t bf_c, bf_r, f16_c, f16_r;
  double max_abs, max_rel;  // -1.0 when the chunk has no finite / no rel pair
  uint32_t amax_abs, amax_rel;  // 0xffffffff when none
  uint32_t pad0, pad1;
  double sum_abs, sum_rel;
};
static_assert(sizeof(ChunkRec) == 160, "ChunkRec layout");

constexpr uint32_t kEqCandRef = 1u;        // bit 0: cand bit-equal to ref
constexpr int kEqCandInpShift = 8;         // bits 8..15: cand bit-equal to input j
constexpr int kEqRefInpShift = 16;         // bits 16..23: ref bit-equal to input j

// Kernel parameters (passed by value).
struct Params {
  const DevCase *cases;  // device table, or nullptr: use `single`
  int32_t n_cases;
  int32_t n_tols;        // 1 .. 8 (the kernel evaluates NT >= n_tols pairs)
  int32_t primary;
  int32_t tile_h, tile_w;
  int32_t k;             // first-k length (0: none)
  int32_t do_tiles;      // 1: tile maps requested
  int32_t do_integ;
  uint32_t unit_elems;   // elements per wave range (one quarter of a chunk)
  uint32_t eqnan_mask;   // bit p: equal_nan of pair p
  uint64_t chunk_lo;     // first global chunk of this launch
  uint64_t case_lo;      // first table index of this launch's cases
  uint64_t case_hi;
  double atol[VC_MAX_TOLS];
  double rtol[VC_MAX_TOLS];

  ChunkRec *recs;        // [total chunks]
  uint32_t *stage;       // [total chunks * 4 * k] first-k staging (offsets)
  uint32_t *tile_maps;   // user tile maps (nullable)
  // finalize outputs
  vc_stats *stats;
  uint64_t *mismatches;
  uint8_t *pass_out;
  int64_t *first_k;
  vc_integrity *integ;
  uint8_t *ws_pass;      // [n_cases * n_tols] always written by finalize
  uint32_t *ws_flags;    // [n_cases]
  double *match_rate;
  double *numeric_rate;
  uint64_t tiles_total;
  DevCase single;
};

// Launchers (vcheck_kernels.hip). Each returns the HIP error of its launch.
hipError_t launch_fill_u32(uint32_t *p, uint64_t n, hipStream_t s);
hipError_t launch_main(int dtype, int nt_class, int integ, const Params &p, uint64_t n_chunks,
                       hipStream_t s);
hipError_t launch_finalize(const Params &p, uint64_t n_cases_in_table, hipStream_t s);
hipError_t launch_rates(const Params &p, hipStream_t s);

}  // namespace vck
