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
// (4 waves) owns one chunk and each wave one contiguous quarter of it, so
// per-wave results combine in flat-index order. Each lane loads 16 bytes of
// cand and 16 bytes of ref per step (one fully coalesced 1 KiB access per
// wave and tensor), with the next step's loads issued before the current
// step is evaluated.
//
// Exactness: the gate is evaluated in binary64 on exactly decoded values with
// separate rounding of rtol*|r| and atol + (.) (no contraction anywhere in
// this file). Per-step fast path: when every pair of the step is finite and
// every |r| is non-zero (detected by the finiteness of the step's approximate
// relative-error sum), the counters are known without per-element class
// tests; otherwise the step is redone element by element on the exact path
// from the registers it already holds. max |c-r| is tracked exactly; max
// |c-r|/|r| candidates are found with the exact sign test
// fma(-M, |r|, d) > 0 <=> d/|r| > M and confirmed with a correctly rounded
// division, so the reported maximum equals the correctly rounded quotient.
// Only sum_rel uses an approximate reciprocal (it is specified to 1e-6
// relative). Counts come from wave ballots and popcounts; no floating-point
// atomics are used, so every result is bit-reproducible.
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

// Exact widening of one storage element to binary64.
template <int DT>
__device__ __forceinline__ double decode(uint32_t raw) {
  if constexpr (DT == VC_F32) {
    return (double)__uint_as_float(raw);
  } else if constexpr (DT == VC_F16) {
    const _Float16 h = __builtin_bit_cast(_Float16, (uint16_t)raw);
    return (double)(float)h;
  } else {
    return (double)__uint_as_float(raw << 16);
  }
}

template <int DT>
__device__ __forceinline__ bool is_zero_bits(uint32_t raw) {
  if constexpr (DT == VC_F32) return (raw & 0x7fffffffu) == 0;
  else return (raw & 0x7fffu) == 0;
}

// binary16 holds the binary32 value exactly (NaN and +-Inf count): the
// round trip through binary16 returns the value unchanged.
__device__ __forceinline__ bool fp16_exact(uint32_t raw) {
  const float f = __uint_as_float(raw);
  const float rt = (float)(_Float16)f;
  return rt == f || f != f;
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ uint32_t popc(uint64_t m) { return (uint32_t)__popcll(m); }
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

template <int DT>
__device__ __forceinline__ void load_vec(const uint8_t *p, uint32_t (&v)[Tr<DT>::V]) {
  const uint4 x = *reinterpret_cast<const uint4 *>(p);
  if constexpr (Tr<DT>::ES == 4) {
    v[0] = x.x;
    v[1] = x.y;
    v[2] = x.z;
    v[3] = x.w;
  } else {
    v[0] = x.x & 0xffffu;
    v[1] = x.x >> 16;
    v[2] = x.y & 0xffffu;
    v[3] = x.y >> 16;
    v[4] = x.z & 0xffffu;
    v[5] = x.z >> 16;
    v[6] = x.w & 0xffffu;
    v[7] = x.w >> 16;
  }
}

// Element loads of positions idx0 .. idx0+V-1 below `end` (others read 0).
template <int DT>
__device__ __forceinline__ void load_guarded(const uint8_t *base, uint64_t idx0, uint64_t end,
                                             uint32_t (&v)[Tr<DT>::V]) {
#pragma unroll
  for (int j = 0; j < Tr<DT>::V; ++j) {
    const uint64_t i = idx0 + j;
    uint32_t x = 0;
    if (i < end) {
      if constexpr (Tr<DT>::ES == 4) x = *reinterpret_cast<const uint32_t *>(base + i * 4);
      else x = *reinterpret_cast<const uint16_t *>(base + i * 2);
    }
    v[j] = x;
  }
}

struct WaveOut {
  uint32_t mism[VC_MAX_TOLS];
  uint32_t nan_c, inf_c, nan_r, inf_r, n_fin, n_rel, n_rel_undef, eq_bits;
  uint32_t nfound, zc, zr, efc, efr, bfc, bfr, hfc, hfr;
  uint32_t amax_abs, amax_rel;
  double max_abs, max_rel, sum_abs, sum_rel;
};

__device__ __forceinline__ void max_merge(double &v, uint32_t &i, double ov, uint32_t oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

template <int DT, int NT, bool INTEG>
__global__ __launch_bounds__(kBlockThreads) void main_kernel(const Params P) {
  constexpr int V = Tr<DT>::V;
  constexpr int ES = Tr<DT>::ES;
  constexpr uint32_t ITER = kWaveSize * V;

  __shared__ uint32_t s_win[kWavesPerBlock][kTileWindow];
  __shared__ WaveOut s_out[kWavesPerBlock];

  const uint32_t lane = threadIdx.x & (kWaveSize - 1);
  const uint32_t wave = threadIdx.x / kWaveSize;
  const uint64_t chunk = P.chunk_lo + blockIdx.x;

  // Locate the case: the last table entry whose first chunk is <= chunk.
  const DevCase *cs = &P.single;
  if (P.cases != nullptr) {
    uint64_t lo = P.case_lo, hi = P.case_hi - 1;
    while (lo < hi) {
      const uint64_t mid = (lo + hi + 1) / 2;
      if (P.cases[mid].chunk_begin <= chunk) lo = mid;
      else hi = mid - 1;
    }
    cs = &P.cases[lo];
  }
  const uint8_t *const cand = cs->cand;
  const uint8_t *const ref = cs->ref;
  const uint64_t numel = cs->numel;
  const uint64_t cols = cs->cols;
  const uint64_t tiles_c = cs->tiles_c;
  const uint64_t tile_off = cs->tile_off;
  const bool vec = cs->vec_ok != 0;
  const uint64_t U = P.unit_elems;
  const uint64_t cstart = (chunk - cs->chunk_begin) * (4 * U);
  const uint64_t cend = min(cstart + 4 * U, numel);
  const uint64_t wlo = min(cstart + wave * U, cend);
  const uint64_t whi = min(wlo + U, cend);

  // per-lane running state
  double run_abs = -1.0, run_rel = -1.0;
  uint32_t arg_abs = 0xffffffffu, arg_rel = 0xffffffffu;
  double sabs = 0.0, srel = 0.0;
  // wave-uniform counters
  uint32_t mism[NT];
#pragma unroll
  for (int p = 0; p < NT; ++p) mism[p] = 0;
  uint32_t nan_c = 0, inf_c = 0, nan_r = 0, inf_r = 0, n_fin = 0, n_rel = 0, n_rel_undef = 0;
  uint32_t zc = 0, zr = 0, efc = 0, efr = 0, bfc = 0, bfr = 0, hfc = 0, hfr = 0;
  uint64_t diff_cr = 0;
  uint32_t eqc = INTEG ? cs->inp_mask : 0u, eqr = eqc;
  uint32_t nfound = 0;
  uint32_t first_c = 0, first_r = 0;
  if constexpr (INTEG) {
    if (numel > 0) {
      if constexpr (ES == 4) {
        first_c = *reinterpret_cast<const uint32_t *>(cand);
        first_r = *reinterpret_cast<const uint32_t *>(ref);
      } else {
        first_c = *reinterpret_cast<const uint16_t *>(cand);
        first_r = *reinterpret_cast<const uint16_t *>(ref);
      }
    }
  }

  // Tile window: LDS counters for the tile-id range this wave can touch.
  const uint32_t th = (uint32_t)P.tile_h, tw = (uint32_t)P.tile_w;
  bool win_ok = false;
  uint64_t win_base = 0;
  if (P.do_tiles && wlo < whi) {
    const uint64_t row_lo = wlo / cols, row_hi = (whi - 1) / cols;
    uint64_t t_min, t_max;
    if (row_lo == row_hi) {
      t_min = (row_lo / th) * tiles_c + (wlo - row_lo * cols) / tw;
      t_max = (row_lo / th) * tiles_c + (whi - 1 - row_lo * cols) / tw;
    } else {
      t_min = (row_lo / th) * tiles_c;
      t_max = (row_hi / th) * tiles_c + tiles_c - 1;
    }
    win_ok = (t_max - t_min) < (uint64_t)kTileWindow;
    win_base = t_min;
    if (win_ok)
      for (uint32_t e = lane; e < (uint32_t)kTileWindow; e += kWaveSize) s_win[wave][e] = 0;
    __builtin_amdgcn_wave_barrier();
  }
  uint32_t *const stage =
      P.stage + ((uint64_t)chunk * kWavesPerBlock + wave) * (uint64_t)(P.k > 0 ? P.k : 0);

  // Evaluate one step: V elements per lane starting at case index i0;
  // element j is present iff bit j of vmask is set.
  auto step = [&](const uint32_t (&cv)[V], const uint32_t (&rv)[V], uint32_t vmask, bool full,
                  uint64_t i0) {
    const uint32_t off0 = (uint32_t)(i0 - cstart);
    uint32_t fb[NT];
    bool done = false;
    if (full) {
      double dd[V], ar[V];
      double s_a = 0.0, s_r = 0.0, dmax = 0.0;
#pragma unroll
      for (int p = 0; p < NT; ++p) fb[p] = 0;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const double c = decode<DT>(cv[j]);
        const double r = decode<DT>(rv[j]);
        const double d = __builtin_fabs(c - r);
        const double a = __builtin_fabs(r);
        dd[j] = d;
        ar[j] = a;
#pragma unroll
        for (int p = 0; p < NT; ++p) {
          const double t = P.atol[p] + P.rtol[p] * a;
          fb[p] |= (d <= t ? 0u : 1u) << j;
        }
        s_a += d;
        s_r += d * __builtin_amdgcn_rcp(a);
        dmax = __builtin_fmax(dmax, d);
      }
      // s_r is finite iff every c and r of the lane is finite and every r != 0
      if (ballot(!__builtin_isfinite(s_r)) == 0) {
        done = true;
        n_fin += ITER;
        n_rel += ITER;
        sabs += s_a;
        srel += s_r;
        if (ballot(dmax > run_abs) != 0) {
          if (dmax > run_abs) {
#pragma unroll
            for (int j = 0; j < V; ++j)
              if (dd[j] > run_abs) {
                run_abs = dd[j];
                arg_abs = off0 + j;
              }
          }
        }
        bool rc = false;
#pragma unroll
        for (int j = 0; j < V; ++j) rc |= __builtin_fma(-run_rel, ar[j], dd[j]) > 0.0;
        if (ballot(rc) != 0) {
          if (rc) {
#pragma unroll
            for (int j = 0; j < V; ++j)
              if (__builtin_fma(-run_rel, ar[j], dd[j]) > 0.0) {
                const double q = dd[j] / ar[j];
                if (q > run_rel) {
                  run_rel = q;
                  arg_rel = off0 + j;
                }
              }
          }
        }
      }
    }
    if (!done) {
      // exact element-by-element path
#pragma unroll
      for (int p = 0; p < NT; ++p) fb[p] = 0;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const bool valid = (vmask >> j) & 1u;
        const double c = decode<DT>(cv[j]);
        const double r = decode<DT>(rv[j]);
        const bool c_nan = __builtin_isnan(c), c_inf = __builtin_isinf(c);
        const bool r_nan = __builtin_isnan(r), r_inf = __builtin_isinf(r);
        nan_c += popc(ballot(valid && c_nan));
        inf_c += popc(ballot(valid && c_inf));
        nan_r += popc(ballot(valid && r_nan));
        inf_r += popc(ballot(valid && r_inf));
        const bool fin = valid && !(c_nan || c_inf || r_nan || r_inf);
        const double d = __builtin_fabs(c - r);
        const double a = __builtin_fabs(r);
#pragma unroll
        for (int p = 0; p < NT; ++p) {
          const double t = P.atol[p] + P.rtol[p] * a;
          const bool close =
              (c == r) || (fin && d <= t) || (((P.eqnan_mask >> p) & 1u) && c_nan && r_nan);
          fb[p] |= ((valid && !close) ? 1u : 0u) << j;
        }
        const bool relok = fin && r != 0.0;
        n_fin += popc(ballot(fin));
        n_rel += popc(ballot(relok));
        n_rel_undef += popc(ballot(fin && r == 0.0 && c != 0.0));
        if (fin) {
          sabs += d;
          if (d > run_abs) {
            run_abs = d;
            arg_abs = off0 + j;
          }
        }
        if (relok) {
          const double q = d / a;
          srel += q;
          if (q > run_rel) {
            run_rel = q;
            arg_rel = off0 + j;
          }
        }
      }
    }
    // mismatch counts for every pair
#pragma unroll
    for (int p = 0; p < NT; ++p)
#pragma unroll
      for (int j = 0; j < V; ++j) mism[p] += popc(ballot((fb[p] >> j) & 1u));

    // localization at the primary pair
    uint32_t pb = 0;
#pragma unroll
    for (int p = 0; p < NT; ++p)
      if (p == P.primary) pb = fb[p];
    if (ballot(pb != 0) != 0) {
      if (P.k > 0 && nfound < (uint32_t)P.k) {
        uint32_t before = 0, total = 0;
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const uint64_t b = ballot((pb >> j) & 1u);
          before += lanes_below(b);
          total += popc(b);
        }
        uint32_t pos = nfound + before;
#pragma unroll
        for (int j = 0; j < V; ++j)
          if ((pb >> j) & 1u) {
            if (pos < (uint32_t)P.k) stage[pos] = off0 + j;
            ++pos;
          }
        nfound = min(nfound + total, (uint32_t)P.k);
      }
      if (P.do_tiles && pb != 0) {
#pragma unroll
        for (int j = 0; j < V; ++j)
          if ((pb >> j) & 1u) {
            const uint64_t i = i0 + j;
            const uint64_t row = i / cols;
            const uint64_t col = i - row * cols;
            const uint64_t t = (row / th) * tiles_c + col / tw;
            if (win_ok && t >= win_base && t - win_base < (uint64_t)kTileWindow)
              atomicAdd(&s_win[wave][t - win_base], 1u);
            else
              atomicAdd(&P.tile_maps[tile_off + t], 1u);
          }
      }
    }

    // degenerate-output detector counts
    if constexpr (INTEG) {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const bool valid = (vmask >> j) & 1u;
        const uint32_t c = cv[j], r = rv[j];
        zc += popc(ballot(valid && is_zero_bits<DT>(c)));
        zr += popc(ballot(valid && is_zero_bits<DT>(r)));
        efc += popc(ballot(valid && c == first_c));
        efr += popc(ballot(valid && r == first_r));
        if constexpr (DT == VC_F32) {
          bfc += popc(ballot(valid && (c & 0xffffu) == 0));
          bfr += popc(ballot(valid && (r & 0xffffu) == 0));
          hfc += popc(ballot(valid && fp16_exact(c)));
          hfr += popc(ballot(valid && fp16_exact(r)));
        }
        diff_cr |= ballot(valid && c != r);
      }
      // operator inputs: read only while cand or ref is still bit-equal
      uint32_t need = eqc | eqr;
      while (need != 0) {
        const int jx = __builtin_ctz(need);
        need &= need - 1;
        const uint8_t *xp = cs->inp[jx];
        uint32_t xv[V];
        if (vec && full) load_vec<DT>(xp + i0 * ES, xv);
        else load_guarded<DT>(xp, i0, whi, xv);
        bool dc = false, dr = false;
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const bool valid = (vmask >> j) & 1u;
          dc |= valid && cv[j] != xv[j];
          dr |= valid && rv[j] != xv[j];
        }
        if (ballot(dc) != 0) eqc &= ~(1u << jx);
        if (ballot(dr) != 0) eqr &= ~(1u << jx);
      }
    }
  };

  const uint64_t n_elems = whi - wlo;
  const uint64_t n_full = n_elems / ITER;
  const uint64_t lane_off = (uint64_t)lane * V;
  uint32_t c_cur[V], r_cur[V];
  const uint32_t all = (1u << V) - 1u;
  if (n_full > 0) {
    const uint64_t i0 = wlo + lane_off;
    if (vec) {
      load_vec<DT>(cand + i0 * ES, c_cur);
      load_vec<DT>(ref + i0 * ES, r_cur);
    } else {
      load_guarded<DT>(cand, i0, whi, c_cur);
      load_guarded<DT>(ref, i0, whi, r_cur);
    }
  }
  for (uint64_t it = 0; it < n_full; ++it) {
    const uint64_t i0 = wlo + it * ITER + lane_off;
    uint32_t c_nxt[V], r_nxt[V];
    const bool more = it + 1 < n_full;
    if (more) {
      const uint64_t i1 = i0 + ITER;
      if (vec) {
        load_vec<DT>(cand + i1 * ES, c_nxt);
        load_vec<DT>(ref + i1 * ES, r_nxt);
      } else {
        load_guarded<DT>(cand, i1, whi, c_nxt);
        load_guarded<DT>(ref, i1, whi, r_nxt);
      }
    }
    step(c_cur, r_cur, all, true, i0);
    if (more) {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        c_cur[j] = c_nxt[j];
        r_cur[j] = r_nxt[j];
      }
    }
  }
  if (n_elems % ITER != 0) {
    const uint64_t i0 = wlo + n_full * ITER + lane_off;
    load_guarded<DT>(cand, i0, whi, c_cur);
    load_guarded<DT>(ref, i0, whi, r_cur);
    uint32_t vmask = 0;
#pragma unroll
    for (int j = 0; j < V; ++j) vmask |= (i0 + j < whi ? 1u : 0u) << j;
    step(c_cur, r_cur, vmask, false, i0);
  }

  // flush the tile window
  if (P.do_tiles && win_ok) {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
    for (uint32_t e = lane; e < (uint32_t)kTileWindow; e += kWaveSize) {
      const uint32_t v = s_win[wave][e];
      if (v != 0) atomicAdd(&P.tile_maps[tile_off + win_base + e], v);
    }
  }

  // wave reduction (fixed butterfly order)
#pragma unroll
  for (int m = kWaveSize / 2; m >= 1; m >>= 1) {
    sabs += __shfl_xor(sabs, m);
    srel += __shfl_xor(srel, m);
    const double oa = __shfl_xor(run_abs, m);
    const uint32_t ia = __shfl_xor(arg_abs, m);
    max_merge(run_abs, arg_abs, oa, ia);
    const double orl = __shfl_xor(run_rel, m);
    const uint32_t irl = __shfl_xor(arg_rel, m);
    max_merge(run_rel, arg_rel, orl, irl);
  }
  if (lane == 0) {
    WaveOut &o = s_out[wave];
#pragma unroll
    for (int p = 0; p < VC_MAX_TOLS; ++p) o.mism[p] = p < NT ? mism[p] : 0u;
    o.nan_c = nan_c;
    o.inf_c = inf_c;
    o.nan_r = nan_r;
    o.inf_r = inf_r;
    o.n_fin = n_fin;
    o.n_rel = n_rel;
    o.n_rel_undef = n_rel_undef;
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
    o.max_abs = run_abs;
    o.amax_abs = arg_abs;
    o.max_rel = run_rel;
    o.amax_rel = arg_rel;
    o.sum_abs = sabs;
    o.sum_rel = srel;
  }
  __syncthreads();
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
    rec.nfound[0] = w0.nfound;
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
      rec.nfound[w] = o.nfound;
    }
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
  const DevCase &cs = P.cases != nullptr ? P.cases[ci] : P.single;
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
