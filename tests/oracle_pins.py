"""Pins that tie the CPU oracle to things other than itself.

Every check here derives its expectation by a route independent of the
oracle's C code: library routines with a documented definition
(``torch.isclose`` on binary64, numpy / torch dtype conversions, numpy
argmax / nonzero / reshape sums, ``math.fsum``), closed forms of the seeded
workloads, invariants that must hold for any input, and hand-built boundary
cases with literal expected values. ``tests/test_oracle_mutants.py`` plants
plausible mistakes in a copy of the oracle and requires at least one pin here
to fail for each, so a pin list that stops covering the oracle is noticed.

Pinned outputs: decode (fp32/fp16/bf16), the gate at every tolerance pair,
NaN/Inf counts, n_finite, n_rel, n_rel_undef, max/argmax abs and rel, sum
abs/rel, tile map, first-k, all integrity counts, input/ref bit-equality
masks, the five detector flags, copy_input, per-case pass and the suite match
rate; and the tensor-statistics probe (counts, first-index min/max, sums,
exponent histogram).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import torch

import oracle
import workloads as wl

F32, F16, BF16 = oracle.F32, oracle.F16, oracle.BF16


# ----------------------------------------------------------------- helpers
def lib_decode(raw: np.ndarray, dtype: int) -> np.ndarray:
    """binary64 values of raw storage via numpy / torch conversions."""
    if dtype == F32:
        with np.errstate(invalid="ignore"):
            return raw.view(np.float32).astype(np.float64)
    if dtype == F16:
        return raw.view(np.float16).astype(np.float64)
    t = torch.from_numpy(raw.view(np.int16).copy()).view(torch.bfloat16)
    return t.double().numpy()


def isclose_mask(c64: np.ndarray, r64: np.ndarray, atol: float, rtol: float, equal_nan=False):
    return torch.isclose(torch.from_numpy(c64), torch.from_numpy(r64), rtol=rtol, atol=atol,
                         equal_nan=bool(equal_nan)).numpy()


def to_raw16(x: np.ndarray, dtype: int) -> np.ndarray:
    if dtype == F16:
        return x.astype(np.float16).view(np.uint16)
    t = torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def random_pairs(rng: np.random.Generator, n: int, dtype: int):
    """Raw cand/ref storage mixing random bit patterns (all classes: NaN,
    +-Inf, +-0, subnormals, huge) with near pairs around the tolerance."""
    if dtype == F32:
        bits = rng.integers(0, 2**32, size=n, dtype=np.uint64).astype(np.uint32)
        r = rng.standard_normal(n).astype(np.float32)
        scale = rng.choice(np.array([1e-7, 1e-5, 1e-4, 1e-3, 1e-2, 1.0], dtype=np.float32), n)
        c = (r + scale * rng.standard_normal(n).astype(np.float32)).astype(np.float32)
        ref = r.view(np.uint32).copy()
        cand = c.view(np.uint32).copy()
        sel = rng.random(n) < 0.2
        ref[sel] = bits[sel]
        sel2 = rng.random(n) < 0.2
        cand[sel2] = rng.integers(0, 2**32, size=int(sel2.sum()), dtype=np.uint64).astype(np.uint32)
        same = rng.random(n) < 0.1
        cand[same] = ref[same]
        specials = np.array([0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000,
                             0x00000001, 0x807FFFFF, 0x7F7FFFFF, 0xFF7FFFFF], dtype=np.uint32)
        pick = rng.random(n) < 0.05
        ref[pick] = rng.choice(specials, int(pick.sum()))
        pick = rng.random(n) < 0.05
        cand[pick] = rng.choice(specials, int(pick.sum()))
        return cand, ref
    r = rng.standard_normal(n).astype(np.float32) * rng.choice([1e-6, 1e-2, 1.0, 100.0], n)
    scale = rng.choice(np.array([1e-4, 1e-3, 1e-2, 1e-1], dtype=np.float32), n)
    c = r + scale * rng.standard_normal(n).astype(np.float32)
    ref = to_raw16(r, dtype)
    cand = to_raw16(c, dtype)
    sel = rng.random(n) < 0.2
    ref[sel] = rng.integers(0, 2**16, size=int(sel.sum()), dtype=np.uint32).astype(np.uint16)
    sel = rng.random(n) < 0.2
    cand[sel] = rng.integers(0, 2**16, size=int(sel.sum()), dtype=np.uint32).astype(np.uint16)
    same = rng.random(n) < 0.1
    cand[same] = ref[same]
    return cand, ref


def as_storage(raw: np.ndarray, dtype: int) -> np.ndarray:
    return raw.view(np.float32) if dtype == F32 else raw.view(np.uint16)


def mismatch_map(lib, cand, ref, dtype, shape, tols, primary=0):
    """Per-element mismatch (0/1) at the primary pair, read from 1x1 tiles."""
    res = oracle.validate_case(as_storage(cand, dtype), as_storage(ref, dtype), dtype, shape, tols,
                               primary=primary, tile=(1, 1), lib=lib)
    return res, res.tile_map.astype(np.int64)


# -------------------------------------------------------------------- pins
def pin_decode(lib):
    """Decode equals numpy/torch conversions for every 16-bit pattern and a
    spread of binary32 patterns (NaN positions and zero signs included)."""
    rng = np.random.default_rng(1)
    cases = [
        (F16, np.arange(65536, dtype=np.uint32).astype(np.uint16)),
        (BF16, np.arange(65536, dtype=np.uint32).astype(np.uint16)),
        (F32, np.concatenate([
            rng.integers(0, 2**32, size=200000, dtype=np.uint64).astype(np.uint32),
            np.array([0, 0x80000000, 1, 0x807FFFFF, 0x00800000, 0x7F7FFFFF, 0x7F800000,
                      0xFF800000, 0x7FC00000, 0x7F800001], dtype=np.uint32)])),
    ]
    for dtype, raw in cases:
        got = oracle.decode(as_storage(raw, dtype), dtype, lib=lib)
        want = lib_decode(raw, dtype)
        nan_g, nan_w = np.isnan(got), np.isnan(want)
        assert np.array_equal(nan_g, nan_w), "decode NaN positions (dtype %d)" % dtype
        ok = ~nan_w
        assert np.array_equal(got[ok], want[ok]), "decode values (dtype %d)" % dtype
        assert np.array_equal(np.signbit(got[ok]), np.signbit(want[ok])), "decode signs"


def pin_gate_isclose(lib):
    """Per-element gate equals torch.isclose on binary64 values, for every
    dtype, several tolerance pairs and both equal_nan settings."""
    rng = np.random.default_rng(2)
    tol_sets = [(1e-5, 1e-5, 0), (1e-3, 1e-3, 1), (0.0, 1e-2, 0), (1e-2, 0.0, 1), (0.0, 0.0, 0),
                (1e-2, 1.6e-2, 0), (3.0, 0.5, 1)]
    for dtype in (F32, F16, BF16):
        n = 6 * 1024
        cand, ref = random_pairs(rng, n, dtype)
        c64, r64 = lib_decode(cand, dtype), lib_decode(ref, dtype)
        for p, t in enumerate(tol_sets):
            res, mm = mismatch_map(lib, cand, ref, dtype, (96, 64), tol_sets, primary=p)
            want = ~isclose_mask(c64, r64, t[0], t[1], t[2])
            assert np.array_equal(mm.astype(bool), want), "gate dtype %d pair %d" % (dtype, p)
            assert res.mismatches[p] == int(want.sum()), "mismatch count dtype %d pair %d" % (dtype, p)


def pin_gate_ties(lib):
    """Hand-built exact threshold cases (values exact in binary32 and binary64):
    d == atol + rtol*|r| passes, one ulp beyond fails, +-0 are equal,
    same-sign infinities are close, NaN never is unless equal_nan."""
    inf, nan = float("inf"), float("nan")
    one_ulp = float(np.nextafter(np.float32(1.5), np.float32(2)))
    ref = np.array([1.0, 1.0, 1.0, -1.0, 0.0, -0.0, inf, inf, -inf, 5.0, nan, nan, 2.0, 0.0],
                   dtype=np.float32)
    cand = np.array([1.5, one_ulp, 0.5, -1.5, -0.0, 0.0, inf, -inf, 5.0, inf, nan, 1.0, 2.5, 0.25],
                    dtype=np.float32)
    # atol = 0.25, rtol = 0.25: t(1) = 0.5, t(2) = 0.75, t(0) = 0.25
    expect_plain = [0, 1, 0, 0, 0, 0, 0, 1, 1, 1, 1, 1, 0, 0]
    expect_eqnan = [0, 1, 0, 0, 0, 0, 0, 1, 1, 1, 0, 1, 0, 0]
    for eqn, expect in ((0, expect_plain), (1, expect_eqnan)):
        res, mm = mismatch_map(lib, cand.view(np.uint32), ref.view(np.uint32), F32, (1, 14),
                               [(0.25, 0.25, eqn)])
        assert mm.tolist() == expect, "ties equal_nan=%d: %s" % (eqn, mm.tolist())
    # 16-bit: fp16 1.0 vs 1.0 + 2^-10 with atol 2^-10, rtol 0 -> close; 2^-9 -> not
    r16 = np.array([1.0, 1.0, 1.0], dtype=np.float16)
    c16 = np.array([1.0 + 2**-10, 1.0 + 2**-9, 1.0 - 2**-11], dtype=np.float16)
    res, mm = mismatch_map(lib, c16.view(np.uint16), r16.view(np.uint16), F16, (3,),
                           [(2.0**-10, 0.0, 0)])
    assert mm.tolist() == [0, 1, 0], "fp16 ties"


def _fma(a: float, b: float, c: float) -> float:
    return float(Fraction(a) * Fraction(b) + Fraction(c))


def pin_no_fma(lib):
    """Where a fused atol + rtol*|r| would flip the decision, the oracle
    follows the separately rounded sum (torch.isclose computes it that way)."""
    rng = np.random.default_rng(3)
    rows = []
    tries = 0
    while len(rows) < 48 and tries < 200000:
        tries += 1
        r = float(np.float32(rng.uniform(0.5, 2.0)))
        c = float(np.float32(r + rng.uniform(1e-4, 1e-2)))
        d = abs(c - r)
        rtol = float(rng.uniform(1e-6, 1e-3))
        a0 = d - rtol * abs(r)
        for step in range(-4, 5):
            atol = float(np.nextafter(a0, np.inf) if step > 0 else a0)
            for _ in range(abs(step) - 1 if step > 0 else -step):
                atol = float(np.nextafter(atol, np.inf if step > 0 else -np.inf))
            if atol < 0:
                continue
            t_sep = atol + rtol * abs(r)
            t_fma = _fma(rtol, abs(r), atol)
            if (d <= t_sep) != (d <= t_fma):
                rows.append((c, r, atol, rtol))
    assert len(rows) >= 16, "too few fma-sensitive cases found"
    cand = np.array([x[0] for x in rows], dtype=np.float32)
    ref = np.array([x[1] for x in rows], dtype=np.float32)
    for i, (c, r, atol, rtol) in enumerate(rows):
        res, mm = mismatch_map(lib, cand[i:i + 1].view(np.uint32), ref[i:i + 1].view(np.uint32),
                               F32, (1,), [(atol, rtol, 0)])
        want = ~isclose_mask(np.array([c]), np.array([r]), atol, rtol)
        assert bool(mm[0]) == bool(want[0]), "fma-sensitive case %r" % ((c, r, atol, rtol),)


def _metrics_expect(c64: np.ndarray, r64: np.ndarray) -> dict:
    fin = np.isfinite(c64) & np.isfinite(r64)
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        d = np.abs(c64 - r64)
        relok = fin & (r64 != 0)
        q = np.where(relok, d / np.where(relok, np.abs(r64), 1.0), 0.0)
    out = {
        "nan_cand": int(np.isnan(c64).sum()), "inf_cand": int(np.isinf(c64).sum()),
        "nan_ref": int(np.isnan(r64).sum()), "inf_ref": int(np.isinf(r64).sum()),
        "n_finite": int(fin.sum()), "n_rel": int(relok.sum()),
        "n_rel_undef": int((fin & (r64 == 0) & (c64 != 0)).sum()),
        "sum_abs": math.fsum(d[fin].tolist()), "sum_rel": math.fsum(q[relok].tolist()),
    }
    if fin.any():
        da = np.where(fin, d, -1.0)
        out["argmax_abs"] = int(np.argmax(da))
        out["max_abs"] = float(da[out["argmax_abs"]])
    else:
        out["argmax_abs"], out["max_abs"] = -1, 0.0
    if relok.any():
        qa = np.where(relok, q, -1.0)
        out["argmax_rel"] = int(np.argmax(qa))
        out["max_rel"] = float(qa[out["argmax_rel"]])
    else:
        out["argmax_rel"], out["max_rel"] = -1, 0.0
    return out


def _check_metrics(st: dict, want: dict, tag: str):
    for key in ("nan_cand", "inf_cand", "nan_ref", "inf_ref", "n_finite", "n_rel", "n_rel_undef",
                "argmax_abs", "argmax_rel"):
        assert st[key] == want[key], "%s %s: %r != %r" % (tag, key, st[key], want[key])
    for key in ("max_abs", "max_rel"):
        assert st[key] == want[key], "%s %s: %r != %r" % (tag, key, st[key], want[key])
    for key in ("sum_abs", "sum_rel"):
        w = want[key]
        assert abs(st[key] - w) <= 1e-9 * abs(w) + 1e-300, "%s %s: %r vs fsum %r" % (
            tag, key, st[key], w)


def pin_metrics_numpy(lib):
    """Counts, max/argmax (first occurrence), and sums (math.fsum) against
    numpy on random, special-value and tie-heavy data."""
    rng = np.random.default_rng(4)
    for dtype in (F32, F16, BF16):
        cand, ref = random_pairs(rng, 4096, dtype)
        res = oracle.validate_case(as_storage(cand, dtype), as_storage(ref, dtype), dtype, (4096,),
                                   [(1e-3, 1e-3, 0)], lib=lib)
        _check_metrics(res.stats, _metrics_expect(lib_decode(cand, dtype), lib_decode(ref, dtype)),
                       "random dtype %d" % dtype)
    # tie-heavy: values from a tiny set so many d and q coincide
    vals = np.array([-2.0, -1.0, -0.5, 0.0, 0.5, 1.0, 2.0, 4.0], dtype=np.float32)
    ref = rng.choice(vals, 3000).astype(np.float32)
    cand = rng.choice(vals, 3000).astype(np.float32)
    res = oracle.validate_case(cand, ref, F32, (3000,), [(0.0, 0.0, 0)], lib=lib)
    _check_metrics(res.stats, _metrics_expect(cand.astype(np.float64), ref.astype(np.float64)),
                   "ties")
    # identical tensors: zero error everywhere, argmax at the first finite pair
    ref = rng.standard_normal(777).astype(np.float32)
    res = oracle.validate_case(ref, ref.copy(), F32, (777,), [(0.0, 0.0, 0)], tile=(8, 8), k=5,
                               lib=lib)
    st = res.stats
    assert st["mismatches"] == 0 and st["max_abs"] == 0.0 and st["argmax_abs"] == 0
    assert st["max_rel"] == 0.0 and st["argmax_rel"] == 0 and st["sum_abs"] == 0.0
    assert res.first_k.tolist() == [-1] * 5 and int(res.tile_map.sum()) == 0
    # no finite pairs at all
    nanv = np.full(10, np.nan, dtype=np.float32)
    res = oracle.validate_case(nanv, nanv.copy(), F32, (10,), [(1.0, 1.0, 0)], lib=lib)
    assert res.stats["argmax_abs"] == -1 and res.stats["max_abs"] == 0.0
    assert res.stats["argmax_rel"] == -1 and res.stats["n_finite"] == 0
    assert res.stats["mismatches"] == 10 and res.stats["nan_cand"] == 10


def _tile_expect(mask2d: np.ndarray, th: int, tw: int) -> np.ndarray:
    rows, cols = mask2d.shape
    tr, tc = -(-rows // th), -(-cols // tw)
    pad = np.zeros((tr * th, tc * tw), dtype=np.int64)
    pad[:rows, :cols] = mask2d
    return pad.reshape(tr, th, tc, tw).sum(axis=(1, 3)).reshape(-1)


def pin_localize_numpy(lib):
    """Tile map equals a padded reshape-sum of the isclose mask; first-k equals
    numpy's ascending nonzero indices, -1 padded; ragged shapes included."""
    rng = np.random.default_rng(5)
    shapes = [(37, 53), (1, 1000), (1000, 1), (64, 64), (7, 3, 11), (5,), (), (130, 67)]
    tiles = [(8, 16), (1, 64), (64, 1), (32, 32), (4, 5), (1, 1), (1, 1), (64, 64)]
    for shape, (th, tw) in zip(shapes, tiles):
        n = int(np.prod(shape)) if shape else 1
        for dtype in (F32, BF16):
            cand, ref = random_pairs(rng, n, dtype)
            rows, cols = oracle.view_rows_cols(shape)
            for k in (0, 3, 64, n + 5):
                res = oracle.validate_case(as_storage(cand, dtype), as_storage(ref, dtype), dtype,
                                           shape, [(1e-2, 1e-2, 0), (1e-3, 1e-3, 1)], primary=1,
                                           tile=(th, tw), k=k, lib=lib)
                mask = ~isclose_mask(lib_decode(cand, dtype), lib_decode(ref, dtype), 1e-3, 1e-3, 1)
                want_t = _tile_expect(mask.reshape(rows, cols).astype(np.int64), th, tw)
                assert np.array_equal(res.tile_map.astype(np.int64), want_t), "tile %r" % (shape,)
                nz = np.flatnonzero(mask)[:k]
                want_k = np.concatenate([nz, -np.ones(k - nz.size, dtype=np.int64)])
                assert np.array_equal(res.first_k, want_k), "first-k %r k=%d" % (shape, k)


def pin_invariants(lib):
    """Sum of tile map == mismatches; counts monotone in the tolerance;
    counts of a concatenation are the sum of the parts."""
    rng = np.random.default_rng(6)
    tols = [(1e-7, 1e-7, 0), (1e-5, 1e-5, 0), (1e-3, 1e-3, 0), (1e-1, 1e-1, 0)]
    cand, ref = random_pairs(rng, 5000, F32)
    c, r = cand.view(np.float32), ref.view(np.float32)
    full = oracle.validate_case(c, r, F32, (50, 100), tols, primary=2, tile=(7, 9), lib=lib)
    assert int(full.tile_map.sum()) == full.mismatches[2]
    assert all(a >= b for a, b in zip(full.mismatches, full.mismatches[1:])), full.mismatches
    a = oracle.validate_case(c[:1234], r[:1234], F32, (1234,), tols, lib=lib)
    b = oracle.validate_case(c[1234:], r[1234:], F32, (3766,), tols, lib=lib)
    whole = oracle.validate_case(c, r, F32, (5000,), tols, lib=lib)
    assert [x + y for x, y in zip(a.mismatches, b.mismatches)] == whole.mismatches
    for key in ("nan_cand", "inf_cand", "nan_ref", "inf_ref", "n_finite", "n_rel", "n_rel_undef"):
        assert a.stats[key] + b.stats[key] == whole.stats[key], key


def pin_fp32_single(lib):
    """Closed form of workload 1 at full size: 1536 mismatches (rows
    1000-1023 x cols 960-1023), first 64 = 1024960..1025023, tile map 768 at
    tiles (31,30) and (31,31) and 0 elsewhere, max_abs = max |ref| over the
    zeroed block."""
    w = wl.fp32_single(device="cpu")
    case = w.cases[0]
    cand, ref = case.cand.numpy(), case.ref.numpy()
    block = np.abs(ref[1000:, 960:].astype(np.float64))
    assert block.min() > 2e-5  # every zeroed element is a definite mismatch for this seed
    res = oracle.validate_case(cand, ref, F32, (1024, 1024), w.tols, tile=w.tile, k=w.k, lib=lib)
    st = res.stats
    assert st["mismatches"] == 1536 and res.mismatches == [1536]
    assert res.first_k.tolist() == list(range(1024960, 1025024))
    tm = res.tile_map.reshape(32, 32)
    assert tm[31, 30] == 768 and tm[31, 31] == 768 and int(tm.sum()) == 1536
    assert st["max_abs"] == float(block.max())
    assert st["nan_cand"] == st["inf_cand"] == 0 and st["n_finite"] == 1024 * 1024


def pin_fp16_batch(lib):
    """Workload 2 structure (4 cases of 256x256): per case 4096 shifted-tile
    mismatches + 3 NaNs = 4099, nan_cand = 3, tile map = 4096 at the shifted
    tile plus one per NaN in its tile; first-k = the smallest fault indices."""
    w = wl.fp16_batch(device="cpu", n_cases=4, rows=256, cols=256)
    for case, f in zip(w.cases, w.meta["faults"]):
        cand, ref = wl.raw_numpy(case.cand), wl.raw_numpy(case.ref)
        res = oracle.validate_case(cand, ref, F16, (256, 256), w.tols, tile=w.tile, k=w.k, lib=lib)
        assert res.mismatches == [4099] and res.stats["nan_cand"] == 3
        ti, tj = f["tile"]
        want = np.zeros((4, 4), dtype=np.int64)
        want[ti, tj] = 4096
        for p in f["nans"]:
            want[(p // 256) // 64, (p % 256) // 64] += 1
        assert np.array_equal(res.tile_map.reshape(4, 4), want)
        tile_idx = [(ti * 64 + a) * 256 + tj * 64 + b for a in range(64) for b in range(64)]
        expect_k = sorted(set(tile_idx) | set(f["nans"].tolist()))[:64]
        assert res.first_k.tolist() == expect_k


def pin_bf16_bursts(lib):
    """Workload 3 structure (2x256x512 bf16): inf_cand = 512 and mismatches =
    512 + the scaled faults that torch.isclose rejects; the rest is
    bit-identical, so max_abs is attained at a scaled fault."""
    w = wl.bf16_bursts(device="cpu", shape=(2, 256, 512), fault_fraction=1e-4)
    case = w.cases[0]
    cand, ref = wl.raw_numpy(case.cand).reshape(-1), wl.raw_numpy(case.ref).reshape(-1)
    res = oracle.validate_case(cand, ref, BF16, (2, 256, 512), w.tols, tile=w.tile, k=w.k, lib=lib)
    sc = w.meta["scaled"]
    c64, r64 = lib_decode(cand[sc], BF16), lib_decode(ref[sc], BF16)
    bad = ~isclose_mask(c64, r64, 1e-2, 1.6e-2)
    assert res.stats["inf_cand"] == 512
    assert res.mismatches == [512 + int(bad.sum())]
    d = np.abs(c64 - r64)
    assert res.stats["max_abs"] == float(d.max())
    s0 = w.meta["burst"][0]
    fails = sorted(set(range(s0, s0 + 512)) | set(sc[bad].tolist()))
    assert res.first_k.tolist() == fails[:64]


def pin_fp32_sweep(lib):
    """Workload 4 structure (40 odd-shaped cases, 2^14 elements max): at
    pairs 1e-4 and 1e-3 the mismatches are exactly the injected faults, which
    all sit in the last tile; first-k lists them; counts are monotone across
    the 4 pairs; the suite match rate at (1e-3, 1e-3) is 20/40."""
    w = wl.fp32_sweep(device="cpu", n_cases=40, max_log2=14, n_cauchy=4, n_faulted=20,
                   fixed=[(1, 7), (3, 1003), (257, 51), (1, 1)])
    mism, status = [], []
    for i, case in enumerate(w.cases):
        r, c = case.ref.shape
        res = oracle.validate_case(case.cand.numpy(), case.ref.numpy(), F32, (r, c), w.tols,
                                   primary=3, tile=w.tile, k=w.k, lib=lib)
        faults = w.meta["faults"][i]
        assert res.mismatches[2] == res.mismatches[3] == len(faults), (i, res.mismatches)
        assert all(a >= b for a, b in zip(res.mismatches, res.mismatches[1:]))
        assert res.first_k[:len(faults)].tolist() == faults.tolist()
        tm = res.tile_map
        assert int(tm[:-1].sum()) == 0 and int(tm[-1]) == len(faults)
        mism.append(res.mismatches)
        status.append(0)
    pas, rate = oracle.suite(np.array(mism, dtype=np.uint64), status, lib=lib)
    assert rate[3] == 0.5 and rate[2] == 0.5, rate
    assert all(a <= b for a, b in zip(rate, rate[1:])), rate


def pin_fp32_integrity(lib):
    """Workload 5 classes (20 cases of 64x64): each class raises exactly its
    flag (correct: none, copy: INPUT_COPY with copy_input 0, zero: ALL_ZERO,
    constant: CONSTANT, bf16: LOWPREC_BF16); the zero class has max_rel 1.0
    and sum_abs = fsum |ref|; the certified match rate is #correct / 20."""
    w = wl.fp32_integrity(device="cpu", n_cases=20, rows=64, cols=64)
    want_flag = {wl.CLASS_CORRECT: 0, wl.CLASS_COPY: oracle.FLAG_INPUT_COPY,
                 wl.CLASS_ZERO: oracle.FLAG_ALL_ZERO, wl.CLASS_CONSTANT: oracle.FLAG_CONSTANT,
                 wl.CLASS_BF16: oracle.FLAG_LOWPREC_BF16}
    mism, flags = [], []
    for case, k in zip(w.cases, w.meta["classes"]):
        x = case.inputs[0].numpy()
        res = oracle.validate_case(case.cand.numpy(), case.ref.numpy(), F32, (64, 64), w.tols,
                                   inputs=[(x, F32)], lib=lib)
        integ = res.integrity
        assert integ["flags"] == want_flag[int(k)], (int(k), integ["flags"])
        assert integ["copy_input"] == (0 if k == wl.CLASS_COPY else -1)
        assert integ["cand_eq_input_mask"] == (1 if k == wl.CLASS_COPY else 0)
        assert integ["ref_eq_input_mask"] == 0
        if k == wl.CLASS_ZERO:
            assert res.stats["max_rel"] == 1.0
            ref64 = case.ref.numpy().astype(np.float64)
            want = math.fsum(np.abs(ref64).ravel().tolist())
            assert abs(res.stats["sum_abs"] - want) <= 1e-9 * want
        if k == wl.CLASS_CORRECT:
            assert res.mismatches == [0]
        mism.append(res.mismatches)
        flags.append(integ["flags"])
    n_correct = int((w.meta["classes"] == wl.CLASS_CORRECT).sum())
    pas, rate = oracle.suite(np.array(mism, dtype=np.uint64), [0] * 20, flags, lib=lib)
    assert rate[0] == n_correct / 20, (rate, n_correct)


def pin_integrity_counts(lib):
    """Detector counts against numpy: zeros (+-0), bit-equality with element 0,
    bf16 representability (torch round trip, bitwise) and fp16
    representability (numpy round trip, NaN counted representable), for
    values built to exercise every branch; bit-equality masks vs numpy."""
    rng = np.random.default_rng(7)
    n = 6000
    base = rng.standard_normal(n).astype(np.float32)
    kinds = rng.integers(0, 8, n)
    v = base.copy()
    v[kinds == 1] = 0.0
    v[kinds == 2] = -0.0
    v[kinds == 3] = np.float16(base[kinds == 3]).astype(np.float32)  # fp16 normals
    sub = rng.integers(1, 1024, int((kinds == 4).sum())).astype(np.float64) * 2.0**-24
    v[kinds == 4] = sub.astype(np.float32)  # fp16 subnormals, odd multiples included
    bf = torch.from_numpy(base[kinds == 5]).to(torch.bfloat16).float().numpy()
    v[kinds == 5] = bf
    v[kinds == 6] = np.array([65504.0, 65520.0, 1e5, 2.0**-25, 3 * 2.0**-26, np.inf, np.nan,
                              6e-8, 65536.0, -65536.0, 98304.0],
                             dtype=np.float32)[rng.integers(0, 11, int((kinds == 6).sum()))]
    # one fraction bit finer than the binary16 grid (pattern ends in 0x1000)
    half_grid = np.float16(base[kinds == 0]).astype(np.float32)
    v[kinds == 0] = (half_grid.view(np.uint32) | np.uint32(0x1000)).view(np.float32)
    v[kinds == 7] = v[0]
    cand = v
    ref = np.where(rng.random(n) < 0.5, v, base).astype(np.float32)
    x1 = cand.copy()
    x0 = rng.standard_normal(n).astype(np.float32)
    x2 = ref.copy()
    x3 = np.zeros(n, dtype=np.uint16)  # different dtype: never eligible
    res = oracle.validate_case(cand, ref, F32, (n,), [(1e-3, 1e-3, 0)],
                               inputs=[(x0, F32), (x1, F32), (x2, F32), (x3, F16)], lib=lib)
    integ = res.integrity

    def bits(a):
        return a.view(np.uint32)

    def bf16rep(a):
        # torch's round trip is bit-exact for every non-NaN value; it rewrites
        # NaN payloads, so a NaN counts when its pattern is a bf16 pattern.
        rt = torch.from_numpy(a.copy()).to(torch.bfloat16).float().numpy()
        nan_kept = np.isnan(a) & ((bits(a) >> 16) << 16 == bits(a))
        return (bits(rt) == bits(a)) | nan_kept

    def fp16rep(a):
        with np.errstate(over="ignore"):
            rt = a.astype(np.float16).astype(np.float32)
        return (rt == a) | np.isnan(a)

    for side, a in (("cand", cand), ("ref", ref)):
        assert integ["zero_" + side] == int((a == 0).sum()), "zero_" + side
        assert integ["eqfirst_" + side] == int((bits(a) == bits(a)[0]).sum()), "eqfirst_" + side
        assert integ["bf16rep_" + side] == int(bf16rep(a).sum()), "bf16rep_" + side
        assert integ["fp16rep_" + side] == int(fp16rep(a).sum()), "fp16rep_" + side
    assert integ["cand_eq_input_mask"] == 0b0010 | (0b0100 if np.array_equal(bits(cand), bits(ref)) else 0)
    assert integ["ref_eq_input_mask"] == 0b0100 | (0b0010 if np.array_equal(bits(cand), bits(ref)) else 0)
    assert integ["cand_eq_ref"] == int(np.array_equal(bits(cand), bits(ref)))
    # 16-bit storage: zero and eqfirst only; representability counters stay 0
    c16 = np.array([0.0, -0.0, 1.0, 1.0], dtype=np.float16).view(np.uint16)
    r16 = np.array([1.0, 2.0, 3.0, 4.0], dtype=np.float16).view(np.uint16)
    res = oracle.validate_case(c16, r16, F16, (4,), [(0.0, 0.0, 0)], inputs=[], lib=lib)
    integ = res.integrity
    assert (integ["zero_cand"], integ["eqfirst_cand"], integ["zero_ref"]) == (2, 1, 0)
    assert integ["bf16rep_cand"] == integ["fp16rep_cand"] == 0


def pin_flags_handbuilt(lib):
    """Literal detector outcomes on small hand-built cases."""
    def flags(cand, ref, inputs=(), dtype=F32):
        res = oracle.validate_case(cand, ref, dtype, (len(cand),), [(1e-5, 1e-5, 0)],
                                   inputs=list(inputs), lib=lib)
        return res.integrity["flags"], res.integrity["copy_input"]

    f32 = lambda a: np.array(a, dtype=np.float32)  # noqa: E731
    x = f32([0.3, -1.2, 2.5, 7.0])
    ref = f32([1.15, 0.4, 2.25, 4.5])
    assert flags(f32([0, 0, 0, 0]), ref) == (oracle.FLAG_ALL_ZERO, -1)
    assert flags(f32([0, -0.0, 0, -0.0]), ref) == (oracle.FLAG_ALL_ZERO, -1)
    assert flags(f32([0, 0, 0, 0]), f32([0, 0, 0, 0])) == (0, -1)  # legitimately zero output
    assert flags(f32([2, 2, 2, 2]), ref) == (oracle.FLAG_CONSTANT, -1)
    assert flags(f32([2, 2, 2, 2]), f32([2, 2, 2, 2])) == (0, -1)
    assert flags(f32([np.nan] * 4), ref) == (oracle.FLAG_CONSTANT, -1)
    assert flags(f32([3.0]), f32([1.0])) == (0, -1)  # n = 1: no constant verdict
    assert flags(x.copy(), ref, [(x, F32)]) == (oracle.FLAG_INPUT_COPY, 0)
    assert flags(x.copy(), x.copy(), [(x, F32)]) == (0, -1)  # identity operator
    assert flags(x.copy(), ref, [(ref, F32), (x, F32)]) == (oracle.FLAG_INPUT_COPY, 1)
    assert flags(x.copy(), ref, [(x[:3], F32)]) == (0, -1)  # size differs: not eligible
    zeros16 = np.zeros(8, dtype=np.uint16)  # 16-bit input, same numel: not eligible
    assert flags(f32([0, 0, 0, 0]), ref, [(zeros16[:4], F16)]) == (oracle.FLAG_ALL_ZERO, -1)
    assert flags(f32([1.5, 0.375, 3.0, -0.75]), ref) == (oracle.FLAG_LOWPREC_BF16, -1)
    half_vals = np.array([1.0009765625, 0.3333, 2.252, 4.496], dtype=np.float16).astype(np.float32)
    assert flags(half_vals, ref) == (oracle.FLAG_LOWPREC_FP16, -1)
    assert flags(half_vals, half_vals.copy()) == (0, -1)


def pin_suite_handbuilt(lib):
    """Literal per-case pass bits and certified match rates."""
    mism = np.array([[0, 0], [3, 0], [0, 0], [5, 0]], dtype=np.uint64)
    pas, rate = oracle.suite(mism, [0, 0, -3, 0], [0, 0, 0, 4], lib=lib)
    assert pas.tolist() == [[1, 1], [0, 1], [0, 0], [0, 1]]
    assert rate.tolist() == [0.25, 0.5]  # case 3 passes at pair 1 but is flagged
    pas, rate = oracle.suite(mism, [0, 0, 0, 0], None, lib=lib)
    assert rate.tolist() == [0.5, 1.0]


def _tstats_expected(raw: np.ndarray, dtype: int) -> dict:
    """Tensor statistics from numpy / torch conversions, numpy reductions,
    frexp and math.fsum (an independent route to every field)."""
    v = lib_decode(raw, dtype).reshape(-1)
    fin = np.isfinite(v)
    fv = v[fin]
    idx = np.flatnonzero(fin)
    e = {"numel": v.size, "nan": int(np.isnan(v).sum()), "inf": int(np.isinf(v).sum()),
         "zero": int((fv == 0).sum()), "n_finite": int(fin.sum())}
    if fv.size:
        e["argmin"] = int(idx[np.argmin(fv)])  # first occurrence
        e["argmax"] = int(idx[np.argmax(fv)])
        e["min"], e["max"] = v[e["argmin"]], v[e["argmax"]]
    else:
        e["argmin"] = e["argmax"] = -1
        e["min"] = e["max"] = 0.0
    nz = fv[fv != 0]
    ex = np.frexp(nz)[1].astype(np.int64) - 1
    bins = np.clip(ex - oracle.HIST_EMIN + 1, 0, oracle.HIST_BINS - 1)
    e["hist"] = np.bincount(bins, minlength=oracle.HIST_BINS).tolist()
    e["fsum"] = (math.fsum(fv.tolist()), math.fsum((fv * fv).tolist()),
                 math.fsum(np.abs(fv).tolist()))
    e["abs_total"] = (math.fsum(np.abs(fv).tolist()), math.fsum((fv * fv).tolist()))
    return e


def _check_tstats(got: dict, e: dict) -> None:
    for k in ("numel", "nan", "inf", "zero", "n_finite", "argmin", "argmax", "hist"):
        assert got[k] == e[k], (k, got[k], e[k])
    for k in ("min", "max"):
        # the value of the element itself, sign of zero included
        assert np.float64(got[k]).tobytes() == np.float64(e[k]).tobytes(), (k, got[k], e[k])
    # a sum in index order is within n * 2^-53 * sum|terms| of the exact sum
    n = max(e["n_finite"], 1)
    bound = n * 2.0 ** -53
    for k, exact, mag in (("sum", e["fsum"][0], e["abs_total"][0]),
                          ("sum_sq", e["fsum"][1], e["abs_total"][1]),
                          ("sum_abs", e["fsum"][2], e["abs_total"][0])):
        assert abs(got[k] - exact) <= bound * mag, (k, got[k], exact)


def pin_tstats_numpy(lib):
    """Tensor statistics of random bit patterns of every dtype (NaN, +-Inf,
    +-0, subnormals, huge values) and of normal data, against numpy."""
    rng = np.random.default_rng(26081)
    for dt in (F32, F16, BF16):
        for n in (0, 1, 7, 1000, 4099):
            cand, ref = random_pairs(rng, n, dt)
            for raw in (cand, ref):
                got = oracle.tensor_stats(as_storage(raw, dt), dt, lib=lib)
                _check_tstats(got, _tstats_expected(raw, dt))


def pin_tstats_handbuilt(lib):
    """Literal tensor statistics of hand-built tensors."""
    x = np.array([1.0, -0.0, 0.0, np.nan, np.inf, 0.75, -3.0, 65504, 2.0 ** -24, 1e-30, 1e30,
                  -3.0], dtype=np.float32)
    d = oracle.tensor_stats(x, F32, lib=lib)
    assert (d["nan"], d["inf"], d["zero"], d["n_finite"]) == (1, 1, 2, 10)
    assert (d["min"], d["argmin"]) == (-3.0, 6)  # the first of the two -3
    assert (d["max"], d["argmax"]) == (float(np.float32(1e30)), 10)
    # exponents: 1 -> 0, 0.75 -> -1, -3 -> 1 (twice), 65504 -> 15, 2^-24 -> -24,
    # 1e-30 -> -100 (first bin), 1e30 -> 99 (last bin)
    want = {41: 1, 40: 1, 42: 2, 56: 1, 17: 1, 0: 1, 63: 1}
    assert {i: c for i, c in enumerate(d["hist"]) if c} == want
    # zeros only: the first zero is both extremes, with its own sign
    z = np.array([-0.0, 0.0, 0.0], dtype=np.float32)
    d = oracle.tensor_stats(z, F32, lib=lib)
    assert d["argmin"] == d["argmax"] == 0 and math.copysign(1.0, d["min"]) == -1.0
    assert d["zero"] == 3 and sum(d["hist"]) == 0
    # nothing finite
    d = oracle.tensor_stats(np.array([np.nan, -np.inf], dtype=np.float32), F32, lib=lib)
    assert (d["n_finite"], d["argmin"], d["argmax"], d["min"], d["sum"]) == (0, -1, -1, 0.0, 0.0)
    # binary16: the smallest subnormal, the largest finite value, 1.5
    h = np.array([2.0 ** -24, 65504.0, 1.5], dtype=np.float16).view(np.uint16)
    d = oracle.tensor_stats(h, F16, lib=lib)
    assert {i: c for i, c in enumerate(d["hist"]) if c} == {17: 1, 56: 1, 41: 1}
    assert d["sum"] == 2.0 ** -24 + 65504.0 + 1.5
    # bfloat16: a subnormal (exponent -133) and -2
    b = np.array([0x0001, 0xC000], dtype=np.uint16)
    d = oracle.tensor_stats(b, BF16, lib=lib)
    assert {i: c for i, c in enumerate(d["hist"]) if c} == {0: 1, 42: 1}
    assert (d["min"], d["argmin"], d["max"], d["argmax"]) == (-2.0, 1, 2.0 ** -133, 0)
    assert d["sum_sq"] == 4.0 + 2.0 ** -266 and d["sum_abs"] == 2.0 + 2.0 ** -133
    d = oracle.tensor_stats(np.zeros(0, dtype=np.uint16), F16, lib=lib)
    assert d["numel"] == 0 and d["argmin"] == -1


def _nearpass_expected(cand, ref, dt, atol, rtol) -> dict:
    """Near-pass statistics from numpy: binary64 arithmetic on numpy / torch
    decoded values, numpy's float32 -> float16 rounding for the grid, frexp
    for the bins."""
    c = lib_decode(cand, dt).reshape(-1)
    r = lib_decode(ref, dt).reshape(-1)
    fin = np.isfinite(c) & np.isfinite(r)
    idx = np.flatnonzero(fin)
    c, r = c[fin], r[fin]
    d = np.abs(c - r)
    t = atol + rtol * np.abs(r)
    fail = d > t
    e = {"numel": cand.size, "n_pairs": int(fin.sum()), "n_fail": int(fail.sum()),
         "n_zero_tol": int(((t == 0) & (d > 0)).sum())}
    pos = t > 0
    if pos.any():
        q = np.zeros_like(d)
        q[pos] = d[pos] / t[pos]
        k = int(np.argmax(np.where(pos, q, -1.0)))  # first occurrence
        e["max_ratio"], e["argmax_ratio"] = float(q[k]), int(idx[k])
    else:
        e["max_ratio"], e["argmax_ratio"] = 0.0, -1
    qf = d[fail & pos] / t[fail & pos]
    rb = np.minimum(np.frexp(qf)[1] - 1, oracle.RATIO_BINS - 1)
    e["ratio_hist"] = np.bincount(rb, minlength=oracle.RATIO_BINS).tolist()
    if dt == F32:
        with np.errstate(over="ignore"):
            gc = c.astype(np.float32).astype(np.float16).view(np.uint16).astype(np.int64)
            gr = r.astype(np.float32).astype(np.float16).view(np.uint16).astype(np.int64)
        mask = 0x7C00
    else:
        gc = cand.reshape(-1)[fin].astype(np.int64)
        gr = ref.reshape(-1)[fin].astype(np.int64)
        mask = 0x7C00 if dt == F16 else 0x7F80
    inside = ((gc & mask) != mask) & ((gr & mask) != mask)
    key = lambda h: np.where(h & 0x8000, -(h & 0x7FFF), h & 0x7FFF)
    dist = np.abs(key(gc) - key(gr))
    bins = np.where(dist == 0, 0, np.frexp(dist.astype(np.float64))[1])
    bins = np.where(inside, bins, oracle.ULP_BINS - 1)
    e["ulp_hist"] = np.bincount(bins, minlength=oracle.ULP_BINS).tolist()
    df = np.where(inside, dist, 0xFFFFFFFF)[fail]
    e["max_ulp_fail"] = int(df.max()) if df.size else 0
    return e


def _check_nearpass(got, e):
    for k in ("numel", "n_pairs", "n_fail", "n_zero_tol", "argmax_ratio", "ratio_hist",
              "ulp_hist", "max_ulp_fail"):
        assert got[k] == e[k], (k, got[k], e[k])
    assert np.float64(got["max_ratio"]).tobytes() == np.float64(e["max_ratio"]).tobytes()


def pin_nearpass_numpy(lib):
    """Near-pass statistics of random pairs of every class and storage type,
    at several tolerances, against numpy."""
    rng = np.random.default_rng(26082)
    for dt in (F32, F16, BF16):
        for n in (0, 1, 5, 3000):
            cand, ref = random_pairs(rng, n, dt)
            for atol, rtol in ((1e-3, 1e-3), (0.0, 1e-2), (0.0, 0.0), (1e-5, 0.0)):
                got = oracle.nearpass(as_storage(cand, dt), as_storage(ref, dt), dt, atol, rtol,
                                      lib=lib)
                _check_nearpass(got, _nearpass_expected(cand, ref, dt, atol, rtol))


def pin_nearpass_handbuilt(lib):
    """Literal near-pass statistics: one binary16 step apart (the fp16
    ceiling), a zero tolerance, values beyond the binary16 range, and the
    binary16 rounding routine at its boundaries."""
    one_up = np.array([1.0 + 2.0 ** -10, 1.0], dtype=np.float16).view(np.uint16)
    d = oracle.nearpass(one_up[:1], one_up[1:], F16, 1e-4, 1e-4, lib=lib)
    # d = 2^-10, t = 2e-4: ratio 4.8828125 (bin 2), one grid step
    assert (d["n_fail"], d["max_ulp_fail"], d["argmax_ratio"]) == (1, 1, 0)
    assert d["max_ratio"] == 2.0 ** -10 / (1e-4 + 1e-4 * 1.0)
    assert d["ratio_hist"][2] == 1 and sum(d["ratio_hist"]) == 1 and d["ulp_hist"][1] == 1
    x = np.array([1e5, 1.0, 3.0], dtype=np.float32)
    y = np.array([1e5 + 8, 1.0, 3.0], dtype=np.float32)
    d = oracle.nearpass(x, y, F32, 0.0, 0.0, lib=lib)
    assert (d["n_fail"], d["n_zero_tol"], d["max_ulp_fail"]) == (1, 1, 0xFFFFFFFF)
    # t == 0 everywhere: no finite violation ratio
    assert d["ulp_hist"][0] == 2 and d["ulp_hist"][17] == 1
    assert (d["argmax_ratio"], d["max_ratio"]) == (-1, 0.0)
    # -0 and +0 are the same grid value; NaN / Inf pairs are left out
    z = np.array([-0.0, np.nan, np.inf], dtype=np.float32)
    w = np.array([0.0, 1.0, np.inf], dtype=np.float32)
    d = oracle.nearpass(z, w, F32, 1e-3, 1e-3, lib=lib)
    assert (d["n_pairs"], d["n_fail"], d["ulp_hist"][0]) == (1, 0, 1)
    # binary16 rounding: ties to even, the last finite value, the overflow threshold
    for v, h in ((1.0 + 2.0 ** -11, 0x3C00), (1.0 + 3 * 2.0 ** -11, 0x3C02), (65504.0, 0x7BFF),
                 (65519.99, 0x7BFF), (65520.0, 0x7C00), (2.0 ** -25, 0x0000),
                 (3 * 2.0 ** -25, 0x0002), (-2.0 ** -24, 0x8001)):
        assert lib.orc_round_binary16(v) == h, (v, hex(lib.orc_round_binary16(v)))


def pin_hash_splitmix(lib):
    """The finalizer against the published SplitMix64 sequence: seeded with
    0, the generator's first outputs are M(k * 0x9E3779B97F4A7C15) for
    k = 1, 2, 3 (Steele, Lea and Flood's reference values)."""
    g = 0x9E3779B97F4A7C15
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    for k, w in zip((1, 2, 3), want):
        assert lib.orc_splitmix_finalize((k * g) % 2 ** 64) == w
    assert lib.orc_splitmix_finalize(0) == 0


def pin_hash_composition(lib):
    """The content hash as the finalizer's sum over 64-bit storage words and
    its invariants: any change of a value, of the order, of the length or of
    the storage type changes it; the words depend on the bytes alone (a
    binary32 tensor and the 16-bit view of its bytes differ in the length /
    type term only); a zero tensor of four words sums the three published
    SplitMix64 outputs (M(0) = 0)."""
    m = lib.orc_splitmix_finalize
    g = 0x9E3779B97F4A7C15
    rng = np.random.default_rng(26084)
    for dt in (F32, F16, BF16):
        for n in (0, 1, 3, 4, 9, 1000):
            raw = rng.integers(0, 2 ** (32 if dt == F32 else 16), n, dtype=np.uint64).astype(
                np.uint32 if dt == F32 else np.uint16)
            h = m(0x243F6A8885A308D3 ^ (dt << 56) ^ n)
            # words built with Python integers from the little-endian bytes
            data = raw.astype('<u4' if dt == F32 else '<u2').tobytes()
            for i in range(0, len(data), 8):
                w = int.from_bytes(data[i:i + 8], 'little')
                h = (h + m(w ^ ((i // 8 * g) % 2 ** 64))) % 2 ** 64
            assert oracle.content_hash(as_storage(raw, dt), dt, lib=lib) == h
            if n >= 2:
                swapped = raw.copy()
                swapped[[0, 1]] = swapped[[1, 0]]
                if swapped[0] != swapped[1]:
                    assert oracle.content_hash(as_storage(swapped, dt), dt, lib=lib) != h
                bumped = raw.copy()
                bumped[n // 2] ^= 1
                assert oracle.content_hash(as_storage(bumped, dt), dt, lib=lib) != h
    published = (0xE220A8397B1DCDAF + 0x6E789E6AA1B965F4 + 0x06C45D188009454F) % 2 ** 64
    for dt, z in ((F32, np.zeros(8, np.float32)), (F16, np.zeros(16, np.uint16)),
                  (BF16, np.zeros(13, np.uint16))):
        meta = m(0x243F6A8885A308D3 ^ (dt << 56) ^ z.size)
        assert oracle.content_hash(z, dt, lib=lib) == (meta + published) % 2 ** 64
    # the same bytes as binary32, binary16 and bfloat16: equal word sums
    x = rng.integers(0, 2 ** 32, 37, dtype=np.uint64).astype(np.uint32)
    body = set()
    for dt, v, n in ((F32, x.view(np.float32), 37), (F16, x.view(np.uint16), 74),
                     (BF16, x.view(np.uint16), 74)):
        body.add((oracle.content_hash(v, dt, lib=lib) - m(0x243F6A8885A308D3 ^ (dt << 56) ^ n))
                 % 2 ** 64)
    assert len(body) == 1
    h16 = oracle.content_hash(np.zeros(4, np.uint16), F16, lib=lib)
    assert h16 != oracle.content_hash(np.zeros(4, np.uint16), BF16, lib=lib)
    assert h16 != oracle.content_hash(np.zeros(5, np.uint16), F16, lib=lib)


PINS = [
    pin_hash_splitmix, pin_hash_composition,
    pin_nearpass_handbuilt, pin_nearpass_numpy,
    pin_tstats_handbuilt, pin_tstats_numpy,
    pin_gate_ties, pin_suite_handbuilt, pin_flags_handbuilt, pin_decode, pin_no_fma,
    pin_metrics_numpy, pin_gate_isclose, pin_localize_numpy, pin_invariants, pin_integrity_counts,
    pin_fp32_integrity, pin_fp32_sweep, pin_fp16_batch, pin_bf16_bursts, pin_fp32_single,
]
