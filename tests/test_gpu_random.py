"""Randomized GPU parity against the oracle, with fixed seeds.

Each round draws a batch of cases: storage type, rank and shape (0-d,
empty, ragged, up to a few hundred thousand elements), data mixing random
bit patterns of every class, near pairs, shifted blocks, bursts of NaN, Inf
and signed zeros and bit-equal pairs, and random options (one to eight
tolerance pairs with or without equal_nan, primary pair, tile shape or none,
first-k length, detectors on or off). vcheck_sweep must match the oracle
field for field; the probe, near-pass and content-hash kernels are checked
on random batches the same way (misaligned views included)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins
from tests.gpu_util import assert_integrity, assert_stats, oracle_case, to_device

pytestmark = pytest.mark.gpu

DTYPES = (oracle.F32, oracle.F16, oracle.BF16)


def _store(x, dt):
    x = np.asarray(x, np.float32)
    if dt == oracle.F32:
        return x.view(np.uint32).copy()
    with np.errstate(over="ignore"):  # beyond 65504 binary16 storage holds infinities
        return oracle_pins.to_raw16(x, dt)


def _pairs(rng, n, dt):
    """Raw (cand, ref) storage of n elements, of one of four kinds."""
    kind = int(rng.integers(0, 4))
    if kind == 0 and n:
        return oracle_pins.random_pairs(rng, n, dt)
    r = (rng.standard_normal(n) * 10.0 ** rng.integers(-3, 3)).astype(np.float32)
    c = (r * (1 + 10.0 ** rng.integers(-7, -2) * rng.standard_normal(n))).astype(np.float32)
    if n and kind >= 2:
        a = int(rng.integers(0, n))
        b = min(n, a + int(rng.integers(1, 5000)))
        c[a:b] += np.float32(rng.choice([0.5, 1e-3, 1e-5]))
        for _ in range(int(rng.integers(0, 5))):
            c[rng.integers(0, n)] = rng.choice([np.nan, np.inf, -np.inf, 0.0, -0.0])
            r[rng.integers(0, n)] = rng.choice([np.nan, 0.0, -0.0, np.inf])
    if n and kind == 3 and rng.random() < 0.5:
        c[:] = r
    return _store(c, dt), _store(r, dt)


def _shape(rng):
    nd = int(rng.integers(0, 4))
    if nd == 0:
        return ()
    if nd == 1:
        return (int(rng.integers(0, 300_000)),)
    if nd == 2:
        return (int(rng.integers(1, 700)), int(rng.integers(1, 3000)))
    return (int(rng.integers(1, 5)), int(rng.integers(1, 300)), int(rng.integers(1, 700)))


@pytest.mark.parametrize("seed", [2608_81, 2608_82])
def test_random_sweeps(seed):
    rng = np.random.default_rng(seed)
    for rnd in range(20):
        cases = []
        for _ in range(int(rng.integers(1, 9))):
            dt = int(rng.choice(DTYPES))
            shape = _shape(rng)
            c, r = _pairs(rng, int(np.prod(shape)), dt)
            ct, rt = to_device(c, dt, shape), to_device(r, dt, shape)
            cases.append((ct, rt, [ct.clone()] if rng.random() < 0.2 else []))
        nt = int(rng.integers(1, 9))
        tols = [(float(rng.choice([0.0, 1e-6, 1e-4, 1e-3, 1e-2])),
                 float(rng.choice([0.0, 1e-6, 1e-4, 1e-3, 1e-2])), int(rng.integers(0, 2)))
                for _ in range(nt)]
        primary = int(rng.integers(0, nt))
        tile = None if rng.random() < 0.2 else (int(rng.integers(1, 130)), int(rng.integers(1, 130)))
        k = int(rng.choice([0, 1, 7, 64, 300]))
        integ = bool(rng.random() < 0.5)
        print("seed %d round %d: %d cases, %d pairs, tile %s, k %d, detectors %s"
              % (seed, rnd, len(cases), nt, tile, k, integ), flush=True)
        res = vc.vcheck_sweep(cases, tols, primary=primary, tile=tile, k=k, integrity=integ)
        for i, (c, r, ins) in enumerate(cases):
            tag = "seed %d round %d case %d %s %s" % (seed, rnd, i, tuple(r.shape), r.dtype)
            o = oracle_case(c, r, tols, primary=primary, tile=tile, k=k if k else None,
                            inputs=ins if integ else None)
            assert_stats(res["stats"][i], o.stats, tag)
            assert [int(x) for x in res["mismatches"][i]] == o.mismatches, tag
            if tile is not None:
                assert np.array_equal(res["tile_maps"][i], o.tile_map), tag + " tiles"
            if k:
                assert np.array_equal(res["first_k"][i], o.first_k), tag + " first-k"
            if integ:
                assert_integrity(res["integrity"][i], o.integrity, tag)


def _device(raw, dt, off):
    """Device view of raw storage starting `off` elements into a buffer."""
    pad = np.zeros(off, raw.dtype)
    t = torch.from_numpy(np.concatenate([pad, raw]).view(np.float32 if dt == oracle.F32 else np.int16))
    if dt != oracle.F32:
        t = t.view(torch.float16 if dt == oracle.F16 else torch.bfloat16)
    return t.cuda()[off:]


@pytest.mark.parametrize("seed", [2608_83, 2608_84])
def test_random_diagnostics(seed):
    rng = np.random.default_rng(seed)
    for rnd in range(15):
        batch = []
        for _ in range(int(rng.integers(1, 6))):
            dt = int(rng.choice(DTYPES))
            n = int(rng.choice([rng.integers(0, 100), rng.integers(100, 70_000),
                                rng.integers(70_000, 2_000_000)]))
            off = int(rng.choice([0, 0, 0, 1, 3]))
            c, r = _pairs(rng, n, dt)
            batch.append((dt, c, r, _device(c, dt, off), _device(r, dt, off)))
        atol = float(rng.choice([0.0, 1e-5, 1e-3, 1e-2]))
        rtol = float(rng.choice([0.0, 1e-5, 1e-3, 1e-2]))
        print("seed %d round %d: %d pairs of tensors, atol %g rtol %g"
              % (seed, rnd, len(batch), atol, rtol), flush=True)
        st = vc.vcheck_tensor_stats([b[3] for b in batch])
        npr = vc.vcheck_nearpass([(b[3], b[4]) for b in batch], atol, rtol)
        hs = vc.vcheck_content_hash([b[3] for b in batch] + [b[4] for b in batch])
        for i, (dt, c, r, _, _) in enumerate(batch):
            tag = "seed %d round %d tensor %d (dtype %d, %d elements)" % (seed, rnd, i, dt, c.size)
            cv, rv = (c.view(np.float32), r.view(np.float32)) if dt == oracle.F32 else (c, r)
            w, g = oracle.tensor_stats(cv, dt), st[i]
            for key in ("numel", "nan", "inf", "zero", "n_finite", "argmin", "argmax", "hist"):
                assert g[key] == w[key], (tag, key, g[key], w[key])
            for key in ("min", "max"):
                assert np.float64(g[key]).tobytes() == np.float64(w[key]).tobytes(), (tag, key)
            for key, mag in (("sum", w["sum_abs"]), ("sum_sq", w["sum_sq"]),
                             ("sum_abs", w["sum_abs"])):
                assert abs(g[key] - w[key]) <= 1e-6 * mag, (tag, key, g[key], w[key])
            w, g = oracle.nearpass(cv, rv, dt, atol, rtol), npr[i]
            for key in ("numel", "n_pairs", "n_fail", "n_zero_tol", "argmax_ratio", "max_ulp_fail",
                        "ratio_hist", "ulp_hist"):
                assert g[key] == w[key], (tag, key, g[key], w[key])
            assert np.float64(g["max_ratio"]).tobytes() == np.float64(w["max_ratio"]).tobytes(), tag
            assert hs[i] == oracle.content_hash(cv, dt), tag
            assert hs[len(batch) + i] == oracle.content_hash(rv, dt), tag
