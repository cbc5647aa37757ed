"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded bytes. Counts, indices, tile maps, flags, max_abs and max_rel are
compared bit-exactly; the binary64 error sums within 1e-6 relative."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins as op
from tests.gpu_util import assert_integrity, assert_stats, oracle_case, to_device

pytestmark = pytest.mark.gpu

F32, F16, BF16 = oracle.F32, oracle.F16, oracle.BF16
DTYPES = {"f32": F32, "f16": F16, "bf16": BF16}
SHAPES = [(), (1,), (7,), (63, 65), (64, 64), (1, 4097), (1000, 1), (2, 3, 4, 5), (257, 513),
          (3, 100003), (5000, 37)]


def clean_pairs(rng, n, dtype, fault_frac=0.01):
    """Finite data (the fast path): ref ~ N(0,1), cand = ref + noise, with a
    fraction of gross faults, exact copies and exact zeros in ref."""
    r = rng.standard_normal(n).astype(np.float32)
    c = r + (1e-4 * rng.standard_normal(n)).astype(np.float32)
    f = rng.random(n) < fault_frac
    c[f] = r[f] * 1.5 + 0.25
    same = rng.random(n) < 0.05
    c[same] = r[same]
    if dtype == F32:
        return c.view(np.uint32), r.view(np.uint32)
    return op.to_raw16(c, dtype), op.to_raw16(r, dtype)


def make(kind, dtype, shape, seed):
    rng = np.random.default_rng(seed)
    n = int(np.prod(shape)) if shape else 1
    if kind == "special":
        c, r = op.random_pairs(rng, n, dtype)
    elif kind == "ties":
        vals = np.array([-2.0, -1.0, -0.5, 0.5, 1.0, 2.0, 4.0], dtype=np.float32)
        r32 = rng.choice(vals, n).astype(np.float32)
        c32 = rng.choice(vals, n).astype(np.float32)
        c, r = (c32.view(np.uint32), r32.view(np.uint32)) if dtype == F32 else \
            (op.to_raw16(c32, dtype), op.to_raw16(r32, dtype))
    else:
        c, r = clean_pairs(rng, n, dtype)
    return to_device(c, dtype, shape), to_device(r, dtype, shape)


@pytest.mark.parametrize("kind", ["clean", "special", "ties"])
@pytest.mark.parametrize("dt", list(DTYPES))
def test_compare_corpus(dt, kind):
    dtype = DTYPES[dt]
    tols = [(1e-3, 1e-3, 0), (0.0, 1e-2, 1), (1e-2, 0.0, 0), (0.0, 0.0, 0)]
    for si, shape in enumerate(SHAPES):
        cand, ref = make(kind, dtype, shape, 1000 * si + dtype)
        for t in tols:
            tag = "%s %s %r tol %r" % (dt, kind, shape, t)
            g = vc.vcheck_compare(cand, ref, t[0], t[1], bool(t[2]))
            o = oracle_case(cand, ref, [t])
            assert_stats(g, o.stats, tag)
            assert g["pass"] == int(o.stats["mismatches"] == 0) and g["case_status"] == 0


@pytest.mark.parametrize("dt", list(DTYPES))
def test_localize_corpus(dt):
    dtype = DTYPES[dt]
    geoms = [((8, 16), 64), ((1, 64), 1), ((64, 1), 1024), ((32, 32), 0), ((5, 3), 7),
             ((1, 1), 100), ((128, 128), 64)]
    for si, shape in enumerate(SHAPES):
        for kind in ("clean", "special"):
            cand, ref = make(kind, dtype, shape, 77 + si)
            for (th, tw), k in geoms:
                tag = "%s %s %r tile %dx%d k %d" % (dt, kind, shape, th, tw, k)
                g = vc.vcheck_localize(cand, ref, 1e-3, 1e-3, th, tw, k)
                o = oracle_case(cand, ref, [(1e-3, 1e-3, 0)], tile=(th, tw), k=k)
                assert_stats(g["stats"], o.stats, tag)
                assert np.array_equal(g["tile_map"], o.tile_map), tag + " tile map"
                assert np.array_equal(g["first_k"], o.first_k), tag + " first-k"


@pytest.mark.parametrize("dt", list(DTYPES))
def test_integrity_corpus(dt):
    dtype = DTYPES[dt]
    rng = np.random.default_rng(5)
    for si, shape in enumerate([(7,), (63, 65), (257, 513), (3, 100003)]):
        cand, ref = make("clean", dtype, shape, 500 + si)
        n = cand.numel()
        other = to_device(op.random_pairs(rng, n, dtype)[0], dtype, shape)
        variants = {
            "plain": (cand, ref, [other]),
            "copy": (other.clone(), ref, [cand, other]),
            "identity": (other.clone(), other.clone(), [other]),
            "zero": (torch.zeros_like(ref), ref, []),
            "signed_zero": (torch.zeros_like(ref).neg_(), ref, []),
            "constant": (torch.full_like(ref, 2.0), ref, []),
            "nan_fill": (torch.full_like(ref, float("nan")), ref, []),
            "bf16_grid": (ref.float().to(torch.bfloat16).to(ref.dtype) * 1.5, ref, []),
            "fp16_grid": (ref.float().half().to(ref.dtype) * 1.25, ref, []),
            "special": (other, ref, [ref, cand]),
        }
        for name, (c, r, ins) in variants.items():
            tag = "%s %r %s" % (dt, shape, name)
            g = vc.vcheck_integrity(c, r, ins, 1e-3, 1e-3)
            o = oracle_case(c, r, [(1e-3, 1e-3, 0)], inputs=ins)
            assert_stats(g["stats"], o.stats, tag)
            assert_integrity(g["integrity"], o.integrity, tag)


def test_fp16_representability_edges():
    """Binary32 values at every binary16 boundary: subnormal grid (odd
    multiples of 2^-24), just off it, 65504/65520/65536, fp32 subnormals."""
    vals = [2.0**-24, 3 * 2.0**-24, 1023 * 2.0**-24, 2.0**-25, 3 * 2.0**-26, 2.0**-14,
            2.0**-14 + 2.0**-24, 65504.0, 65520.0, 65536.0, -65504.0, 1.0 + 2.0**-10,
            1.0 + 2.0**-11, 1e-40, -1e-45, 0.0, -0.0, float("inf"), float("nan")]
    rng = np.random.default_rng(9)
    base = np.array(vals, dtype=np.float32)
    for rep in range(3):
        cand = np.concatenate([base, rng.choice(base, 4000)]).astype(np.float32)
        ref = rng.standard_normal(cand.size).astype(np.float32)
        c, r = to_device(cand.view(np.uint32), F32, cand.shape), to_device(
            ref.view(np.uint32), F32, ref.shape)
        g = vc.vcheck_integrity(c, r, [], 1e-3, 1e-3)
        o = oracle_case(c, r, [(1e-3, 1e-3, 0)], inputs=[])
        assert_integrity(g["integrity"], o.integrity, "fp16 edges")
        assert_stats(g["stats"], o.stats, "fp16 edges")


def test_gate_ties_and_no_fma():
    """The hand-built exact-threshold cases and the fma-sensitive cases of the
    oracle's pins give identical per-element decisions on the GPU."""
    inf, nan = float("inf"), float("nan")
    one_ulp = float(np.nextafter(np.float32(1.5), np.float32(2)))
    ref = np.array([1.0, 1.0, 1.0, -1.0, 0.0, -0.0, inf, inf, -inf, 5.0, nan, nan, 2.0, 0.0],
                   dtype=np.float32)
    cand = np.array([1.5, one_ulp, 0.5, -1.5, -0.0, 0.0, inf, -inf, 5.0, inf, nan, 1.0, 2.5, 0.25],
                    dtype=np.float32)
    for eqn in (False, True):
        c, r = to_device(cand.view(np.uint32), F32, (14,)), to_device(ref.view(np.uint32), F32, (14,))
        g = vc.vcheck_localize(c, r, 0.25, 0.25, 1, 1, 14, equal_nan=eqn)
        o = oracle_case(c, r, [(0.25, 0.25, int(eqn))], tile=(1, 1), k=14)
        assert np.array_equal(g["tile_map"], o.tile_map)
        assert_stats(g["stats"], o.stats, "ties")
    rng = np.random.default_rng(3)
    found = 0
    for _ in range(20000):
        r = float(np.float32(rng.uniform(0.5, 2.0)))
        c = float(np.float32(r + rng.uniform(1e-4, 1e-2)))
        d = abs(c - r)
        rtol = float(rng.uniform(1e-6, 1e-3))
        atol = d - rtol * abs(r)
        if atol < 0:
            continue
        for _s in range(4):
            t_sep = atol + rtol * abs(r)
            t_fma = op._fma(rtol, abs(r), atol)
            if (d <= t_sep) != (d <= t_fma):
                cc = to_device(np.array([c], dtype=np.float32).view(np.uint32), F32, (1,))
                rr = to_device(np.array([r], dtype=np.float32).view(np.uint32), F32, (1,))
                g = vc.vcheck_compare(cc, rr, atol, rtol)
                o = oracle_case(cc, rr, [(atol, rtol, 0)])
                assert g["mismatches"] == o.stats["mismatches"], (c, r, atol, rtol)
                found += 1
            atol = float(np.nextafter(atol, np.inf))
        if found >= 24:
            break
    assert found >= 8


def _sweep_cases(rng):
    cases, inputs = [], []
    kinds = ["clean", "special", "ties"]
    for i in range(40):
        dtype = [F32, F16, BF16][i % 3]
        shape = SHAPES[i % len(SHAPES)]
        cand, ref = make(kinds[i % 3], dtype, shape, 9000 + i)
        ins = [cand.clone()] if i % 5 == 0 else [ref.clone()] if i % 7 == 0 else []
        cases.append((cand if i % 5 else ins[0], ref, ins))
    # per-case outcomes: differing shapes, differing dtypes, empty, misaligned
    a = torch.randn(16, device="cuda")
    cases.append((a[:8].reshape(2, 4), a[8:].reshape(4, 2), []))
    cases.append((a[:8].half(), a[8:], []))
    cases.append((torch.empty(0, 5, device="cuda"), torch.empty(0, 5, device="cuda"), []))
    buf_c = torch.randn(1 + 5000, device="cuda")
    buf_r = buf_c.clone()
    buf_r[100:110] += 1.0
    cases.append((buf_c[1:], buf_r[1:], [buf_c[1:].clone()]))  # 4-byte but not 16-byte aligned
    return cases


def test_sweep_mixed():
    rng = np.random.default_rng(11)
    cases = _sweep_cases(rng)
    tols = [(1e-6, 1e-6, 0), (1e-4, 1e-4, 1), (1e-3, 1e-3, 0), (1e-2, 1e-2, 0)]
    for primary, tile, k, integ in [(2, (16, 16), 32, True), (0, None, 0, False),
                                    (3, (1, 7), 1024, True), (1, (64, 64), 5, False)]:
        res = vc.vcheck_sweep(cases, tols, primary=primary, tile=tile, k=k, integrity=integ)
        mism_o, status_o, flags_o = [], [], []
        for i, (c, r, ins) in enumerate(cases):
            tag = "case %d primary %d" % (i, primary)
            gs = res["stats"][i]
            if c.dtype != r.dtype or c.shape != r.shape:
                assert gs["case_status"] in (-2, -3), tag
                assert gs["pass"] == 0 and list(res["pass"][i]) == [0] * len(tols)
                mism_o.append([0] * len(tols))
                status_o.append(gs["case_status"])
                flags_o.append(0)
                continue
            o = oracle_case(c, r, tols, primary=primary, tile=tile, k=k if k else None,
                            inputs=ins if integ else None)
            assert_stats(gs, o.stats, tag)
            assert [int(x) for x in res["mismatches"][i]] == o.mismatches, tag
            if tile is not None:
                assert np.array_equal(res["tile_maps"][i], o.tile_map), tag + " tiles"
            if k:
                assert np.array_equal(res["first_k"][i], o.first_k), tag + " first-k"
            if integ:
                assert_integrity(res["integrity"][i], o.integrity, tag)
            mism_o.append(o.mismatches)
            status_o.append(0)
            flags_o.append(o.integrity["flags"] if integ else 0)
        pas, rate = oracle.suite(np.array(mism_o, dtype=np.uint64), status_o,
                                 flags_o if integ else None)
        assert np.array_equal(res["pass"], pas)
        assert np.array_equal(res["match_rate"], rate), (res["match_rate"], rate)
        _, nrate = oracle.suite(np.array(mism_o, dtype=np.uint64), status_o, None)
        assert np.array_equal(res["numeric_rate"], nrate)


def test_sweep_empty_and_repeat_determinism():
    res = vc.vcheck_sweep([], [(1e-3, 1e-3)])
    assert res["match_rate"].tolist() == [0.0]
    rng = np.random.default_rng(12)
    cases = [(c, r) for c, r, _ in _sweep_cases(rng)[:20]]
    sw = vc.Sweep(cases, [(1e-4, 1e-4), (1e-3, 1e-3)], primary=1, tile=(8, 8), k=16)
    outs = []
    for _ in range(5):
        sw.launch()
        r = sw.results()
        outs.append((sw.stats.cpu().numpy().tobytes(), r["mismatches"].tobytes(),
                     sw.tmaps.cpu().numpy().tobytes(), sw.fk.cpu().numpy().tobytes()))
    assert all(o == outs[0] for o in outs)
