"""The allocation-free sweep (vcheck_sweep_noalloc): it runs in the library's
static device scratch instead of a caller workspace. Its results must equal
those of vcheck_sweep on the same inputs, call after call (the scratch keeps
the previous call's contents, so a second, smaller sweep checks that nothing
of the first one leaks into it); a sweep that needs more scratch than the
array holds is refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins as op
from tests.gpu_util import assert_integrity, assert_stats, oracle_case, to_device

pytestmark = pytest.mark.gpu


def _case(rng, dt, shape, n_bad):
    n = int(np.prod(shape)) if shape else 1
    r32 = rng.standard_normal(n).astype(np.float32)
    c32 = r32 + (1e-4 * rng.standard_normal(n)).astype(np.float32)
    if n_bad:
        c32[rng.choice(n, size=min(n_bad, n), replace=False)] += 0.75
    if dt == oracle.F32:
        c, r = c32.view(np.uint32), r32.view(np.uint32)
    else:
        c, r = op.to_raw16(c32, dt), op.to_raw16(r32, dt)
    return to_device(c, dt, shape), to_device(r, dt, shape)


def _same(a, b, tag):
    for key in ("mismatches", "pass", "match_rate", "numeric_rate"):
        assert np.array_equal(a[key], b[key]), (tag, key)
    assert a["stats"] == b["stats"], tag
    for key in ("integrity", "tile_maps", "first_k"):
        assert (key in a) == (key in b), (tag, key)
    if "integrity" in a:
        assert a["integrity"] == b["integrity"], tag
    if "tile_maps" in a:
        assert len(a["tile_maps"]) == len(b["tile_maps"]), tag
        for x, y in zip(a["tile_maps"], b["tile_maps"]):
            assert np.array_equal(x, y), tag
    if "first_k" in a:
        assert np.array_equal(a["first_k"], b["first_k"]), tag


def test_noalloc_matches_sweep_on_consecutive_calls():
    rng = np.random.default_rng(2608_0007)
    big = []
    for dt, shape, bad in [(oracle.F16, (1024, 2048), 900), (oracle.F32, (257, 513), 40),
                           (oracle.BF16, (3, 100003), 17), (oracle.F16, (1, 7), 2),
                           (oracle.F32, (), 0), (oracle.BF16, (2, 3, 4, 5), 3)]:
        c, r = _case(rng, dt, shape, bad)
        big.append((c, r, [r.clone()]))
    # an all-zero candidate and a bit copy of the input trip the detectors
    big.append((torch.zeros_like(big[1][1]), big[1][1], [big[1][1].clone()]))
    big.append((big[0][2][0].clone(), big[0][1], big[0][2]))
    tols = [(1e-3, 1e-3, 0), (1e-2, 1e-2, 1), (1e-5, 1e-5, 0)]
    kw = dict(primary=0, tile=(16, 32), k=40, integrity=True)
    got = vc.vcheck_sweep_noalloc(big, tols, **kw)
    want = vc.vcheck_sweep(big, tols, **kw)
    _same(got, want, "first call")
    first = want
    for i in (0, 3, 6, 7):
        c, r, ins = big[i]
        o = oracle_case(c, r, tols, primary=0, tile=(16, 32), k=40, inputs=ins)
        assert_stats(got["stats"][i], o.stats, "case %d" % i)
        assert np.array_equal(got["tile_maps"][i], o.tile_map), i
        assert np.array_equal(got["first_k"][i], o.first_k), i
        assert_integrity(got["integrity"][i], o.integrity, "case %d" % i)

    # second call: fewer, smaller cases, other options, in the same scratch
    small = [(big[3][0], big[3][1]), _case(rng, oracle.F32, (33, 65), 5)]
    tols2 = [(1e-4, 1e-4, 0)]
    kw2 = dict(primary=0, tile=(8, 8), k=4)
    got = vc.vcheck_sweep_noalloc(small, tols2, **kw2)
    want = vc.vcheck_sweep(small, tols2, **kw2)
    _same(got, want, "second call")
    want = first
    for i, (c, r) in enumerate(small):
        o = oracle_case(c, r, tols2, primary=0, tile=(8, 8), k=4)
        assert_stats(got["stats"][i], o.stats, "small case %d" % i)
        assert np.array_equal(got["tile_maps"][i], o.tile_map), i
        assert np.array_equal(got["first_k"][i], o.first_k), i

    # back to the first sweep: the same results as the first time
    again = vc.vcheck_sweep_noalloc(big, tols, **kw)
    _same(again, want, "third call")


def test_noalloc_refuses_oversize_sweeps():
    # 1 x 1 tiles over 2^24 elements need 64 MiB of tile counters: more than
    # the scratch array holds
    n = 1 << 24
    r = torch.zeros(n, dtype=torch.float16, device="cuda")
    with pytest.raises(vc.VcheckError) as e:
        vc.vcheck_sweep_noalloc([(r, r)], [(1e-3, 1e-3)], tile=(1, 1))
    assert e.value.status == -8  # VC_ERR_LIMIT
    # a workable sweep still runs afterwards
    c, r2 = r[:4096].clone(), r[:4096].clone()
    c[7] = 1.0
    got = vc.vcheck_sweep_noalloc([(c, r2)], [(1e-3, 1e-3)], tile=(1, 64), k=2)
    assert got["stats"][0]["mismatches"] == 1
    assert got["first_k"][0].tolist() == [7, -1]
    assert int(got["tile_maps"][0].sum()) == 1 and int(got["tile_maps"][0][0]) == 1
