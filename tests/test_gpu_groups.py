"""GPU parity of the two-level merge of a case with more than one chunk group
(more than 256 chunks): each group block merges its chunk records into a
group record, and the block completing the case's last group merges the
group records (counts summed in 64 bits, global indices, first-k lists
across group boundaries). A case of about 20M elements, alone in its dtype,
is cut into 4883 chunks of 4096 elements: 20 groups. Mismatches, the largest
|c - r|, a tie of the largest quotient and NaNs are planted on both sides of
the group boundary at element 4096 * 4096; every output is compared with the
oracle."""
import numpy as np
import pytest

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins as op
from tests.gpu_util import assert_stats, oracle_case, to_device

pytestmark = pytest.mark.gpu

N = 20_000_003                # 4883 chunks of 4096 elements, 20 groups of 256 chunks
BOUNDARY = 4096 * 4096        # first element of group 16


def _store(x, dt):
    x = np.asarray(x, np.float32)
    return x.view(np.uint32).copy() if dt == oracle.F32 else op.to_raw16(x, dt)


def _case(dt, seed):
    rng = np.random.default_rng(seed)
    r = rng.uniform(0.5, 1.0, N).astype(np.float32)
    c = r + (1e-4 * rng.standard_normal(N)).astype(np.float32)
    # mismatches just before and after the boundary (first-k spans it)
    near = np.arange(BOUNDARY - 6, BOUNDARY + 9)
    c[near] = r[near] + 0.5
    # the largest quotient, tied on both sides (the first index must win)
    r[[BOUNDARY - 1000, BOUNDARY + 1000]] = 0.5
    c[[BOUNDARY - 1000, BOUNDARY + 1000]] = 2.0
    # the largest |c - r| (8, quotient 0.08) in the second group only
    r[BOUNDARY + 777], c[BOUNDARY + 777] = 100.0, 108.0
    c[[5, BOUNDARY + 3_000_000, N - 1]] = np.nan
    return _store(c, dt), _store(r, dt)


@pytest.mark.parametrize("k", [0, 16, 1024])
def test_two_group_case_sweep(k):
    tol = (1e-2, 1e-2, 0)  # above the bfloat16 rounding of the noise
    cases, want = [], []
    for i, dt in enumerate((oracle.F32, oracle.BF16)):
        c, r = _case(dt, 90_210 + i)
        cand, ref = to_device(c, dt, (N,)), to_device(r, dt, (N,))
        cases.append((cand, ref))
        want.append(oracle_case(cand, ref, [tol], tile=(1, 4096), k=k))
    got = vc.vcheck_sweep(cases, [tol], tile=(1, 4096), k=k)
    for i, o in enumerate(want):
        tag = "case %d k %d" % (i, k)
        assert_stats(got["stats"][i], o.stats, tag)
        assert o.stats["argmax_rel"] == BOUNDARY - 1000, tag
        assert o.stats["argmax_abs"] == BOUNDARY + 777, tag
        assert np.array_equal(got["tile_maps"][i], o.tile_map), tag + " tile map"
        if k:
            assert np.array_equal(got["first_k"][i], o.first_k), tag + " first-k"
    assert got["mismatches"][:, 0].tolist() == [o.stats["mismatches"] for o in want]
