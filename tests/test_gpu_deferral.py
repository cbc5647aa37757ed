"""GPU parity on large cases whose steps are mostly deferred to the exact tier.

Steps holding a NaN, or a mismatch while mismatch positions are recorded,
are evaluated after the streaming loop (with several tolerance pairs a
mismatching step is committed in the loop and only its positions are found
afterwards); when more of them pile up than a wave lists, the list is
evaluated mid-stream. These cases are large enough
(2^29 binary32 elements in the batch) for the planner to give each wave 64
steps, so both the list overflow and the final evaluation run, on an aligned
case (vector loads) and on a misaligned one (element loads). Equal maxima are
planted in deferred and in streamed steps: the first index must win."""
import numpy as np
import pytest

from paper_2608_02712_amd import vcheck as vc
from tests.gpu_util import assert_stats, oracle_case

pytestmark = pytest.mark.gpu

ROWS, COLS = 16384, 16384


def _case(rng, n):
    r = rng.standard_normal(n, dtype=np.float32)
    c = r + np.float32(1e-5) * rng.standard_normal(n, dtype=np.float32)
    # NaNs in about half of the 256-element steps: those steps are deferred
    nan_at = rng.choice(n, size=n // 300, replace=False)
    c[nan_at] = np.nan
    # equal largest differences (|c - r| = 8) in some deferred steps and
    # some streamed ones, plus ordinary mismatches
    big = np.sort(rng.choice(n, size=64, replace=False))
    r[big] = 0.5
    c[big] = 8.5
    c[nan_at] = np.nan
    bad = rng.choice(n, size=n // 5000, replace=False)
    c[bad] += 1.0
    return c, r


@pytest.mark.parametrize(
    "tols,primary",
    [
        ([(1e-3, 1e-3, 0)], 0),
        ([(1e-5, 1e-5, 0), (1e-3, 1e-3, 0), (0.5, 0.5, 1)], 1),
    ],
    ids=["one-pair", "three-pairs"],
)
def test_deferred_steps_large(tols, primary):
    import torch

    rng = np.random.default_rng(2608_77)
    n = ROWS * COLS
    c0, r0 = _case(rng, n)
    c1, r1 = _case(rng, n)
    cand0 = torch.from_numpy(c0).reshape(ROWS, COLS).cuda()
    ref0 = torch.from_numpy(r0).reshape(ROWS, COLS).cuda()
    # misaligned views: data pointers 4 bytes past a 16-byte boundary
    cbuf = torch.empty(n + 1, dtype=torch.float32, device="cuda")
    rbuf = torch.empty(n + 1, dtype=torch.float32, device="cuda")
    cbuf[1:] = torch.from_numpy(c1).cuda()
    rbuf[1:] = torch.from_numpy(r1).cuda()
    cand1, ref1 = cbuf[1:].view(ROWS, COLS), rbuf[1:].view(ROWS, COLS)
    assert cand1.data_ptr() % 16 == 4
    del c0, r0, c1, r1
    cases = [(cand0, ref0), (cand1, ref1)]
    print("deferral: sweep of 2 x %d fp32 elements, %d pairs" % (n, len(tols)), flush=True)
    res = vc.vcheck_sweep(cases, tols, primary=primary, tile=(64, 64), k=64)
    for i, (c, r) in enumerate(cases):
        tag = "case %d" % i
        o = oracle_case(c, r, tols, primary=primary, tile=(64, 64), k=64)
        assert_stats(res["stats"][i], o.stats, tag)
        assert [int(x) for x in res["mismatches"][i]] == o.mismatches, tag
        assert np.array_equal(res["tile_maps"][i], o.tile_map), tag + " tiles"
        assert np.array_equal(res["first_k"][i], o.first_k), tag + " first-k"
        assert o.stats["max_abs"] == 8.0, tag
