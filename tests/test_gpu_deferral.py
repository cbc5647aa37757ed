"""GPU parity on large cases whose steps are mostly deferred past the streaming loop.

Steps holding a NaN are evaluated by the exact tier after the streaming
loop. A step with mismatches while mismatch positions are recorded is
committed in the loop; its positions are found afterwards (from mismatch
bits kept in LDS for 16-bit storage with one tolerance pair, by re-reading
the step otherwise), except for binary32 storage with one pair, where the
exact tier evaluates it whole. When more steps pile up than a wave lists,
the list is evaluated mid-stream.

Each batch is large enough for the planner to give every wave 64 steps
(2^29 binary32 or 2^30 binary16 elements). In the dense cases nearly every
step holds a NaN or a mismatch, so the list overflows and is evaluated
mid-stream; in the sparse ones about a fifth do, and the four waves evaluate
their merged lists together after streaming. Each runs on an aligned case
(vector loads) and on a misaligned one (element loads). Equal maxima are
planted in deferred and in streamed steps: the first index must win."""
import numpy as np
import pytest

from paper_2608_02712_amd import vcheck as vc
from tests.gpu_util import assert_stats, oracle_case

pytestmark = pytest.mark.gpu

SHAPES = {"fp32": (8192, 16384), "fp16": (16384, 16384)}


def _case(torch, dtype, rng, gen, shape, every, misaligned):
    n = shape[0] * shape[1]
    r32 = torch.randn(n, generator=gen, device="cuda")
    if dtype == "fp32":
        r = r32
        c = r32 + 1e-5 * torch.randn(n, generator=gen, device="cuda")
    else:
        r = r32.half()
        c = (r32 + 1e-4 * torch.randn(n, generator=gen, device="cuda")).half()
    del r32

    def at(size):
        return torch.from_numpy(rng.choice(n, size=size, replace=False)).cuda()

    # mismatches, NaNs, then equal largest differences (|c - r| = 8) in
    # deferred and streamed steps
    bad = at(n // every)
    c[bad] = c[bad] + 1.0
    c[at(n // (2 * every))] = float("nan")
    big = at(64)
    r[big] = 0.5
    c[big] = 8.5
    if misaligned:
        # data pointers 4 bytes past a 16-byte boundary
        cb = torch.empty(n + 4 // c.element_size(), dtype=c.dtype, device="cuda")
        rb = torch.empty_like(cb)
        off = 4 // c.element_size()
        cb[off:] = c
        rb[off:] = r
        c, r = cb[off:], rb[off:]
        assert c.data_ptr() % 16 == 4
    return c.view(shape), r.view(shape)


@pytest.mark.parametrize("dtype", ["fp32", "fp16"])
@pytest.mark.parametrize(
    "tols,primary",
    [
        ([(1e-3, 1e-3, 0)], 0),
        ([(1e-5, 1e-5, 0), (1e-3, 1e-3, 0), (0.5, 0.5, 1)], 1),
    ],
    ids=["one-pair", "three-pairs"],
)
def test_deferred_steps_large(dtype, tols, primary):
    import torch

    rng = np.random.default_rng(2608_77)
    gen = torch.Generator(device="cuda").manual_seed(2608_78)
    shape = SHAPES[dtype]
    # (fault spacing, misaligned): dense lists overflow, sparse ones do not
    cases = [_case(torch, dtype, rng, gen, shape, every, mis)
             for every, mis in ((20, False), (2000, False), (20, True), (2000, True))]
    print("deferral: sweep of 4 x %s %s, %d pairs" % (shape, dtype, len(tols)), flush=True)
    res = vc.vcheck_sweep(cases, tols, primary=primary, tile=(64, 64), k=64)
    for i, (c, r) in enumerate(cases):
        tag = "case %d" % i
        o = oracle_case(c, r, tols, primary=primary, tile=(64, 64), k=64)
        assert_stats(res["stats"][i], o.stats, tag)
        assert [int(x) for x in res["mismatches"][i]] == o.mismatches, tag
        assert np.array_equal(res["tile_maps"][i], o.tile_map), tag + " tiles"
        assert np.array_equal(res["first_k"][i], o.first_k), tag + " first-k"
        assert o.stats["max_abs"] == 8.0, tag
