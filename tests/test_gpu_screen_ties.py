"""GPU parity of the largest-quotient screen that the four waves of a block
share: the screen of every wave uses the largest quotient |c - r| / |r| that
any wave of the block has found, so a wave may see that value before it
reaches an equal quotient at a smaller index in its own steps. Ties must
still go to the first index (the reduction of the maximum takes the smallest
index among equal values), and a strictly larger quotient found late must
still win. The data is tame (the fast tiers take nearly every step, and
with the loose tolerance also the steps of the planted values); the tied
quotients sit at the same element of consecutive steps, so that they
fall to different waves of one round, in every chunk, and the ties of the
absolute difference come with them. Each case is compared with the oracle."""
import numpy as np
import pytest

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins as op
from tests.gpu_util import assert_stats, oracle_case, to_device

pytestmark = pytest.mark.gpu

N = (1 << 20) + 77  # many chunks and a ragged tail
DTYPES = {"f32": oracle.F32, "f16": oracle.F16, "bf16": oracle.BF16}


def _store(x, dt):
    x = np.asarray(x, np.float32)
    return x.view(np.uint32).copy() if dt == oracle.F32 else op.to_raw16(x, dt)


def _data(dt, seed, late_larger):
    rng = np.random.default_rng(seed)
    r = rng.uniform(0.5, 1.0, N).astype(np.float32)
    c = r + (1e-4 * rng.standard_normal(N)).astype(np.float32)
    step = 256 if dt == oracle.F32 else 512  # elements per wave step
    # the tied largest quotient 0.25 (r = 1, c = 1.25: exact in every
    # format), at element 37 of four consecutive steps, from step s0 on,
    # every 64 steps, with a random extra tie in between
    idx = []
    for s0 in range(3, N // step - 4, 64):
        idx += [(s0 + j) * step + 37 for j in range(4)]
        idx.append(int(rng.integers(s0 * step, (s0 + 60) * step)))
    idx = np.array(sorted(set(i for i in idx if i < N)))
    r[idx], c[idx] = 1.0, 1.25
    if late_larger:
        # a strictly larger quotient near the end, then its own ties
        big = np.array([N - 5000, N - 4000 + 1, N - 900])
        r[big], c[big] = 1.0, 1.5
    return _store(c, dt), _store(r, dt), int(idx[0])


@pytest.mark.parametrize("tol", [(1.0, 0.0, 0), (1e-3, 1e-3, 0)])
@pytest.mark.parametrize("late_larger", [False, True])
@pytest.mark.parametrize("dt", list(DTYPES))
def test_shared_quotient_screen_ties(dt, late_larger, tol):
    dtype = DTYPES[dt]
    c, r, first = _data(dtype, 4242 + dtype, late_larger)
    cand, ref = to_device(c, dtype, (N,)), to_device(r, dtype, (N,))
    g = vc.vcheck_compare(cand, ref, *tol)
    o = oracle_case(cand, ref, [tol])
    tag = "%s late_larger=%s tol %r" % (dt, late_larger, tol)
    assert_stats(g, o.stats, tag)
    if not late_larger:
        assert g["argmax_rel"] == first and g["max_rel"] == 0.25, tag
    else:
        assert g["argmax_rel"] == N - 5000 and g["max_rel"] == 0.5, tag
    # the same tensors through a sweep of two copies (chunks of both cases)
    sw = vc.vcheck_sweep([(cand, ref), (cand, ref)], [tol])
    for s in sw["stats"]:
        assert_stats(s, o.stats, tag + " sweep")
