"""GPU parity of the probe and near-pass kernels on data shaped for their
branch-free usual-step paths: long runs of finite, tame steps, with the
events that must leave those paths planted late in a wave's range.

Probe: a strict new minimum and maximum after many usual steps (each in a
later element of its step), ties of both extremes after them (the first
index must win), zeros of both signs
throughout (counted on the usual path in the histogram's zero slot), binary16
subnormals and one late NaN.

Near-pass: pairs well inside the tolerance, with late failures, a late new
largest ratio followed by an exact tie (first index), zeros of both signs
(grid distance 0 between -0 and +0), opposite-sign pairs a few grid steps
apart, values beyond the binary16 range and one late infinity."""
import numpy as np
import pytest

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins

pytestmark = pytest.mark.gpu

N = (1 << 20) + 77  # several chunks, a ragged tail
DTYPES = (oracle.F32, oracle.F16, oracle.BF16)


def _store(x, dt):
    x = np.asarray(x, np.float32)
    if dt == oracle.F32:
        return x.view(np.uint32).copy()
    with np.errstate(over="ignore"):  # beyond 65504 binary16 storage holds infinities
        return oracle_pins.to_raw16(x, dt)


def _tensor(torch, raw, dt):
    if dt == oracle.F32:
        return torch.from_numpy(raw.view(np.float32).copy()).cuda()
    t = torch.from_numpy(raw.view(np.int16).copy())
    return t.view(torch.float16 if dt == oracle.F16 else torch.bfloat16).cuda()


def _view(raw, dt):
    return raw.view(np.float32) if dt == oracle.F32 else raw


def _probe_data(rng):
    x = rng.uniform(-1.0, 1.0, N).astype(np.float32)
    zeros = rng.choice(N, N // 10, replace=False)
    x[zeros] = np.where(rng.random(zeros.size) < 0.5, -0.0, 0.0).astype(np.float32)
    x[rng.choice(N, 500, replace=False)] = 3e-7  # binary16 subnormal
    # late strict extremes, then exact ties of both; each in a step of its
    # own, at an element other than the step's first two (so a screen that
    # looked at only part of the step would miss it)
    x[700_005], x[700_014] = -5.0, 6.0
    x[900_003], x[1_000_007] = -5.0, 6.0
    x[N - 3] = np.nan
    return x


def test_probe_usual_steps_parity():
    import torch

    rng = np.random.default_rng(2608_71)
    x = _probe_data(rng)
    raws = [(_store(x, dt), dt) for dt in DTYPES]
    print("probe usual steps: %d tensors of %d elements" % (len(raws), N), flush=True)
    res = vc.vcheck_tensor_stats([_tensor(torch, raw, dt) for raw, dt in raws])
    for (raw, dt), got in zip(raws, res):
        want = oracle.tensor_stats(_view(raw, dt), dt)
        for k in ("numel", "nan", "inf", "zero", "n_finite", "argmin", "argmax", "hist"):
            assert got[k] == want[k], (dt, k, got[k], want[k])
        for k in ("min", "max"):
            assert np.float64(got[k]).tobytes() == np.float64(want[k]).tobytes(), (dt, k)
        for k in ("sum", "sum_sq", "sum_abs"):
            assert abs(got[k] - want[k]) <= 1e-6 * max(want["sum_abs"], want["sum_sq"]), (dt, k)
        assert (got["argmin"], got["argmax"]) == (700_005, 700_014)
        assert got["zero"] > N // 20  # most planted zeros survive the later plants


def _nearpass_data(rng):
    r = rng.uniform(0.5, 2.0, N).astype(np.float32) * np.where(rng.random(N) < 0.5, -1, 1)
    c = (r * (1 + 1e-4 * rng.standard_normal(N))).astype(np.float32)
    zeros = rng.choice(N, N // 20, replace=False)
    r[zeros] = -0.0
    c[zeros] = 0.0
    # opposite signs a few grid steps apart around zero
    tiny = rng.choice(N, 300, replace=False)
    r[tiny], c[tiny] = 6e-8, -1.2e-7
    # beyond the binary16 range (outside the grid for binary32 storage)
    big = rng.choice(N, 400, replace=False)
    r[big] = 1e5
    c[big] = np.float32(1e5) * np.float32(1 + 1e-6)
    # late failures, a late largest ratio and its exact tie
    c[800_000] = r[800_000] + np.float32(0.25)
    r[900_000], c[900_000] = 1.0, 1.5
    r[950_000], c[950_000] = 1.0, 1.5
    c[N - 5] = np.inf
    return c, r


@pytest.mark.parametrize("atol,rtol", [(1e-3, 1e-3), (0.0, 1e-2)])
def test_nearpass_usual_steps_parity(atol, rtol):
    import torch

    rng = np.random.default_rng(2608_72)
    c, r = _nearpass_data(rng)
    cases = [(_store(c, dt), _store(r, dt), dt) for dt in DTYPES]
    print("nearpass usual steps: %d cases of %d elements, atol %g rtol %g"
          % (len(cases), N, atol, rtol), flush=True)
    res = vc.vcheck_nearpass([(_tensor(torch, cr, dt), _tensor(torch, rr, dt))
                              for cr, rr, dt in cases], atol, rtol)
    for (cr, rr, dt), got in zip(cases, res):
        want = oracle.nearpass(_view(cr, dt), _view(rr, dt), dt, atol, rtol)
        for k in ("numel", "n_pairs", "n_fail", "n_zero_tol", "argmax_ratio", "max_ulp_fail",
                  "ratio_hist", "ulp_hist"):
            assert got[k] == want[k], (dt, k, got[k], want[k])
        assert np.float64(got["max_ratio"]).tobytes() == np.float64(want["max_ratio"]).tobytes()
        assert got["n_fail"] > 0 and got["argmax_ratio"] >= 0


@pytest.mark.parametrize("atol,rtol", [(1e-3, 1e-3), (1e-2, 0.0), (0.0, 1e-2)])
def test_nearpass_usual_steps_tolerance_boundary(atol, rtol):
    """Pairs whose difference lies within a few binary32 rounding steps of
    the tolerance (both sides), planted late among well-inside pairs, so the
    usual-step screen meets them once a largest ratio exists: a screen that
    let one of them through would lose a failure, a ratio bin or the largest
    ratio. The oracle decides each pair exactly."""
    import torch

    rng = np.random.default_rng(2608_73)
    r = (rng.uniform(0.5, 2.0, N) * np.where(rng.random(N) < 0.5, -1, 1)).astype(np.float32)
    c = (r * (1 + 1e-5 * rng.standard_normal(N))).astype(np.float32)
    # a early failure sets a largest ratio above 1, then one below 1 is
    # planted first in a second case (below)
    pos = rng.choice(np.arange(N // 2, N), 4000, replace=False)
    rel = np.array([-2.0 ** -18, -2.0 ** -21, -2.0 ** -23, -2.0 ** -24, 0.0, 2.0 ** -24,
                    2.0 ** -23, 2.0 ** -21, 2.0 ** -18])
    r64 = r[pos].astype(np.float64)
    t64 = atol + rtol * np.abs(r64)
    d64 = t64 * (1.0 + rel[rng.integers(0, rel.size, pos.size)])
    c[pos] = (r64 + np.where(rng.random(pos.size) < 0.5, -1.0, 1.0) * d64).astype(np.float32)
    c_hi = c.copy()
    c_hi[1000] = r[1000] + np.float32(4.0) * np.float32(atol + rtol * abs(float(r[1000])) + 1e-3)
    cases = [(_store(c_hi, dt), _store(r, dt), dt) for dt in DTYPES]
    cases.append((_store(c, oracle.F32), _store(r, oracle.F32), oracle.F32))
    res = vc.vcheck_nearpass([(_tensor(torch, cr, dt), _tensor(torch, rr, dt))
                              for cr, rr, dt in cases], atol, rtol)
    for i, ((cr, rr, dt), got) in enumerate(zip(cases, res)):
        want = oracle.nearpass(_view(cr, dt), _view(rr, dt), dt, atol, rtol)
        for k in ("numel", "n_pairs", "n_fail", "n_zero_tol", "argmax_ratio", "max_ulp_fail",
                  "ratio_hist", "ulp_hist"):
            assert got[k] == want[k], (i, dt, k, got[k], want[k])
        assert np.float64(got["max_ratio"]).tobytes() == np.float64(want["max_ratio"]).tobytes()
    # the binary32 case without the early failure: its largest ratio is one
    # of the planted boundary pairs, and some of them fail
    last = res[-1]
    assert last["n_fail"] > 0 and last["argmax_ratio"] in set(pos.tolist())


def test_nearpass_largest_unit():
    """Cases totalling 2^29 pairs take the largest wave range (32768 pairs:
    64 full steps per wave through the inner usual-step loop, each step's
    loads one step ahead) and chunks of 131072 pairs; each case of 2^27
    pairs spans four merge groups. Most pairs are equal, a sparse few
    perturbed; a late new largest ratio below 1 (c = 1 + 2^-9 against 1:
    0.977 in binary16 and binary32, equal in bfloat16) and its exact tie, a
    late failure, zeros of both signs and a late infinity sit in every
    case."""
    import torch

    rng = np.random.default_rng(2608_74)
    n = 1 << 27
    atol, rtol = 1e-3, 1e-3
    cases = []
    for dt in (oracle.F16, oracle.F16, oracle.BF16, oracle.F32):
        r = rng.uniform(0.5, 2.0, n).astype(np.float32)
        r[rng.random(n) < 0.5] *= -1
        c = r.copy()
        pert = rng.choice(n, n // 10000, replace=False)
        c[pert] = r[pert] * (1 + 3e-4 * rng.standard_normal(pert.size)).astype(np.float32)
        zeros = rng.choice(n, n // 50, replace=False)
        r[zeros], c[zeros] = -0.0, 0.0
        late = n - 6 * 131072 + 1001
        r[[late, late + 4096]] = 1.0
        c[[late, late + 4096]] = np.float32(1.0 + 2.0 ** -9)
        r[n - 3 * 131072 + 5], c[n - 3 * 131072 + 5] = 1.0, 1.5  # a late failure
        c[n - 17] = np.inf
        cases.append((_store(c, dt), _store(r, dt), dt))
    print("nearpass largest unit: %d cases of %d pairs" % (len(cases), n), flush=True)
    res = vc.vcheck_nearpass([(_tensor(torch, cr, dt), _tensor(torch, rr, dt))
                              for cr, rr, dt in cases], atol, rtol)
    for (cr, rr, dt), got in zip(cases, res):
        want = oracle.nearpass(_view(cr, dt), _view(rr, dt), dt, atol, rtol)
        for k in ("numel", "n_pairs", "n_fail", "n_zero_tol", "argmax_ratio", "max_ulp_fail",
                  "ratio_hist", "ulp_hist"):
            assert got[k] == want[k], (dt, k, got[k], want[k])
        assert np.float64(got["max_ratio"]).tobytes() == np.float64(want["max_ratio"]).tobytes()
        assert got["n_fail"] > 0
