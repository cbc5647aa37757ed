"""GPU parity of the tensor-statistics probe against the oracle.

One batch mixes every storage type, empty, single-element, ragged and
misaligned tensors, random bit patterns of every class (NaN, +-Inf, +-0,
subnormals, huge values), repeated extremes (the first index must win) and
one tensor large enough to span several merge groups. Counts, extremes and
their indices and the histogram must match exactly; each binary64 sum
within 1e-6 of the sum of its terms' magnitudes."""
import numpy as np
import pytest

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins

pytestmark = pytest.mark.gpu

EXACT = ("numel", "nan", "inf", "zero", "n_finite", "argmin", "argmax", "hist")


def _raw_to_tensor(torch, raw, dtype):
    if dtype == oracle.F32:
        return torch.from_numpy(raw.view(np.float32).copy())
    t = torch.from_numpy(raw.view(np.int16).copy())
    return t.view(torch.float16 if dtype == oracle.F16 else torch.bfloat16)


def _batch(torch, rng):
    """(device tensor, raw host storage, dtype code) of the probe batch."""
    out = []
    for dt in (oracle.F32, oracle.F16, oracle.BF16):
        for n in (0, 1, 7, 513, 4099, 100003):
            cand, ref = oracle_pins.random_pairs(rng, n, dt)
            out.append((cand, dt))
            out.append((ref, dt))
        # normal data with planted extremes: equal minima and maxima (first
        # index wins), zeros of both signs, NaN and Inf
        x = rng.standard_normal(300001).astype(np.float32)
        x[[5, 70000, 250000]] = -9.0
        x[[9, 80000]] = 9.0
        x[[1, 2]] = [-0.0, 0.0]
        x[[3, 4]] = [np.nan, np.inf]
        raw = x.view(np.uint32).copy() if dt == oracle.F32 else oracle_pins.to_raw16(x, dt)
        out.append((raw, dt))
    dev = []
    for raw, dt in out:
        t = _raw_to_tensor(torch, raw, dt).cuda()
        dev.append((t, raw, dt))
    # misaligned views: one element past the start of a buffer
    for dt in (oracle.F32, oracle.F16):
        raw = oracle_pins.random_pairs(rng, 5001, dt)[0]
        buf = _raw_to_tensor(torch, np.concatenate([raw[:1], raw]), dt).cuda()
        dev.append((buf[1:], raw, dt))
    # a tensor spanning several merge groups (more than 256 chunks)
    big = rng.standard_normal(1 << 25).astype(np.float32)
    big[rng.choice(big.size, 1000, replace=False)] = np.nan
    big[123456789 % big.size] = 1e30
    dev.append((torch.from_numpy(big).cuda(), big.view(np.uint32), oracle.F32))
    return dev


def _check(got, want, tag):
    for k in EXACT:
        assert got[k] == want[k], (tag, k, got[k], want[k])
    for k in ("min", "max"):
        assert np.float64(got[k]).tobytes() == np.float64(want[k]).tobytes(), (tag, k)
    for k, mag in (("sum", want["sum_abs"]), ("sum_sq", want["sum_sq"]),
                   ("sum_abs", want["sum_abs"])):
        assert abs(got[k] - want[k]) <= 1e-6 * mag, (tag, k, got[k], want[k])


def test_probe_batch_parity():
    import torch

    rng = np.random.default_rng(2608_61)
    batch = _batch(torch, rng)
    print("probe: batch of %d tensors" % len(batch), flush=True)
    res = vc.vcheck_tensor_stats([t for t, _, _ in batch])
    assert len(res) == len(batch)
    for i, ((t, raw, dt), got) in enumerate(zip(batch, res)):
        want = oracle.tensor_stats(raw.view(np.float32) if dt == oracle.F32 else raw, dt)
        _check(got, want, "tensor %d (%s, %d elements)" % (i, t.dtype, t.numel()))


def test_probe_repeat_is_bitwise_identical():
    import torch

    rng = np.random.default_rng(2608_62)
    x = torch.from_numpy(rng.standard_normal(3_000_001).astype(np.float32)).cuda()
    ts = vc.TensorStats([x, x.half(), x.bfloat16()])
    ts.launch()
    a = ts.results()
    ts.launch()
    b = ts.results()
    assert a == b


def test_probe_extreme_magnitudes():
    """Values far outside [2^-60, 2^60) (binary32 and bfloat16 subnormals,
    huge values) next to ordinary ones: the sums keep them."""
    import torch

    x = np.array([1e-30, 3e-38, 1e-45, 1.5, -2.5e30, 3e38, -3e38, 0.0, 1e-20, 7.0] * 301,
                 dtype=np.float32)
    tiny = np.full(1001, 1e-30, dtype=np.float32)
    batch = [(x.view(np.uint32), oracle.F32), (tiny.view(np.uint32), oracle.F32),
             (oracle_pins.to_raw16(x, oracle.BF16), oracle.BF16),
             (oracle_pins.to_raw16(tiny, oracle.BF16), oracle.BF16)]
    tensors = [_raw_to_tensor(torch, raw, dt).cuda() for raw, dt in batch]
    res = vc.vcheck_tensor_stats(tensors)
    for i, ((raw, dt), got) in enumerate(zip(batch, res)):
        want = oracle.tensor_stats(raw.view(np.float32) if dt == oracle.F32 else raw, dt)
        _check(got, want, "extreme %d" % i)
        assert got["sum_sq"] > 0.0


def test_probe_largest_unit():
    """A batch of 2^29 elements takes the largest wave range (32768 elements:
    64 full steps per wave through the inner usual-step loop) and chunks of
    131072 elements; each tensor of 2^27 elements spans four merge groups.
    Late strict extremes, their ties, zeros of both signs, binary16
    subnormals, NaN and Inf sit in every tensor."""
    import torch

    rng = np.random.default_rng(2608_63)
    n = 1 << 27
    batch = []
    for dt in (oracle.F16, oracle.F16, oracle.BF16, oracle.F32):
        x = rng.standard_normal(n, dtype=np.float32)
        x[rng.choice(n, n // 50, replace=False)] = 0.0
        x[rng.choice(n, 1000, replace=False)] = -0.0
        x[rng.choice(n, 1000, replace=False)] = 3e-7  # binary16 subnormal
        lo, hi = n - 5 * 131072 + 77, n - 3 * 131072 + 12345
        x[[lo, hi]] = [-50.0, 60.0]          # strict extremes late in a chunk
        x[[lo + 4096, hi + 9]] = [-50.0, 60.0]  # their ties: the first index wins
        x[[17, n // 3, n - 1]] = [np.nan, np.inf, np.nan]
        raw = x.view(np.uint32).copy() if dt == oracle.F32 else oracle_pins.to_raw16(x, dt)
        batch.append((raw, dt))
    print("probe largest unit: %d tensors of %d elements" % (len(batch), n), flush=True)
    tensors = [_raw_to_tensor(torch, raw, dt).cuda() for raw, dt in batch]
    res = vc.vcheck_tensor_stats(tensors)
    for i, ((raw, dt), got) in enumerate(zip(batch, res)):
        want = oracle.tensor_stats(raw.view(np.float32) if dt == oracle.F32 else raw, dt)
        _check(got, want, "large tensor %d" % i)
        assert (got["argmin"], got["argmax"]) == (n - 5 * 131072 + 77, n - 3 * 131072 + 12345)
