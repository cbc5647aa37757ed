"""GPU parity on the five synthetic workloads at their full sizes, in the
launch configuration the benchmark times (one sweep call per workload).
The oracle checks every output of sampled cases element for element; the
closed forms of the injected faults are checked for every case."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from paper_2608_02712_amd import vcheck as vc
from tests.gpu_util import assert_integrity, assert_stats, oracle_case

pytestmark = pytest.mark.gpu


def run_sweep(w):
    sw = vc.Sweep([(c.cand, c.ref, c.inputs) for c in w.cases], w.tols, primary=w.primary,
                  tile=w.tile, k=w.k or 0, integrity=w.integrity)
    sw.launch()
    return sw.results()


def check_case(res, w, i, tag):
    c = w.cases[i]
    o = oracle_case(c.cand, c.ref, w.tols, primary=w.primary, tile=w.tile, k=w.k,
                    inputs=c.inputs if w.integrity else None)
    assert_stats(res["stats"][i], o.stats, tag)
    assert [int(x) for x in res["mismatches"][i]] == o.mismatches, tag
    if w.tile is not None:
        assert np.array_equal(res["tile_maps"][i], o.tile_map), tag + " tile map"
    if w.k:
        assert np.array_equal(res["first_k"][i], o.first_k), tag + " first-k"
    if w.integrity:
        assert_integrity(res["integrity"][i], o.integrity, tag)
    return o


def test_fp32_single_full():
    w = wl.fp32_single("cuda")
    ref = w.cases[0].ref
    assert ref[1000:, 960:].abs().min().item() > 2e-5
    res = run_sweep(w)
    check_case(res, w, 0, "cfg1")
    st = res["stats"][0]
    assert st["mismatches"] == 1536
    assert res["first_k"][0].tolist() == list(range(1024960, 1025024))
    tm = res["tile_maps"][0].reshape(32, 32)
    assert tm[31, 30] == 768 and tm[31, 31] == 768 and int(tm.sum()) == 1536
    assert res["match_rate"].tolist() == [0.0]


def test_fp16_batch_full():
    """Every case through the oracle, and every case's tile map and first-k
    against the closed form of its faults: the shifted tile (4096
    mismatches) plus one per planted NaN, nothing else."""
    w = wl.fp16_batch("cuda")
    res = run_sweep(w)
    rows = cols = 2048
    t = w.meta["tile_size"]
    for i, f in enumerate(w.meta["faults"]):
        check_case(res, w, i, "cfg2 case %d" % i)
        st = res["stats"][i]
        assert st["mismatches"] == 4099 and st["nan_cand"] == 3, i
        ti, tj = f["tile"]
        want = np.zeros((rows // t, cols // t), dtype=np.uint32)
        want[ti, tj] = t * t
        for p in f["nans"]:
            want[(p // cols) // t, (p % cols) // t] += 1
        assert np.array_equal(res["tile_maps"][i].reshape(want.shape), want), i
        blk = ((ti * t + np.arange(t))[:, None] * cols + tj * t + np.arange(t)[None, :]).ravel()
        fk = np.sort(np.concatenate([blk, np.asarray(f["nans"], dtype=np.int64)]))[:w.k]
        assert res["first_k"][i].tolist() == fk.tolist(), i
    assert res["match_rate"].tolist() == [0.0]


def test_bf16_bursts_full():
    w = wl.bf16_bursts("cuda")
    res = run_sweep(w)
    o = check_case(res, w, 0, "cfg3")
    assert res["stats"][0]["inf_cand"] == 512
    sc = w.meta["scaled"]
    c = w.cases[0].cand.view(-1)[torch.as_tensor(sc, device="cuda")].double()
    r = w.cases[0].ref.view(-1)[torch.as_tensor(sc, device="cuda")].double()
    bad = ~torch.isclose(c.cpu(), r.cpu(), rtol=1.6e-2, atol=1e-2)
    assert o.mismatches == [512 + int(bad.sum())]


def test_fp32_sweep_full():
    w = wl.fp32_sweep("cuda")
    res = run_sweep(w)
    sample = sorted(set(range(5)) | set(range(5, 500, 9)) | set(w.meta["faulted"][:20]))
    for i in sample:
        check_case(res, w, i, "cfg4 case %d %r" % (i, w.meta["shapes"][i]))
    for i, f in enumerate(w.meta["faults"]):
        m = res["mismatches"][i]
        assert int(m[2]) == int(m[3]) == len(f), (i, m)
        assert all(int(a) >= int(b) for a, b in zip(m, m[1:])), (i, m)
        assert res["first_k"][i][:len(f)].tolist() == f.tolist()
        tm = res["tile_maps"][i]
        assert int(tm[:-1].sum()) == 0 and int(tm[-1]) == len(f)
    assert res["match_rate"][3] == 0.5 and res["match_rate"][2] == 0.5


def test_fp32_integrity_full():
    w = wl.fp32_integrity("cuda")
    res = run_sweep(w)
    classes = w.meta["classes"]
    want = {wl.CLASS_CORRECT: 0, wl.CLASS_COPY: vc.FLAG_INPUT_COPY, wl.CLASS_ZERO: vc.FLAG_ALL_ZERO,
            wl.CLASS_CONSTANT: vc.FLAG_CONSTANT, wl.CLASS_BF16: vc.FLAG_LOWPREC_BF16}
    for k in range(5):
        idx = np.flatnonzero(classes == k)[:2]
        for i in idx:
            check_case(res, w, int(i), "cfg5 case %d class %s" % (i, wl.CLASS_NAMES[k]))
    for i, k in enumerate(classes):
        g = res["integrity"][i]
        assert g["flags"] == want[int(k)], (i, int(k), g["flags"])
        assert g["copy_input"] == (0 if k == wl.CLASS_COPY else -1)
        if k == wl.CLASS_CORRECT:
            assert res["stats"][i]["mismatches"] == 0
        if k == wl.CLASS_ZERO:
            assert res["stats"][i]["max_rel"] == 1.0
    assert res["match_rate"][0] == int((classes == wl.CLASS_CORRECT).sum()) / 256
