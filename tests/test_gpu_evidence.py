"""GPU tests of the full-coverage evidence: content hashes against the
oracle (every storage type, empty, ragged, misaligned and multi-chunk
tensors), the two-stage escalation with its signed evidence record, and the
best-candidate bookkeeping driven by escalation records, checked against
decisions derived from the oracle's suite verdicts on the same bytes."""
import numpy as np
import pytest

import oracle
from paper_2608_02712_amd import vcheck as vc
from tests import oracle_pins

pytestmark = pytest.mark.gpu


def _tensor(torch, raw, dt):
    if dt == oracle.F32:
        return torch.from_numpy(raw.view(np.float32).copy())
    t = torch.from_numpy(raw.view(np.int16).copy())
    return t.view(torch.float16 if dt == oracle.F16 else torch.bfloat16)


def test_content_hash_parity():
    import torch

    rng = np.random.default_rng(2608_64)
    batch = []
    for dt in (oracle.F32, oracle.F16, oracle.BF16):
        for n in (0, 1, 7, 513, 4099, 300001):
            raw = oracle_pins.random_pairs(rng, n, dt)[0]
            batch.append((_tensor(torch, raw, dt).cuda(), raw, dt))
        raw = oracle_pins.random_pairs(rng, 9001, dt)[0]
        buf = _tensor(torch, np.concatenate([raw[:1], raw]), dt).cuda()
        batch.append((buf[1:], raw, dt))  # misaligned view
    big = rng.integers(0, 2 ** 16, 1 << 25, dtype=np.uint32).astype(np.uint16)
    batch.append((_tensor(torch, big, oracle.F16).cuda(), big, oracle.F16))
    print("content hash: %d tensors" % len(batch), flush=True)
    got = vc.vcheck_content_hash([t for t, _, _ in batch])
    for i, ((t, raw, dt), h) in enumerate(zip(batch, got)):
        want = oracle.content_hash(raw.view(np.float32) if dt == oracle.F32 else raw, dt)
        assert h == want, (i, t.dtype, t.numel(), hex(h), hex(want))
    assert got == vc.vcheck_content_hash([t for t, _, _ in batch])


def test_escalation_and_evidence(tmp_path):
    import torch

    g = torch.Generator(device="cuda").manual_seed(2608_65)

    def case(n, bad=False):
        r = torch.randn(n, generator=g, device="cuda")
        c = r + 1e-6 * torch.randn(n, generator=g, device="cuda")
        if bad:
            c[n // 2] += 1.0
        return c, r

    compact = [case(1000), case(4097)]
    extended = compact + [case(1 << 20), case(333, bad=True)]
    tols = [(1e-4, 1e-4)]
    path = tmp_path / "evidence.json"
    rec = vc.escalate(compact, extended, tols, evidence_path=str(path))
    assert rec["compact"]["match_rate"] == [1.0]
    assert rec["extended"] is not None and rec["extended"]["n_cases"] == 4
    assert rec["extended"]["cases"][3]["pass"] == [0]
    assert rec["extended"]["match_rate"] == [0.75] and not rec["accepted"]
    assert vc.verify_evidence(rec)
    import json
    assert vc.verify_evidence(json.loads(path.read_text()))
    # the hashes in the record are the tensors' content hashes
    c0, r0 = compact[0]
    assert rec["compact"]["cases"][0]["cand_hash"] == "%016x" % vc.vcheck_content_hash([c0])[0]
    # editing the record, or re-running on a changed output, is detected
    forged = json.loads(json.dumps(rec))
    forged["extended"]["cases"][3]["pass"] = [1]
    assert not vc.verify_evidence(forged)
    compact[1][0][7] += 1e-7
    rec2 = vc.escalate(compact, extended[:2], tols)
    assert rec2["compact"]["cases"][1]["cand_hash"] != rec["compact"]["cases"][1]["cand_hash"]
    assert rec2["compact"]["case_set_hash"] != rec["compact"]["case_set_hash"]
    assert rec2["accepted"]
    # a compact set below the gate stops before the extended set
    rec3 = vc.escalate([case(100, bad=True)], extended, tols)
    assert rec3["extended"] is None and not rec3["accepted"]


# ---- best-candidate bookkeeping from escalation records --------------------

SPECS = [(oracle.F32, (64, 33)), (oracle.F16, (1000,)),            # the compact set
         (oracle.BF16, (7, 129)), (oracle.F32, (4097,)), (oracle.F16, (3, 5, 7)),
         (oracle.F32, (2, 2048))]
N_COMPACT = 2


def _raw_of(x32, dt):
    return x32.view(np.uint32).copy() if dt == oracle.F32 else oracle_pins.to_raw16(x32, dt)


def _candidate(kind, r32, x32, rng):
    """A candidate output of one case: exact, inside the tolerance, one
    faulty element, all zero, constant fill or a copy of the input."""
    c = r32.copy()
    if kind == "near":
        c = c + np.float32(2e-4) * np.abs(c) * rng.uniform(-1, 1, c.size).astype(np.float32)
    elif kind == "fault":
        c[c.size // 3] += np.float32(0.5)
    elif kind == "zero":
        c[:] = 0.0
    elif kind == "const":
        c[:] = np.float32(0.25)
    elif kind == "copy":
        c = x32.copy()
    return c.astype(np.float32)


def test_best_candidate_from_escalation():
    import torch

    rng = np.random.default_rng(2608_66)
    tols = [(1e-3, 1e-3), (1e-2, 1e-2)]
    base = []  # per case: storage type, shape, input x and reference r (binary32 values)
    for dt, shape in SPECS:
        n = int(np.prod(shape))
        x = rng.standard_normal(n).astype(np.float32)
        r = (x * np.float32(0.5) + np.float32(1.0)).astype(np.float32)
        # round-trip through the storage type, so the binary32 values are exact
        xr, rr = _raw_of(x, dt), _raw_of(r, dt)
        x = oracle_pins.lib_decode(xr, dt) if dt != oracle.F32 else x
        r = oracle_pins.lib_decode(rr, dt) if dt != oracle.F32 else r
        base.append((dt, shape, x.astype(np.float32), r.astype(np.float32)))
    # repair attempts: one candidate kind per case
    attempts = [
        ("a0", ["fault", "exact", "exact", "exact", "exact", "exact"]),   # compact fails
        ("a1", ["exact", "near", "fault", "exact", "near", "exact"]),     # 5 of 6
        ("a2", ["exact", "exact", "fault", "fault", "exact", "exact"]),   # 4 of 6
        ("a3", ["near", "exact", "zero", "exact", "exact", "exact"]),     # detector flag
        ("a4", ["exact", "exact", "exact", "near", "exact", "exact"]),    # all certified
        ("a5", ["exact", "exact", "copy", "exact", "const", "exact"]),    # two flags
        ("a6", ["exact", "fault", "exact", "exact", "exact", "exact"]),   # compact fails
        ("a7", ["exact", "exact", "exact", "exact", "exact", "exact"]),   # ties the best
    ]
    got_bc, want_bc = vc.BestCandidate(), vc.BestCandidate()
    got_dec, want_dec, scores = [], [], []
    for name, kinds in attempts:
        dev_cases, orc = [], []
        for (dt, shape, x, r), kind in zip(base, kinds):
            c = _candidate(kind, r, x, rng)
            craw, rraw, xraw = _raw_of(c, dt), _raw_of(r, dt), _raw_of(x, dt)
            dev = [_tensor(torch, a, dt).reshape(shape).cuda() for a in (craw, rraw, xraw)]
            dev_cases.append((dev[0], dev[1], [dev[2]]))
            o = oracle.validate_case(craw.view(np.float32) if dt == oracle.F32 else craw,
                                     rraw.view(np.float32) if dt == oracle.F32 else rraw,
                                     dt, shape, tols, primary=0,
                                     inputs=[(xraw.view(np.float32) if dt == oracle.F32
                                              else xraw, dt)])
            orc.append(o)
        rec = vc.escalate(dev_cases[:N_COMPACT], dev_cases, tols, primary=0, gate=1.0)
        got_dec.append(got_bc.record_evidence(name, rec))

        def rate(results):
            m = np.array([o.mismatches for o in results], dtype=np.uint64)
            st = np.zeros(len(results), dtype=np.int32)  # every case is evaluated
            fl = np.array([o.integrity["flags"] for o in results], dtype=np.uint32)
            return oracle.suite(m, st, fl)[1]

        compact_rate = rate(orc[:N_COMPACT])
        score = float(rate(orc)[0]) if compact_rate[0] >= 1.0 else 0.0
        want_dec.append(want_bc.record(name, score))
        scores.append(score)
        assert rec["compact"]["match_rate"] == [float(v) for v in compact_rate], name
        if compact_rate[0] >= 1.0:
            assert rec["extended"]["match_rate"][0] == score, name
            assert rec["accepted"] == (score == 1.0), name
        else:
            assert rec["extended"] is None and not rec["accepted"], name
        # the evidence rows carry the oracle's verdicts
        for stage, cases in (("compact", orc[:N_COMPACT]), ("extended", orc)):
            if rec[stage] is None:
                continue
            for row, o in zip(rec[stage]["cases"], cases):
                assert row["mismatches"] == o.mismatches, (name, stage)
                assert row["flags"] == o.integrity["flags"], (name, stage)
    assert got_dec == want_dec, (got_dec, want_dec, scores)
    assert scores == [0.0, 5 / 6, 4 / 6, 5 / 6, 1.0, 4 / 6, 0.0, 1.0]
    assert got_dec == ["promote", "promote", "continue", "rollback", "promote", "continue",
                       "rollback", "continue"]
    assert (got_bc.best, got_bc.best_score) == ("a4", 1.0)
