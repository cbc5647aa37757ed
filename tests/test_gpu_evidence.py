"""GPU tests of the full-coverage evidence: content hashes against the
oracle (every storage type, empty, ragged, misaligned and multi-chunk
tensors), and the two-stage escalation with its evidence record."""
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
