"""The best-candidate bookkeeping (CPU): promotion on a strictly higher
match rate, rollback after two consecutive non-improving attempts, and the
signature check of the evidence records it scores."""
import pytest

from paper_2608_02712_amd import vcheck as vc


def test_promote_and_rollback_sequence():
    b = vc.BestCandidate()
    got = [b.record(n, s) for n, s in [("a0", 0.5), ("a1", 0.75), ("a2", 0.75), ("a3", 0.6),
                                         ("a4", 0.9), ("a5", 0.2), ("a6", 0.9), ("a7", 0.95)]]
    assert got == ["promote", "promote", "continue", "rollback", "promote", "continue",
                   "rollback", "promote"]
    assert (b.best, b.best_score) == ("a7", 0.95)


def test_patience_and_first_attempt():
    b = vc.BestCandidate(patience=1)
    assert b.record("x", 0.0) == "promote"  # the first attempt is the best so far
    assert b.record("y", 0.0) == "rollback"
    assert b.record("z", 0.0) == "rollback"
    with pytest.raises(ValueError):
        vc.BestCandidate(patience=0)


def test_evidence_scores():
    b = vc.BestCandidate()
    rec = {"primary": 0, "extended": {"match_rate": [0.8]}, "compact": {}}
    rec["mac"] = vc._evidence_mac(rec)
    assert b.record_evidence("r0", rec) == "promote" and b.best_score == 0.8
    forged = dict(rec, extended={"match_rate": [1.0]})
    assert b.record_evidence("r1", forged) == "continue"  # signature no longer matches: score 0
    stopped = {"primary": 0, "extended": None, "compact": {}}
    stopped["mac"] = vc._evidence_mac(stopped)
    assert b.record_evidence("r2", stopped) == "rollback"


def test_forged_record_with_recomputed_hash_is_rejected():
    """A forger who edits a record and recomputes a plain SHA-256 digest of it
    (or signs it with another key) does not hold the engine's key."""
    import hashlib
    import json

    rec = {"primary": 0, "extended": {"match_rate": [0.5]}, "compact": {}}
    rec["mac"] = vc._evidence_mac(rec)
    assert vc.verify_evidence(rec)
    forged = {"primary": 0, "extended": {"match_rate": [1.0]}, "compact": {}}
    body = json.dumps(forged, sort_keys=True, separators=(",", ":")).encode()
    forged["mac"] = hashlib.sha256(body).hexdigest()
    assert not vc.verify_evidence(forged)
    forged["mac"] = vc._evidence_mac({k: v for k, v in forged.items() if k != "mac"},
                                     key=b"not the engine's key")
    assert not vc.verify_evidence(forged)
    assert vc.BestCandidate().record_evidence("f", forged) == "promote"  # scored 0.0
    # a caller-held key verifies across processes
    key = b"k" * 32
    signed = dict(rec)
    signed["mac"] = vc._evidence_mac({k: v for k, v in rec.items() if k != "mac"}, key=key)
    assert vc.verify_evidence(signed, key=key) and not vc.verify_evidence(signed)
    assert not vc.verify_evidence({"primary": 0})  # unsigned
