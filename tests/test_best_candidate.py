"""The best-candidate bookkeeping (CPU): promotion on a strictly higher
match rate, rollback after two consecutive non-improving attempts."""
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
    rec["digest"] = vc._evidence_digest(rec)
    assert b.record_evidence("r0", rec) == "promote" and b.best_score == 0.8
    forged = dict(rec, extended={"match_rate": [1.0]})
    assert b.record_evidence("r1", forged) == "continue"  # digest no longer matches: score 0
    stopped = {"primary": 0, "extended": None, "compact": {}}
    stopped["digest"] = vc._evidence_digest(stopped)
    assert b.record_evidence("r2", stopped) == "rollback"
