"""Host-side checks of bench.py (CPU only): the multi-GPU refusal, the
kernel-source key that guards the stored HBM counter readings, and the
algorithmic byte count of a workload."""
import json
import os
import subprocess
import sys

import bench
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_refuses_several_gpus():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_kernel_key_ignores_comments_only():
    src = "int a = 1;  // one\n\n// note\nint b = a + 1;\n"
    same = "int a = 1;\n// other note\nint b = a + 1;  // two\n"
    other = "int a = 2;\nint b = a + 1;\n"
    assert bench.kernel_hash(src) == bench.kernel_hash(same)
    assert bench.kernel_hash(src) != bench.kernel_hash(other)


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    f = tmp_path / "traffic.json"
    key = bench.kernel_hash()
    f.write_text(json.dumps({"w": {"kernel_sha": key, "hbm_bytes_per_launch": 123},
                             "old": {"kernel_sha": "0" * 16, "hbm_bytes_per_launch": 456}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.traffic_for("w", None) == 123
    assert bench.traffic_for("old", None) is None
    assert bench.traffic_for("missing", None) is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "absent.json"))
    assert bench.traffic_for("w", None) is None


def test_algorithmic_bytes():
    w = wl.fp16_batch(device="cpu", n_cases=2, rows=64, cols=128)
    assert bench.algorithmic_bytes(w) == 2 * 2 * 64 * 128 * 2
    w = wl.fp32_integrity(device="cpu", n_cases=6, rows=8, cols=16)
    classes = w.meta["classes"]
    n_copy = sum(int(k) == wl.CLASS_COPY for k in classes)
    per_case = 8 * 16 * 4
    assert bench.algorithmic_bytes(w, classes) == 6 * 2 * per_case + n_copy * per_case
