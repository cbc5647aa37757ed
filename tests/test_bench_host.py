"""Host-side checks of bench.py (CPU only): the multi-GPU refusal, the
source key that guards the stored HBM counter readings, the reading of
rocprofv3 counter output into traffic figures, the host description of the
CPU baseline and the algorithmic byte count of a workload."""
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
    plan = "unit = 1024;\n"
    assert bench.kernel_hash([src, plan]) == bench.kernel_hash([same, plan])
    assert bench.kernel_hash([src, plan]) != bench.kernel_hash([other, plan])
    # the key covers every listed source, the planner included
    assert bench.kernel_hash([src, plan]) != bench.kernel_hash([src, "unit = 2048;\n"])
    names = [os.path.basename(p) for p in bench.KERNEL_SRCS]
    assert {"vcheck_kernels.hip", "vcheck_probe.hip", "vcheck_api.cpp"} <= set(names)


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    f = tmp_path / "traffic.json"
    key = bench.kernel_hash()
    f.write_text(json.dumps({"w": {"kernel_sha": key, "hbm_bytes_per_launch": 123},
                             "old": {"kernel_sha": "0" * 16, "hbm_bytes_per_launch": 456}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.traffic_for("w") == 123
    assert bench.traffic_for("old") is None
    assert bench.traffic_for("missing") is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "absent.json"))
    assert bench.traffic_for("w") is None


def _pmc_csv(path, rows):
    path.mkdir(parents=True)
    with open(path / "run_counter_collection.csv", "w") as f:
        f.write('"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value"\n')
        for i, (k, c, v) in enumerate(rows):
            f.write('%d,"%s","%s",%f\n' % (i, k, c, v))


def test_short_kernel_names():
    assert bench.short_kernel("void vck::(anonymous namespace)::main_kernel<1, 1, false>"
                              "(vck::Params)") == "main_kernel<1, 1, false>"
    assert bench.short_kernel("vck::(anonymous namespace)::finalize_kernel(vck::Params)") \
        == "finalize_kernel"


def test_record_traffic_from_counter_output(tmp_path, monkeypatch):
    main = "void vck::(anonymous namespace)::main_kernel<0, 1, true>(vck::Params)"
    other = "void vck::(anonymous namespace)::finalize_kernel(vck::Params)"
    copy = "__amd_rocclr_copyBuffer"
    _pmc_csv(tmp_path / "f", [(main, "FETCH_SIZE", 100.0), (main, "FETCH_SIZE", 300.0),
                              (main, "FETCH_SIZE", 200.0), (other, "FETCH_SIZE", 9e9)])
    _pmc_csv(tmp_path / "w", [(main, "WRITE_SIZE", 4.0)])
    _pmc_csv(tmp_path / "cf", [(copy, "FETCH_SIZE", 524288.0)])  # half of 1 GiB
    _pmc_csv(tmp_path / "cw", [(copy, "WRITE_SIZE", 1048576.0)])
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))

    class A:
        fetch, write, copy_fetch, copy_write = (str(tmp_path / d) for d in ("f", "w", "cf", "cw"))
        kernel, copy_kernel, kernel_label = "main_kernel", "copyBuffer", "main_kernel<0, 1, true>"
        workload, alg_bytes = "wl", 409600

    bench.record_traffic(A)
    ent = json.loads(out.read_text())["wl"]
    # median fetch 200 KiB, scaled x2 by the copy; write 4 KiB, scale 1
    assert ent["hbm_bytes_per_launch"] == 200 * 1024 * 2 + 4 * 1024
    assert ent["kernel_sha"] == bench.kernel_hash()
    assert bench.traffic_for("wl") == ent["hbm_bytes_per_launch"]


def test_host_info_fields():
    h = bench.host_info()
    assert h["os_cpu_count"] == os.cpu_count()
    assert h["affinity"] == len(os.sched_getaffinity(0))
    assert "model" in h


def test_algorithmic_bytes():
    w = wl.fp16_batch(device="cpu", n_cases=2, rows=64, cols=128)
    assert bench.algorithmic_bytes(w) == 2 * 2 * 64 * 128 * 2
    w = wl.fp32_integrity(device="cpu", n_cases=6, rows=8, cols=16)
    classes = w.meta["classes"]
    n_copy = sum(int(k) == wl.CLASS_COPY for k in classes)
    per_case = 8 * 16 * 4
    assert bench.algorithmic_bytes(w, classes) == 6 * 2 * per_case + n_copy * per_case
