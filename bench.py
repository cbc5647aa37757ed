#!/usr/bin/env python3
"""Throughput of the validation hot path on one MI355X.

One step = one vcheck_sweep call over a whole synthetic workload (tolerance
gate, NaN/Inf counts, exact max abs/rel, error sums, tile map, first-k,
detectors and suite match rate: every stage of the path), inputs resident in
HBM. The Infinity Cache is flushed (512 MiB write) before every step, outside
the timed interval; each step is timed with HIP events on the launch stream.
The streaming kernels are timed in a second pass with events the library
records around them.

Headline line: the largest single-GPU workload, the integrity batch of 256
fp32 cases of 4096x4096 (34.4 GB of cand and ref per call). ``probe``
reports the tensor-statistics probe over the 128 cand and ref tensors of the
fp16 batch (64 cases of 2048x2048) in one call, ``nearpass`` the near-pass
statistics of its 64 cases, ``content_hash`` the content hashes of its 128
tensors. ``workloads`` holds the same figures for all five workloads,
measured in the same run. ``roofline`` reports the headline's streaming
kernel: achieved HBM bandwidth (algorithmic bytes / its event-timed average
duration) against the 8 TB/s peak, and the HBM bytes per launch from the
committed counter readings (profiles/traffic.json) when they were taken on
the current sources; ``cpu_baseline`` times the CPU oracle on a bounded
sample of the headline workload on this host.

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--headline-only]
       python bench.py --only N [--diag]    (one workload; --diag adds the probe,
                                             near-pass and hash over it)
       python bench.py --pmc-summary DIR... (medians of rocprofv3 --pmc output)
       python bench.py --record-traffic ... (profiles/traffic.json entry)
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "validated GB/s (ref+cand bytes) and % of HBM peak; test cases/sec"
HBM_PEAK_GBS = 8000.0
HEADLINE = 5  # the largest workload
DIAG_WORKLOAD = 2  # the fp16 batch: probe, near-pass and hash are timed over it
CSRC = os.path.join(ROOT, "paper_2608_02712_amd", "csrc")
KERNEL_SRCS = [os.path.join(CSRC, n) for n in
               ("vcheck_kernels.hip", "vcheck_probe.hip", "vcheck_api.cpp", "vcheck_internal.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def kernel_hash(texts=None):
    """Hash of the kernel sources and the planner (which sets unit sizes and
    launch shapes) with // comments and blank lines removed, so that stored
    counter readings stay valid across comment-only edits and lapse on any
    code change."""
    if texts is None:
        texts = []
        for path in KERNEL_SRCS:
            with open(path) as f:
                texts.append(f.read())
    code = []
    for text in texts:
        for line in text.splitlines():
            line = line.split("//", 1)[0].rstrip()
            if line:
                code.append(line)
        code.append("\x00")
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


def algorithmic_bytes(w, classes=None):
    """ref + cand bytes, plus operator-input bytes read while cand is a copy."""
    b = w.ref_cand_bytes
    if w.integrity and classes is not None:
        import workloads as wl

        for case, k in zip(w.cases, classes):
            if int(k) == wl.CLASS_COPY:
                b += sum(x.numel() * x.element_size() for x in case.inputs)
    return b


def prewarm(launch, seconds):
    """Untimed calls for about `seconds` before a measurement, so that the
    GPU's clocks have left the idle state (the CPU baseline or a workload's
    generation may precede it); nothing of it enters a timed region."""
    import torch

    if seconds <= 0:
        return
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(4):
            launch()
        torch.cuda.synchronize()


def time_sweep(sw, steps, warmup, flush, prewarm_s=0.0):
    """`steps` pairs of calls, the Infinity Cache flushed before every call:
    the first call of a pair is timed whole (events around the call only),
    the second has the streaming kernels timed alone (events the library
    records just before and after them; recording them adds a gap between
    the kernels, so they are not used for the call time)."""
    import torch
    from paper_2608_02712_amd import vcheck as vc

    prewarm(sw.launch, prewarm_s)
    for _ in range(warmup):
        sw.launch()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for quad in evs:
        for e in quad:
            e.record(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        flush.fill_(i & 0xFF)
        evs[i][0].record(stream)
        sw.launch(stream)
        evs[i][1].record(stream)
        flush.fill_((i + 1) & 0xFF)
        vc.vcheck_profile_events(evs[i][2], evs[i][3])
        sw.launch(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    call_ms = sorted(a.elapsed_time(b) for a, b, _, _ in evs)
    main_ms = [m0.elapsed_time(m1) for _, _, m0, m1 in evs]
    return call_ms, main_ms, wall


def measure(cfg, steps, warmup, flush, prewarm_s=0.0):
    import torch

    import workloads as wl
    from paper_2608_02712_amd import vcheck as vc

    t = time.perf_counter()
    w = wl.WORKLOADS[cfg]("cuda")
    torch.cuda.synchronize()
    log("workload %d (%s) generated in %.1f s" % (cfg, w.name, time.perf_counter() - t))
    sw = vc.Sweep([(c.cand, c.ref, c.inputs) for c in w.cases], w.tols, primary=w.primary,
                  tile=w.tile, k=w.k or 0, integrity=w.integrity)
    call_ms, main_ms, wall = time_sweep(sw, steps, warmup, flush, prewarm_s)
    res = sw.results()
    ms = call_ms[len(call_ms) // 2]
    main_avg = sum(main_ms) / len(main_ms)
    rc = w.ref_cand_bytes
    alg = algorithmic_bytes(w, w.meta.get("classes"))
    out = {
        "workload": w.name,
        "storage": {torch.float32: "fp32", torch.float16: "fp16",
                    torch.bfloat16: "bf16"}[w.cases[0].ref.dtype],
        "tols": [[float(a), float(r)] for (a, r, *_) in w.tols],
        "tile": list(w.tile) if w.tile else None,
        "k": w.k or 0,
        "integrity": bool(w.integrity),
        "n_cases": len(w.cases),
        "elements": w.numel,
        "ref_cand_bytes": rc,
        "ms_per_call": round(ms, 5),
        "gbps": round(rc / (ms * 1e-3) / 1e9, 2),
        "pct_hbm_peak": round(100.0 * rc / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
        "cases_per_s": round(len(w.cases) / (ms * 1e-3), 1),
        "main_kernel_ms": round(main_avg, 5),
        "main_kernel_alg_bytes": alg,
        "main_kernel_gbps": round(alg / (main_avg * 1e-3) / 1e9, 2),
        "match_rate": [float(x) for x in res["match_rate"]],
        "wall_s_timed_loop": round(wall, 3),
        "prewarm_s": prewarm_s,
    }
    log("workload %d: %.3f ms/call, %.1f GB/s (%.1f%% of peak), main kernel %.3f ms" % (
        cfg, ms, out["gbps"], out["pct_hbm_peak"], main_avg))
    return w, out


def measure_probe(w, steps, warmup, flush, prewarm_s=0.0):
    """The tensor-statistics probe over every cand and ref tensor of workload
    w in one call (the tensors of a batch of pipeline-boundary probes): call
    time per step (events around the call, cache flushed before it) and the
    streaming kernel's time (events the library records around it)."""
    import torch

    import oracle
    import workloads as wl
    from paper_2608_02712_amd import vcheck as vc

    tensors = [t for c in w.cases for t in (c.cand, c.ref)]
    ts = vc.TensorStats(tensors)
    prewarm(ts.launch, prewarm_s)
    for _ in range(warmup):
        ts.launch()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for quad in evs:  # (torch only times events it has seen recorded)
        for e in quad:
            e.record(stream)
    torch.cuda.synchronize()
    for i in range(steps):
        flush.fill_(i & 0xFF)
        evs[i][0].record(stream)
        ts.launch(stream)
        evs[i][1].record(stream)
    for i in range(steps):
        flush.fill_((i + 1) & 0xFF)
        vc.vcheck_profile_events(evs[i][2], evs[i][3])
        ts.launch(stream)
    torch.cuda.synchronize()
    call = sorted(a.elapsed_time(b) for a, b, _, _ in evs)[steps // 2]
    kern = sum(c.elapsed_time(d) for _, _, c, d in evs) / steps
    nbytes = sum(t.numel() * t.element_size() for t in tensors)
    # the oracle on a few tensors, one thread
    spent, done = 0.0, 0
    for t in tensors:
        raw = wl.raw_numpy(t).reshape(-1)
        t0 = time.perf_counter()
        oracle.tensor_stats(raw, wl.dtype_code(t.dtype))
        spent += time.perf_counter() - t0
        done += raw.nbytes
        if spent >= 2.0:
            break
    out = {
        "workload": "tensor statistics of the %d cand and ref tensors of %s" % (
            len(tensors), w.name),
        "n_tensors": len(tensors),
        "bytes": nbytes,
        "ms_per_call": round(call, 5),
        "gbps": round(nbytes / (call * 1e-3) / 1e9, 2),
        "pct_hbm_peak": round(100.0 * nbytes / (call * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
        "tensors_per_s": round(len(tensors) / (call * 1e-3), 1),
        "stream_kernel_ms": round(kern, 5),
        "stream_kernel_gbps": round(nbytes / (kern * 1e-3) / 1e9, 2),
        "oracle_one_thread_gbps": round(done / spent / 1e9, 4),
        "prewarm_s": prewarm_s,
    }
    log("probe: %.3f ms/call, %.1f GB/s (%.1f%% of peak), streaming kernel %.3f ms" % (
        call, out["gbps"], out["pct_hbm_peak"], kern))
    return out


def measure_nearpass(w, steps, warmup, flush, prewarm_s=0.0):
    """Near-pass statistics over every case of workload w at its primary
    tolerance pair, one call: call time (events around the call, cache
    flushed before it) and the streaming kernel's time."""
    import torch

    import oracle
    import workloads as wl
    from paper_2608_02712_amd import vcheck as vc

    atol, rtol = w.tols[w.primary][:2]
    npass = vc.NearPass([(c.cand, c.ref) for c in w.cases], atol, rtol)
    prewarm(npass.launch, prewarm_s)
    for _ in range(warmup):
        npass.launch()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for quad in evs:  # (torch only times events it has seen recorded)
        for e in quad:
            e.record(stream)
    torch.cuda.synchronize()
    for i in range(steps):
        flush.fill_(i & 0xFF)
        evs[i][0].record(stream)
        npass.launch(stream)
        evs[i][1].record(stream)
    for i in range(steps):
        flush.fill_((i + 1) & 0xFF)
        vc.vcheck_profile_events(evs[i][2], evs[i][3])
        npass.launch(stream)
    torch.cuda.synchronize()
    call = sorted(a.elapsed_time(b) for a, b, _, _ in evs)[steps // 2]
    kern = sum(c.elapsed_time(d) for _, _, c, d in evs) / steps
    nbytes = w.ref_cand_bytes
    res = npass.results()
    spent, done = 0.0, 0
    for case in w.cases:
        c, r = wl.raw_numpy(case.cand).reshape(-1), wl.raw_numpy(case.ref).reshape(-1)
        t0 = time.perf_counter()
        oracle.nearpass(c, r, wl.dtype_code(case.ref.dtype), atol, rtol)
        spent += time.perf_counter() - t0
        done += c.nbytes + r.nbytes
        if spent >= 2.0:
            break
    out = {
        "workload": "near-pass statistics of %s at (%g, %g)" % (w.name, atol, rtol),
        "n_cases": len(w.cases),
        "bytes": nbytes,
        "ms_per_call": round(call, 5),
        "gbps": round(nbytes / (call * 1e-3) / 1e9, 2),
        "pct_hbm_peak": round(100.0 * nbytes / (call * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
        "cases_per_s": round(len(w.cases) / (call * 1e-3), 1),
        "stream_kernel_ms": round(kern, 5),
        "stream_kernel_gbps": round(nbytes / (kern * 1e-3) / 1e9, 2),
        "fp16_ceiling_cases": sum(1 for d in res if d["fp16_ceiling"]),
        "oracle_one_thread_gbps": round(done / spent / 1e9, 4),
        "prewarm_s": prewarm_s,
    }
    log("near-pass: %.3f ms/call, %.1f GB/s (%.1f%% of peak), streaming kernel %.3f ms" % (
        call, out["gbps"], out["pct_hbm_peak"], kern))
    return out


def measure_hash(w, steps, warmup, flush, prewarm_s=0.0):
    """Content hashes of every cand and ref tensor of workload w, one call
    (the evidence of a full-coverage evaluation): call time, events around
    the call, cache flushed before it."""
    import torch

    import oracle
    import workloads as wl
    from paper_2608_02712_amd import vcheck as vc

    tensors = [t for c in w.cases for t in (c.cand, c.ref)]
    ch = vc.ContentHash(tensors)
    prewarm(ch.launch, prewarm_s)
    for _ in range(warmup):
        ch.launch()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    for i in range(steps):
        flush.fill_(i & 0xFF)
        evs[i][0].record(stream)
        ch.launch(stream)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    call = sorted(a.elapsed_time(b) for a, b in evs)[steps // 2]
    nbytes = sum(t.numel() * t.element_size() for t in tensors)
    spent, done = 0.0, 0
    for t in tensors:
        raw = wl.raw_numpy(t).reshape(-1)
        t0 = time.perf_counter()
        oracle.content_hash(raw, wl.dtype_code(t.dtype))
        spent += time.perf_counter() - t0
        done += raw.nbytes
        if spent >= 1.0:
            break
    out = {
        "workload": "content hashes of the %d cand and ref tensors of %s" % (len(tensors), w.name),
        "bytes": nbytes,
        "ms_per_call": round(call, 5),
        "gbps": round(nbytes / (call * 1e-3) / 1e9, 2),
        "pct_hbm_peak": round(100.0 * nbytes / (call * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
        "oracle_one_thread_gbps": round(done / spent / 1e9, 4),
        "prewarm_s": prewarm_s,
    }
    log("content hash: %.3f ms/call, %.1f GB/s (%.1f%% of peak)" % (
        call, out["gbps"], out["pct_hbm_peak"]))
    return out


CPU_SHARE = 16  # host threads per GPU on the measurement machines


def host_info():
    """Core counts and CPU model of this host (read before the GPU is
    initialised: lscpu runs as a child process)."""
    import subprocess

    model = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            if line.strip().startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    if model is None:
        try:
            with open("/proc/cpuinfo") as f:
                for line in f:
                    if line.startswith("model name"):
                        model = line.split(":", 1)[1].strip()
                        break
        except OSError:
            pass
    return {"os_cpu_count": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)),
            "model": model}


def cpu_baseline(w, seconds, host):
    """The CPU oracle on whole cases of the workload (with the operator inputs
    when the workload runs the detectors): first one thread until the time
    budget is used (at least one case), then the same cases spread over the
    host's cores (one case per thread at a time; the oracle is plain C
    without shared state, and ctypes releases the interpreter lock while it
    runs). The threads are the affinity cores, at most the host's CPU share
    of one GPU. The multi-threaded rate is the baseline; the single-thread
    figure is reported beside it."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    import workloads as wl

    oracle.default_lib()
    dt = wl.dtype_code(w.cases[0].ref.dtype)
    host_cases, spent = [], 0.0

    def one(item):
        c, r, shape, ins = item
        oracle.validate_case(c, r, dt, shape, w.tols, primary=w.primary, tile=w.tile, k=w.k,
                             inputs=ins)

    for case in w.cases:
        cand, ref = wl.raw_numpy(case.cand).reshape(-1), wl.raw_numpy(case.ref).reshape(-1)
        ins = None
        if w.integrity:
            ins = [(wl.raw_numpy(x).reshape(-1), wl.dtype_code(x.dtype)) for x in case.inputs]
        item = (cand, ref, tuple(case.ref.shape), ins)
        host_cases.append(item)
        t = time.perf_counter()
        one(item)
        spent += time.perf_counter() - t
        if spent >= seconds:
            break
    n_bytes = sum(c.nbytes + r.nbytes for c, r, _, _ in host_cases)
    threads = max(1, min(CPU_SHARE, host["affinity"], len(host_cases)))
    with ThreadPoolExecutor(max_workers=threads) as pool:
        t = time.perf_counter()
        list(pool.map(one, host_cases))
        wall = time.perf_counter() - t
    log("cpu oracle: %d cases, %.2f s on one thread, %.2f s on %d threads" % (
        len(host_cases), spent, wall, threads))
    elems = n_bytes // (2 * w.cases[0].ref.element_size())
    return {"value": round(n_bytes / wall / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "cases_per_s": round(len(host_cases) / wall, 3),
            "single_thread": {"value": round(n_bytes / spent / 1e9, 4), "unit": "GB/s",
                              "cases_per_s": round(len(host_cases) / spent, 3)},
            "host": host,
            "sample": "%d of %d cases (%d elements%s), plain C oracle, whole cases on %d threads "
                      "(the affinity cores, at most %d: the host CPU share of one GPU)"
                      % (len(host_cases), len(w.cases), elems,
                         ", with the operator inputs" if w.integrity else "", threads, CPU_SHARE)}


def traffic_for(name):
    """HBM bytes per launch from the committed rocprofv3 counter readings of
    a workload's streaming kernel, if they were taken on the current sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    ent = data.get(name)
    if not ent or ent.get("kernel_sha") != kernel_hash():
        return None
    return ent.get("hbm_bytes_per_launch")


# ---- rocprofv3 counter output --------------------------------------------------

def short_kernel(name):
    """'main_kernel<1, 1, false>' from a demangled kernel name."""
    n = name.replace("void ", "").replace("vck::(anonymous namespace)::", "")
    n = n.replace("vck::", "")
    depth, out = 0, []
    for ch in n:  # drop the parameter list, keep template arguments
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).strip()


def read_pmc(path):
    """{kernel: {counter: [values per dispatch]}} of every
    *counter_collection.csv under path."""
    import csv
    import glob

    acc = {}
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    for fn in sorted(files):
        with open(fn) as f:
            for row in csv.DictReader(f):
                k = short_kernel(row["Kernel_Name"])
                acc.setdefault(k, {}).setdefault(row["Counter_Name"], []).append(
                    float(row["Counter_Value"]))
    return acc


def median(v):
    v = sorted(v)
    n = len(v)
    return v[n // 2] if n % 2 else 0.5 * (v[n // 2 - 1] + v[n // 2])


def pmc_summary(dirs, match):
    """Median of each counter per dispatch, per kernel whose name contains one
    of `match`, over the given rocprofv3 output directories."""
    for d in dirs:
        acc = read_pmc(d)
        print("== %s" % d)
        for k in sorted(acc):
            if not any(m in k for m in match):
                continue
            cs = acc[k]
            n = max(len(v) for v in cs.values())
            print("  %s (%d dispatches)" % (k, n))
            for c in sorted(cs):
                print("    %-28s %.6g" % (c, median(cs[c])))


def record_traffic(args):
    """Writes the profiles/traffic.json entry of a workload from four
    FETCH_SIZE / WRITE_SIZE runs (the workload, and a plain copy of known
    size that scales the counters)."""
    def one(path, counter, match):
        acc = read_pmc(path)
        vals = [v for k, cs in acc.items() if match in k for v in cs.get(counter, [])]
        if not vals:
            raise SystemExit("no %s readings of a kernel matching %r under %s" % (
                counter, match, path))
        return median(vals), len(vals)

    fk, nf = one(args.fetch, "FETCH_SIZE", args.kernel)
    wk, nw = one(args.write, "WRITE_SIZE", args.kernel)
    cfk, ncf = one(args.copy_fetch, "FETCH_SIZE", args.copy_kernel)
    cwk, ncw = one(args.copy_write, "WRITE_SIZE", args.copy_kernel)
    copy_bytes = 1 << 30
    fs, ws = copy_bytes / (cfk * 1024), copy_bytes / (cwk * 1024)
    hbm = int(round(fk * 1024 * fs + wk * 1024 * ws))
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        data = {}
    data[args.workload] = {
        "kernel": args.kernel_label,
        "kernel_sha": kernel_hash(),
        "fetch_kib_per_dispatch": fk, "fetch_dispatches": nf,
        "write_kib_per_dispatch": wk, "write_dispatches": nw,
        "copy_probe_bytes": copy_bytes, "copy_fetch_kib": cfk, "copy_write_kib": cwk,
        "fetch_scale": round(fs, 6), "write_scale": round(ws, 6),
        "hbm_bytes_per_launch": hbm,
        "algorithmic_bytes_per_launch": args.alg_bytes,
        "traffic_over_algorithmic": round(hbm / args.alg_bytes, 4),
    }
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    print("%s: FETCH_SIZE %.4f KiB (%d dispatches) x 1024 x %.6f + WRITE_SIZE %.4f KiB (%d) x "
          "1024 x %.6f = %d bytes per launch; algorithmic %d; ratio %.4f; copy of %d bytes read "
          "%.4f KiB fetch, %.4f KiB write; sources key %s" % (
              args.workload, fk, nf, fs, wk, nw, ws, hbm, args.alg_bytes, hbm / args.alg_bytes,
              copy_bytes, cfk, cwk, kernel_hash()))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--prewarm-s", type=float, default=0.3,
                    help="untimed calls for this many seconds before each workload other than the "
                         "first measured (and before the probe, near-pass and hash lines); the "
                         "first keeps exactly --warmup untimed calls")
    ap.add_argument("--headline-only", action="store_true",
                    help="only the headline workload (and the CPU baseline)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run 5 device-to-device copies of 1 GiB (a plain copy of known "
                         "size, to scale the HBM byte counters of a profiler run)")
    ap.add_argument("--only", type=int, default=0,
                    help="measure only this workload (1-5) and report it as the headline; "
                         "for profiling single workloads")
    ap.add_argument("--diag", action="store_true",
                    help="with --only: also time the probe, near-pass and hash over it")
    ap.add_argument("--pmc-summary", nargs="+", metavar="DIR",
                    help="print per-kernel counter medians of rocprofv3 --pmc output and exit")
    ap.add_argument("--match", nargs="+", default=["main_kernel", "finalize_kernel",
                                                   "probe_kernel", "nearpass_kernel",
                                                   "hash_kernel", "copyBuffer"])
    ap.add_argument("--record-traffic", action="store_true",
                    help="write a profiles/traffic.json entry from --fetch/--write/--copy-fetch/"
                         "--copy-write rocprofv3 output directories and exit")
    ap.add_argument("--workload")
    ap.add_argument("--kernel", default="main_kernel")
    ap.add_argument("--kernel-label", default="main_kernel")
    ap.add_argument("--copy-kernel", default="copyBuffer")
    ap.add_argument("--alg-bytes", type=int)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary, args.match)
        return
    if args.record_traffic:
        record_traffic(args)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the validation path runs on a single MI355X "
              "(--gpus 1); runs on several GPUs are not measured.", file=sys.stderr)
        sys.exit(2)
    host = None if args.no_cpu else host_info()

    import torch

    torch.cuda.init()
    if args.copy_probe:
        src = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("copy probe: 5 copies of %d bytes" % src.numel())
        return
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    results = {}
    first = args.only or HEADLINE
    w, head = measure(first, args.steps, args.warmup, flush)
    results[first] = head
    cpu = None if args.no_cpu else cpu_baseline(w, args.cpu_seconds, host)
    probe = nearpass = chash = None
    if args.only and args.diag:
        pw = args.prewarm_s
        probe = measure_probe(w, args.steps, args.warmup, flush, pw)
        nearpass = measure_nearpass(w, args.steps, args.warmup, flush, pw)
        chash = measure_hash(w, args.steps, args.warmup, flush, pw)
    del w
    torch.cuda.empty_cache()
    if not args.only and not args.headline_only:
        pw = args.prewarm_s
        wd, r = measure(DIAG_WORKLOAD, args.steps, args.warmup, flush, pw)
        results[DIAG_WORKLOAD] = r
        probe = measure_probe(wd, args.steps, args.warmup, flush, pw)
        nearpass = measure_nearpass(wd, args.steps, args.warmup, flush, pw)
        chash = measure_hash(wd, args.steps, args.warmup, flush, pw)
        del wd
        torch.cuda.empty_cache()
        for cfg in (1, 3, 4):
            wk, r = measure(cfg, args.steps, args.warmup, flush, pw)
            results[cfg] = r
            del wk
            torch.cuda.empty_cache()

    achieved = head["main_kernel_gbps"]
    traffic = traffic_for(head["workload"])
    line = {
        "metric": METRIC,
        "value": head["gbps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_call"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": head["workload"], "storage": head["storage"],
                   "n_cases": head["n_cases"], "tols": head["tols"], "tile": head["tile"],
                   "k": head["k"],
                   "pct_hbm_peak": head["pct_hbm_peak"], "cases_per_s": head["cases_per_s"],
                   "ref_cand_bytes": head["ref_cand_bytes"], "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": "main_kernel (%s, %d tolerance pair%s%s)" % (
                         head["storage"], len(head["tols"]), "" if len(head["tols"]) == 1 else "s",
                         ", detectors" if head.get("integrity") else ""),
                     "alg_bytes_per_launch": head["main_kernel_alg_bytes"],
                     "avg_launch_ms": head["main_kernel_ms"]},
        "cpu_baseline": cpu,
        "workloads": {str(k): v for k, v in sorted(results.items())},
        "probe": probe,
        "nearpass": nearpass,
        "content_hash": chash,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
