#!/usr/bin/env python3
"""Throughput of the validation hot path on one MI355X.

One step = one vcheck_sweep call over a whole synthetic workload (tolerance
gate, NaN/Inf counts, exact max abs/rel, error sums, tile map, first-k,
detectors and suite match rate: every stage of the path), inputs resident in
HBM. The Infinity Cache is flushed (512 MiB write) before every step, outside
the timed interval; each step is timed with HIP events on the launch stream.
The streaming kernels are timed in a second pass with events the library
records around them.

Headline line: the fp16 batch of 64 cases of 2048x2048 (the configuration the
metric is quoted on). ``probe`` reports the tensor-statistics probe over the
128 cand and ref tensors of that batch in one call, ``nearpass`` the near-pass
statistics of its 64 cases, ``content_hash`` the content hashes of its 128
tensors. ``workloads`` holds the same figures for all five
workloads, measured in the same run. ``roofline`` reports the main streaming
kernel's achieved HBM bandwidth (algorithmic bytes / its event-timed average
duration) against the 8 TB/s peak; ``cpu_baseline`` times the CPU oracle on a
bounded sample of the headline workload on this host.

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--headline-only]
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
HEADLINE = 2
KERNEL_SRC = os.path.join(ROOT, "paper_2608_02712_amd", "csrc", "vcheck_kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def kernel_hash(text=None):
    """Hash of the kernel source with // comments and blank lines removed, so
    that the stored counter readings stay valid across comment-only edits."""
    if text is None:
        with open(KERNEL_SRC) as f:
            text = f.read()
    code = []
    for line in text.splitlines():
        line = line.split("//", 1)[0].rstrip()
        if line:
            code.append(line)
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


def time_sweep(sw, steps, warmup, flush):
    """`steps` pairs of calls, the Infinity Cache flushed before every call:
    the first call of a pair is timed whole (events around the call only),
    the second has the streaming kernels timed alone (events the library
    records just before and after them; recording them adds a gap between
    the kernels, so they are not used for the call time)."""
    import torch
    from paper_2608_02712_amd import vcheck as vc

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


def measure(cfg, steps, warmup, flush):
    import torch

    import workloads as wl
    from paper_2608_02712_amd import vcheck as vc

    t = time.perf_counter()
    w = wl.WORKLOADS[cfg]("cuda")
    torch.cuda.synchronize()
    log("workload %d (%s) generated in %.1f s" % (cfg, w.name, time.perf_counter() - t))
    sw = vc.Sweep([(c.cand, c.ref, c.inputs) for c in w.cases], w.tols, primary=w.primary,
                  tile=w.tile, k=w.k or 0, integrity=w.integrity)
    call_ms, main_ms, wall = time_sweep(sw, steps, warmup, flush)
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
    }
    log("workload %d: %.3f ms/call, %.1f GB/s (%.1f%% of peak), main kernel %.3f ms" % (
        cfg, ms, out["gbps"], out["pct_hbm_peak"], main_avg))
    return w, out


def measure_probe(w, steps, warmup, flush):
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
    }
    log("probe: %.3f ms/call, %.1f GB/s (%.1f%% of peak), streaming kernel %.3f ms" % (
        call, out["gbps"], out["pct_hbm_peak"], kern))
    return out


def measure_nearpass(w, steps, warmup, flush):
    """Near-pass statistics over every case of workload w at its primary
    tolerance pair, one call: call time (events around the call, cache
    flushed before it) and the streaming kernel's time."""
    import torch

    import oracle
    import workloads as wl
    from paper_2608_02712_amd import vcheck as vc

    atol, rtol = w.tols[w.primary][:2]
    npass = vc.NearPass([(c.cand, c.ref) for c in w.cases], atol, rtol)
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
    }
    log("near-pass: %.3f ms/call, %.1f GB/s (%.1f%% of peak), streaming kernel %.3f ms" % (
        call, out["gbps"], out["pct_hbm_peak"], kern))
    return out


def measure_hash(w, steps, warmup, flush):
    """Content hashes of every cand and ref tensor of workload w, one call
    (the evidence of a full-coverage evaluation): call time, events around
    the call, cache flushed before it."""
    import torch

    import oracle
    import workloads as wl
    from paper_2608_02712_amd import vcheck as vc

    tensors = [t for c in w.cases for t in (c.cand, c.ref)]
    ch = vc.ContentHash(tensors)
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
    }
    log("content hash: %.3f ms/call, %.1f GB/s (%.1f%% of peak)" % (
        call, out["gbps"], out["pct_hbm_peak"]))
    return out


def cpu_baseline(w, seconds):
    """The CPU oracle on whole cases of the workload: first one thread until
    the time budget is used (at least one case), then the same cases spread
    over the host's cores (one case per thread at a time; the oracle is plain
    C without shared state, and ctypes releases the interpreter lock while it
    runs). The multi-threaded rate is the baseline; the single-thread figure
    is reported beside it."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    import workloads as wl

    oracle.default_lib()
    dt = wl.dtype_code(w.cases[0].ref.dtype)
    host, spent = [], 0.0
    for case in w.cases:
        cand, ref = wl.raw_numpy(case.cand).reshape(-1), wl.raw_numpy(case.ref).reshape(-1)
        host.append((cand, ref, tuple(case.ref.shape)))
        t = time.perf_counter()
        oracle.validate_case(cand, ref, dt, tuple(case.ref.shape), w.tols, primary=w.primary,
                             tile=w.tile, k=w.k)
        spent += time.perf_counter() - t
        if spent >= seconds:
            break
    n_bytes = sum(c.nbytes + r.nbytes for c, r, _ in host)
    threads = max(1, min(16, len(os.sched_getaffinity(0)), len(host)))

    def one(item):
        c, r, shape = item
        oracle.validate_case(c, r, dt, shape, w.tols, primary=w.primary, tile=w.tile, k=w.k)

    with ThreadPoolExecutor(max_workers=threads) as pool:
        t = time.perf_counter()
        list(pool.map(one, host))
        wall = time.perf_counter() - t
    log("cpu oracle: %d cases, %.2f s on one thread, %.2f s on %d threads" % (
        len(host), spent, wall, threads))
    elems = n_bytes // (2 * w.cases[0].ref.element_size())
    return {"value": round(n_bytes / wall / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "cases_per_s": round(len(host) / wall, 3),
            "single_thread": {"value": round(n_bytes / spent / 1e9, 4), "unit": "GB/s",
                              "cases_per_s": round(len(host) / spent, 3)},
            "sample": "%d of %d cases (%d elements), plain C oracle, whole cases on %d threads"
                      % (len(host), len(w.cases), elems, threads)}


def traffic_for(name, launches_bytes):
    """HBM bytes per launch from the committed rocprofv3 counter runs, if they
    were taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    ent = data.get(name)
    if not ent or ent.get("kernel_sha") != kernel_hash():
        return None
    return ent.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--headline-only", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run 5 device-to-device copies of 1 GiB (a plain copy of known "
                         "size, to scale the HBM byte counters of a profiler run)")
    ap.add_argument("--only", type=int, default=0,
                    help="measure only this workload (1-5) and report it as the headline; "
                         "for profiling single workloads")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the validation path runs on a single MI355X "
              "(--gpus 1); runs on several GPUs are not measured.", file=sys.stderr)
        sys.exit(2)

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
    cpu = None if args.no_cpu else cpu_baseline(w, args.cpu_seconds)
    probe = nearpass = chash = None
    if not args.only:
        probe = measure_probe(w, args.steps, args.warmup, flush)
        nearpass = measure_nearpass(w, args.steps, args.warmup, flush)
        chash = measure_hash(w, args.steps, args.warmup, flush)
    del w
    torch.cuda.empty_cache()
    if not args.headline_only and not args.only:
        for cfg in (1, 3, 4, 5):
            wk, r = measure(cfg, args.steps, args.warmup, flush)
            results[cfg] = r
            del wk
            torch.cuda.empty_cache()

    achieved = head["main_kernel_gbps"]
    traffic = traffic_for(head["workload"], head["main_kernel_alg_bytes"])
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
                     "kernel": "main_kernel (%s, %d tolerance pair%s)" % (
                         head["storage"], len(head["tols"]), "" if len(head["tols"]) == 1 else "s"),
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
