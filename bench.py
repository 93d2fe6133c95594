#!/usr/bin/env python3
"""Benchmark of the ChebBooster online stage on one MI355X.

A step is one skipped diffusion step: readiness check and weight row for the
target (host, fp64) plus the prediction of every cached module output (one
launch of the streaming kernel) over the FLUX.1-dev 1024x1024 feature cache
(19 x [1,4096,3072] + 19 x [1,512,3072] + 38 x [1,4608,3072] bf16, six
history entries) held in the interleaved layout (32 KiB chunks of the six
entries taken in turn).  Inputs are seeded synthetic features already
resident in HBM.  The history is filled once before timing through the
full-step push, which is timed on its own and reported beside the step.
The same step over the slot layout, and trivial-body streams with the same
access patterns (the ceilings), are timed in the same run.

Prints one JSON line.  Throughput counts algorithmic bytes: (K+1) entries read
plus one output written, per step.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "achieved HBM GB/s and µs per skipped step, FLUX-1024 cache shape, 1 MI355X"
PEAK_HBM_GBPS = 8000.0
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_23429_amd", "csrc", "kernels.hip")
PROFILES = os.path.join(ROOT, "profiles")
CEILING_LIB = os.path.join(ROOT, "bench_ceiling.so")
LAYOUT = "interleaved"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_sha256():
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they
    were taken on the current kernel source; else None."""
    path = os.path.join(PROFILES, f"traffic_extrapolate_{workload}_{LAYOUT}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not val or sha.group(1) != kernel_sha256():
        return None
    return float(val.group(1))


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="flux_dev_1024")
    ap.add_argument("--block", type=int, default=None)
    ap.add_argument("--unroll", type=int, default=None)
    ap.add_argument("--nontemporal", type=int, default=None)
    ap.add_argument("--blocks-per-cu", type=int, default=None)
    ap.add_argument("--waves-per-cu", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time budget of the oracle baseline")
    ap.add_argument("--no-other-configs", dest="other_configs", action="store_false",
                    help="skip timing the other four workloads (per_config)")
    ap.add_argument("--no-slots", dest="slots", action="store_false",
                    help="time only the interleaved layout (no slot-layout comparison, no "
                         "ceilings): for profiler runs that attribute dispatches by kernel")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain device copy of known size (counter calibration)")
    return ap.parse_args(argv)


def copy_probe(torch):
    nbytes = 2 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(10):
        dst.copy_(src)
    e.record()
    e.synchronize()
    ms = s.elapsed_time(e) / 10
    print(json.dumps({"copy_probe_bytes_read": nbytes, "copy_probe_bytes_written": nbytes,
                      "ms": ms, "gbps": 2 * nbytes / ms / 1e6}), flush=True)


def setup_workload(torch, cheb, cfg, layout, entries=None):
    """Seeded history on the device (generated unless given), pushed through
    the ring of a cache in `layout`."""
    from synth import make_history, split_segments
    dt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[cfg.dtype]
    if entries is None:
        t0 = time.time()
        entries = make_history(cfg, "cuda")
        torch.cuda.synchronize()
        log(f"[bench] {cfg.name}: generated {cfg.n_hist} x {cfg.numel} elements "
            f"in {time.time() - t0:.1f} s")
    cache = cheb.ChebCache(cfg.n_hist, dt, cfg.seg_numel, layout=layout)
    stream = torch.cuda.current_stream()
    handle = int(stream.cuda_stream)
    # Segment addresses are gathered before the timed region, so the events
    # bracket the C call (its argument checks and launches) only.
    ptrs = [[v.data_ptr() for v in split_segments(e, cfg)] for e in entries]
    push_ms = []
    for rep in range(2):          # second pass: warm, and the ring keeps the same entries
        for x, p in zip(cfg.nodes, ptrs):
            s, f = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            s.record(stream)
            cheb.cheb_cache_push(cache.handle, x, p, handle)
            f.record(stream)
            f.synchronize()
            if rep == 1:
                push_ms.append(s.elapsed_time(f))
    return entries, cache, push_ms


def time_steps(torch, cache, targets, out, steps, warmup):
    """Whole-region and per-launch HIP-event timing of `steps` skipped steps
    on torch's current stream (the stream the kernel is launched on)."""
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        cache.extrapolate_at(targets[i % len(targets)], out, stream=stream)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for i in range(steps):
        cache.extrapolate_at(targets[i % len(targets)], out, stream=stream)
    end.record(stream)
    end.synchronize()
    region_ms = start.elapsed_time(end) / steps
    # per-launch durations, same stream, events right around each launch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for i, (a, b) in enumerate(evs):
        a.record(stream)
        cache.extrapolate_at(targets[i % len(targets)], out, stream=stream)
        b.record(stream)
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) for a, b in evs)
    return region_ms, per


def time_multi(torch, cfg, cache, steps, warmup):
    """All skipped steps between two full steps (the workload's targets) from
    one pass over the history: cheb_extrapolate_at_multi."""
    stream = torch.cuda.current_stream()
    outs = [cache.new_output() for _ in cfg.targets]
    for _ in range(warmup):
        cache.extrapolate_at_multi(cfg.targets, outs, stream=stream)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        cache.extrapolate_at_multi(cfg.targets, outs, stream=stream)
    end.record(stream)
    end.synchronize()
    ms = start.elapsed_time(end) / steps
    M = len(cfg.targets)
    B = (cfg.n_hist + M) * cfg.numel * cfg.elem_size
    del outs
    return {"targets_per_pass": M, "us_per_pass": ms * 1e3, "us_per_skipped_step": ms * 1e3 / M,
            "bytes_per_pass": B, "gbps": B / (ms * 1e6),
            "note": "the workload's skipped steps between two full steps predicted in one "
                    "pass over the history (cheb_extrapolate_at_multi); not in value"}


def time_residual(torch, cheb, cfg, entries, cache, steps, warmup):
    """Skipped step's residual update x_out = x_in + (every predicted module
    output added into the residual stream): the full form over the whole
    history (cheb_residual_apply), and the collapsed history (push-time
    reduction per full step, cheb_residual_reduce, then the prediction from
    residual-sized entries; the entry either reduced from the module outputs
    or taken as the difference of the residual stream across the block
    stack)."""
    from synth import split_segments
    res_off, res_n = cfg.residual_map()
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    w = cheb.cheb_precompute_weights(cache.history(), [cfg.targets[0]])[0]
    x_in = torch.randn(res_n, device="cuda")
    x_out = torch.empty_like(x_in)

    def timed(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        b.synchronize()
        return a.elapsed_time(b) / n * 1e3

    S = cfg.numel * cfg.elem_size
    R = res_n * 4
    us_full = timed(lambda: cache.residual_apply(w, res_off, x_out, x_in, stream=stream), steps)
    hist = cheb.ResidualHistory(cfg.n_hist, res_off, res_n)
    segs = [split_segments(e, cfg) for e in entries]
    for x, sg in zip(cfg.nodes, segs):
        hist.push(x, sg, stream=stream)
    k = [0]

    def push_one():
        hist.push(cfg.nodes[k[0] % cfg.n_hist] + 1e-3 * (1 + k[0]), segs[k[0] % cfg.n_hist],
                  stream=stream)
        k[0] += 1
    us_reduce = timed(push_one, max(5, steps // 5))
    x_after = torch.randn(res_n, device="cuda")

    def push_diff():
        hist.push_difference(cfg.nodes[k[0] % cfg.n_hist] + 1e-3 * (1 + k[0]), x_after, x_in,
                             stream=stream)
        k[0] += 1
    us_diff = timed(push_diff, max(5, steps // 5))
    for x, sg in zip(cfg.nodes, segs):
        hist.push(x, sg, stream=stream)
    wc = cheb.cheb_precompute_weights(hist.history(), [float(hist.history()[-1]) - 0.02])[0]
    us_pred = timed(lambda: hist.cache.residual_apply(wc, [0], x_out, x_in, stream=stream), steps)
    hist.close()
    return {
        "full_form": {"us": us_full, "bytes": cfg.n_hist * S + 2 * R,
                      "gbps": (cfg.n_hist * S + 2 * R) / (us_full * 1e3)},
        "collapsed_push_reduce": {"us": us_reduce, "bytes": S + R, "gbps": (S + R) / (us_reduce * 1e3)},
        "collapsed_push_difference": {"us": us_diff, "bytes": 3 * R,
                                      "gbps": 3 * R / (us_diff * 1e3),
                                      "note": "entry as x_after - x_before of the full step's "
                                              "residual stream"},
        "collapsed_predict": {"us": us_pred, "bytes": (cfg.n_hist + 2) * R,
                              "gbps": (cfg.n_hist + 2) * R / (us_pred * 1e3)},
        "residual_elements": res_n,
        "note": "skipped-step residual update (block stack with every module output "
                "predicted); full form reads the whole history, collapsed form keeps one "
                "residual-sized fp32 entry per full step; not in value",
    }


def time_online_run(torch, cheb, cfg, entries, reps=3):
    """The online stage over one whole sampling run of T = 50 steps from the
    offline table (Section 3.3 schedule with s0 = s1 = 1, r = 6, history of
    the workload's size; steps before the history fills run in full): every
    full step pushes its features, every run of skipped steps is predicted
    in one pass (per-module form); and the same run with the collapsed
    residual history (entry from the residual difference per full step, one
    residual prediction per skipped step)."""
    import numpy as np
    from synth import split_segments
    T, s0, s1, r, n = 50, 1, 1, 6, cfg.n_hist
    x = 1.0 - np.arange(T) / 50.0 if cfg.time_scale == 1.0 else 999.0 - 20.0 * np.arange(T)
    table = cheb.ChebTable(T, s0, s1, r, n, x, cheb.CHEB_SHORT_FULL)
    predicted = [table.step(s)[0] for s in range(T)]
    runs = dict(table.runs())
    dt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[cfg.dtype]
    cache = cheb.ChebCache(n, dt, cfg.seg_numel, layout=LAYOUT)
    outs = [cache.new_output() for _ in range(max(runs.values()))]
    segs = [split_segments(e, cfg) for e in entries]
    res_off, res_n = cfg.residual_map()
    hist = cheb.ResidualHistory(n, res_off, res_n)
    x_before = torch.randn(res_n, device="cuda")
    x_after = torch.randn(res_n, device="cuda")
    x_out = torch.empty_like(x_before)

    def per_module():
        cache.reset()
        s, k = 0, 0
        while s < T:
            if not predicted[s]:
                cache.push(float(x[s]), segs[k % len(segs)])
                k += 1
                s += 1
            else:
                c = runs[s]
                cache.extrapolate_steps(table, s, c, outs[:c])
                s += c

    def collapsed():
        hist.cache.reset()
        for s in range(T):
            if not predicted[s]:
                hist.push_difference(float(x[s]), x_after, x_before)
            else:
                hist.predict(float(x[s]), x_out, x_before)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ms = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            ms.append(a.elapsed_time(b))
        return sorted(ms)[len(ms) // 2]

    n_full = T - sum(predicted)
    res = {
        "table": f"T={T} s0={s0} s1={s1} r={r} n={n}, short history run in full",
        "full_steps": n_full, "predicted_steps": T - n_full,
        "per_module_ms": timed(per_module),
        "collapsed_residual_ms": timed(collapsed),
        "single_target_predictions_ms": None,
        "note": "device time of the online stage for one image (pushes and predictions; "
                "the DiT forward of the full steps is not included); "
                "single_target_predictions_ms is the predicted steps alone at one launch "
                "each, for comparison; not in value",
    }
    cache.close()
    hist.close()
    table.close()
    del outs
    torch.cuda.empty_cache()
    return res


def oracle_parity_sample(torch, cfg, entries, cache, out, target, count=1 << 16):
    """Part of the CPU-baseline leg: the same oracle, untimed, recomputes a
    sample of the device's prediction at `target` from the stored history."""
    import numpy as np
    import oracle
    idx = np.unique(np.random.default_rng(cfg.seed).integers(0, cfg.numel, count))
    it = torch.from_numpy(idx).to("cuda")
    cache.extrapolate_at(target, out)
    torch.cuda.synchronize()
    w = oracle.weights_row(cfg.nodes, target)
    if cfg.dtype == "bf16":
        hosts = [e.index_select(0, it).view(torch.int16).cpu().numpy().view(np.uint16)
                 for e in entries]
        exp, mag = oracle.extrapolate_bf16(hosts, w)
        got = oracle.bf16_to_f64(out.index_select(0, it).view(torch.int16).cpu().numpy()
                                 .view(np.uint16))
    else:
        hosts = [e.index_select(0, it).cpu().numpy() for e in entries]
        exp, mag = oracle.extrapolate_f32(hosts, w)
        got = out.index_select(0, it).cpu().numpy().astype(np.float64)
    err = oracle.parity_error(got, exp, mag)
    return {"samples": int(idx.size), "floored_rel_err": err[0], "normwise_err": err[2],
            "bound": 1e-2 if cfg.dtype == "bf16" else 1e-5}


def _time_oracle(run, hosts, rows, seconds):
    passes, spent = 0, 0.0
    while spent < seconds or passes == 0:
        t0 = time.perf_counter()
        run(hosts, rows[passes % len(rows)], want_absmag=False)
        spent += time.perf_counter() - t0
        passes += 1
    return passes, spent


def cpu_baseline(torch, cfg, entries, targets, seconds, max_host_bytes=16 << 30):
    """The oracle, as it stands, timed on the host: whole skipped steps of the
    workload (every element, targets cycled) repeated until about a third of
    `seconds` of CPU time have been spent, three times on every core the
    process may use (the median is the value); then a quarter of `seconds` on
    one core over the first sixteenth of every entry.  Falls back to a leading
    slice of every entry when the history would not fit `max_host_bytes` of
    host memory."""
    import numpy as np
    import oracle
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    threads = oracle.set_threads(min(cores, int(os.environ.get("OMP_NUM_THREADS", cores))))
    n = min(cfg.numel, max(1, max_host_bytes // (cfg.n_hist * cfg.elem_size)))
    if cfg.dtype == "bf16":
        hosts = [e[:n].view(torch.int16).cpu().numpy().view(np.uint16) for e in entries]
        run = oracle.extrapolate_bf16
    else:
        hosts = [e[:n].cpu().numpy() for e in entries]
        run = oracle.extrapolate_f32
    rows = [oracle.weights_row(cfg.nodes, t) for t in targets]
    step_bytes = (cfg.n_hist + 1) * cfg.elem_size
    runs = []
    for _ in range(3):
        passes, spent = _time_oracle(run, hosts, rows, seconds / 3.0)
        runs.append((passes * step_bytes * n / spent / 1e9, passes, spent))
    runs_sorted = sorted(runs)
    value, passes, spent = runs_sorted[1]
    oracle.set_threads(1)
    n1 = max(1, n // 16)
    p1, s1 = _time_oracle(run, [h[:n1] for h in hosts], rows, seconds / 4.0)
    oracle.set_threads(threads)
    what = "every element" if n == cfg.numel else f"the first {n} elements"
    return {"value": value, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "seconds": sum(r[2] for r in runs) + s1,
            "runs_gbps": [r[0] for r in runs],
            "us_per_step": spent / passes * 1e6 * cfg.numel / n,
            "one_core": {"value": p1 * step_bytes * n1 / s1 / 1e9, "unit": "GB/s",
                         "elements": n1, "steps": p1, "seconds": s1},
            "sample": f"three runs of {passes} skipped steps each of the {cfg.name} workload "
                      f"({what} of each of the {cfg.n_hist} history entries, targets "
                      f"cycled; median run), then one core on the first {n1} elements; "
                      f"fp64 oracle; value counts the same algorithmic bytes per element as "
                      f"the GPU step"}


def time_graph(torch, pairs, targets, steps):
    """Per-step time of `steps` predictions captured once in a HIP graph and
    replayed (for steps short enough that host launch cost shows).  Step i
    predicts into pairs[i % len(pairs)] = (cache, output)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            for i in range(steps):
                cache, out = pairs[i % len(pairs)]
                cache.extrapolate_at(targets[i % len(targets)], out)
    torch.cuda.current_stream().wait_stream(side)
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        g.replay()
    b.record()
    b.synchronize()
    del g
    return a.elapsed_time(b) / (5 * steps) * 1e3


def time_rotated(torch, cheb, cfg, entries, sets=32, steps=64):
    """Graph-replayed steps that cycle over `sets` copies of the history, each
    with its own output, so that the working set (sets x (K+2) entries) is
    larger than the 256 MB last-level cache and every step streams from HBM."""
    from synth import split_segments
    dt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[cfg.dtype]
    pairs = []
    for _ in range(sets):
        c = cheb.ChebCache(cfg.n_hist, dt, cfg.seg_numel, layout=LAYOUT)
        for x, e in zip(cfg.nodes, entries):
            c.push(x, split_segments(e, cfg))
        pairs.append((c, c.new_output()))
    torch.cuda.synchronize()
    us = time_graph(torch, pairs, cfg.targets, steps)
    for c, _ in pairs:
        c.close()
    del pairs
    return us, sets * (cfg.n_hist + 1) * cfg.numel * cfg.elem_size


def measure_config(torch, cheb, cfg, steps, warmup, layout=LAYOUT, entries=None):
    entries, cache, push_ms = setup_workload(torch, cheb, cfg, layout, entries)
    out = cache.new_output()
    res = measure_cache(torch, cheb, cfg, cache, out, push_ms, entries, steps, warmup, layout)
    return res, entries, cache, out


def measure_cache(torch, cheb, cfg, cache, out, push_ms, entries, steps, warmup, layout):
    region_ms, per = time_steps(torch, cache, cfg.targets, out, steps, warmup)
    avg_launch_ms = sum(per) / len(per)
    B = cfg.bytes_per_step
    res = {
        "workload": cfg.name, "layout": layout, "elements": cfg.numel, "history": cfg.n_hist,
        "dtype": cfg.dtype,
        "bytes_per_step": B, "us_per_step": region_ms * 1e3,
        "gbps": B / (region_ms * 1e6), "frac_of_8tbps": B / (region_ms * 1e6) / PEAK_HBM_GBPS,
        "launch_us_median": per[len(per) // 2] * 1e3, "launch_us_p10": per[len(per) // 10] * 1e3,
        "launch_us_p90": per[(9 * len(per)) // 10] * 1e3, "launch_us_avg": avg_launch_ms * 1e3,
        "push_us_median": sorted(push_ms)[len(push_ms) // 2] * 1e3,
        "push_gbps": 2 * cfg.numel * cfg.elem_size / (sorted(push_ms)[len(push_ms) // 2] * 1e6),
    }
    if region_ms < 0.05 and layout == LAYOUT:   # launch-bound: also replay from a HIP graph
        g_us = time_graph(torch, [(cache, out)], cfg.targets, 64)
        res["graph_us_per_step"] = g_us
        res["graph_gbps"] = B / (g_us * 1e3)
        r_us, r_bytes = time_rotated(torch, cheb, cfg, entries)
        res["hbm_rotated"] = {"us_per_step": r_us, "gbps": B / (r_us * 1e3),
                              "working_set_bytes": r_bytes,
                              "note": "graph-replayed steps cycling over 32 history copies "
                                      "(working set above the 256 MB last-level cache)"}
    return res


def device_summary(torch):
    """Name, compute units and LDS per compute unit of device 0 (the LDS is
    what the occupancy cap of the prediction divides)."""
    import ctypes
    lib = ctypes.CDLL(CEILING_LIB)
    lib.ceiling_lds_per_cu.restype = ctypes.c_int
    lds = lib.ceiling_lds_per_cu()
    p = torch.cuda.get_device_properties(0)
    return {"name": p.name, "gcn_arch": getattr(p, "gcnArchName", None),
            "compute_units": p.multi_processor_count,
            "lds_per_cu_bytes": lds if lds >= 0 else None,
            "lds_reserved_per_64_lane_block_at_7_waves": lds // 7 // 512 * 512
            if lds > 0 else None}


def stream_ceilings(torch, slots_cache, il_cache, out, reps=10, warmup=2):
    """Trivial-body streams (bench_ceiling.hip) over the benchmark's own
    buffers, one entry-sized stream each, timed per launch with HIP events on
    the current stream: six entries read, a copy, a write, and six entries
    read with one stream written from the slot layout and from the
    interleaved layout; and the interleaved 6:1 stream with its stores
    folded into a 64 MiB window (held by the last-level cache: the stores
    leave each XCD but not the chip) or a 1 MiB window (held by the XCDs'
    L2: the stores stay in the XCD).  GB/s counts the bytes each kernel
    would move with every store reaching HBM, so the windows read as the
    rate the reads allow when the stores cost less.  Every case runs in both
    launch shapes of the prediction: 1024-lane blocks at full occupancy, and
    64-lane blocks capped at 8 waves per compute unit (suffix _w8); the
    6:1 streams also at 7 waves (_w7), the cap the prediction takes for six
    entries and one output."""
    import ctypes
    lib = ctypes.CDLL(CEILING_LIB)
    lib.ceiling_stream.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_void_p), ctypes.c_int,
                                   ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                   ctypes.c_int, ctypes.c_void_p]
    lib.ceiling_stream.restype = ctypes.c_int
    import paper_2608_23429_amd as cheb
    stream = torch.cuda.current_stream()
    handle = int(stream.cuda_stream)
    n = slots_cache.n_slots
    S = slots_cache.slot_numel * torch.empty((), dtype=slots_cache.dtype).element_size()
    n_vec = S // 16
    slots = [slots_cache.arena.data_ptr() + k * slots_cache.slot_stride_bytes for k in range(n)]
    # the interleaved region starts at its lowest lane
    region = min(cheb.cheb_cache_entry(il_cache.handle, a) for a in range(n))
    # (name, kind, sources, bytes counted, store window in vectors)
    cases = [
        ("read_only_6", 0, slots, n * S, 0),
        ("read_only_6_interleaved", 4, [region], n * S, 0),
        ("copy", 1, slots[:1], 2 * S, 0),
        ("write_only", 3, [], S, 0),
        ("mix_6_1_slots", 1, slots, (n + 1) * S, 0),
        ("mix_6_1_interleaved", 2, [region], (n + 1) * S, 0),
        ("mix_6_1_interleaved_stores_in_64MiB", 5, [region], (n + 1) * S, (64 << 20) // 16),
        ("mix_6_1_interleaved_stores_in_1MiB", 5, [region], (n + 1) * S, (1 << 20) // 16),
    ]
    shaped = []
    for name, kind, src, nbytes, window in cases:
        shaped.append((name, kind, src, nbytes, window, 0))
        if name.startswith("mix_6_1") and window == 0:
            shaped.append((name + "_w7", kind, src, nbytes, window, 7))
        shaped.append((name + "_w8", kind, src, nbytes, window, 8))
    res = {}
    for name, kind, src, nbytes, window, waves in shaped:
        arr = (ctypes.c_void_p * max(1, len(src)))(*src) if src else None
        n_src = n if kind in (2, 4, 5) else max(1, len(src))
        def launch():
            rc = lib.ceiling_stream(kind, arr, n_src, out.data_ptr(), n_vec, window, waves,
                                    handle)
            if rc != 0:
                raise RuntimeError(f"ceiling_stream({name}) returned {rc}")
        for _ in range(warmup):
            launch()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for a, b in evs:
            a.record(stream)
            launch()
            b.record(stream)
        torch.cuda.synchronize()
        ms = sorted(a.elapsed_time(b) for a, b in evs)
        res[name] = {"bytes": nbytes, "us_median": ms[len(ms) // 2] * 1e3, "us_best": ms[0] * 1e3,
                     "gbps_median": nbytes / (ms[len(ms) // 2] * 1e6),
                     "gbps_best": nbytes / (ms[0] * 1e6)}
        log(f"[bench] ceiling {name}: {res[name]['gbps_median']:.0f} GB/s median")
    return res


def main(argv=None):
    args = parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the skipped-step prediction needs no "
              "communication, and this benchmark runs on a single MI355X. Run with --gpus 1.",
              file=sys.stderr, flush=True)
        return 2
    import torch
    import paper_2608_23429_amd as cheb
    from synth import by_name

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    if args.copy_probe:
        copy_probe(torch)
        return 0

    shape = cheb.cheb_get_launch_config()
    for k, v in (("block", args.block), ("unroll", args.unroll), ("nontemporal", args.nontemporal),
                 ("blocks_per_cu", args.blocks_per_cu), ("waves_per_cu", args.waves_per_cu)):
        if v is not None:
            shape[k] = v
    cheb.cheb_set_launch_config(**shape)

    cfg = by_name(args.config)
    log(f"[bench] workload {cfg.name}, launch shape {shape}, "
        f"{args.warmup} warmup + {args.steps} timed steps")
    # Both layouts' caches are filled first; an untimed settle phase then runs
    # the step on both for about a tenth of a second so that the first timed
    # layout does not pay for the GPU's ramp from idle.  Then each layout:
    # W warmup steps and K timed steps.
    entries, cache, push_ms = setup_workload(torch, cheb, cfg, LAYOUT)
    out = cache.new_output()
    if args.slots:
        _, cache_sl, push_sl = setup_workload(torch, cheb, cfg, "slots", entries)
        out_sl = cache_sl.new_output()
    for _ in range(25):
        cache.extrapolate_at(cfg.targets[0], out)
        if args.slots:
            cache_sl.extrapolate_at(cfg.targets[0], out_sl)
    torch.cuda.synchronize()
    res = measure_cache(torch, cheb, cfg, cache, out, push_ms, entries, args.steps, args.warmup,
                        LAYOUT)
    log(f"[bench] {cfg.name} ({LAYOUT}): {res['us_per_step']:.1f} us/step, {res['gbps']:.0f} GB/s")
    res_sl, ceilings = None, None
    if args.slots:
        res_sl = measure_cache(torch, cheb, cfg, cache_sl, out_sl, push_sl, entries, args.steps,
                               args.warmup, "slots")
        log(f"[bench] {cfg.name} (slots): {res_sl['us_per_step']:.1f} us/step, "
            f"{res_sl['gbps']:.0f} GB/s")
        ceilings = stream_ceilings(torch, cache_sl, cache, out_sl)
        cache_sl.close()
        del cache_sl, out_sl
        torch.cuda.empty_cache()
    multi = time_multi(torch, cfg, cache, max(10, args.steps // 2), args.warmup)
    log(f"[bench] {cfg.name} multi-target: {multi['us_per_skipped_step']:.1f} us per skipped "
        f"step ({multi['gbps']:.0f} GB/s over {multi['targets_per_pass']} targets)")
    resid = time_residual(torch, cheb, cfg, entries, cache, max(10, args.steps // 2), args.warmup)
    online = time_online_run(torch, cheb, cfg, entries)
    online["single_target_predictions_ms"] = online["predicted_steps"] * res["us_per_step"] / 1e3
    log(f"[bench] {cfg.name} one sampling run ({online['full_steps']} full, "
        f"{online['predicted_steps']} predicted steps): per-module {online['per_module_ms']:.2f} ms, "
        f"collapsed residual {online['collapsed_residual_ms']:.2f} ms")
    log(f"[bench] {cfg.name} residual: full form {resid['full_form']['us']:.1f} us, collapsed "
        f"predict {resid['collapsed_predict']['us']:.1f} us + push-time reduce "
        f"{resid['collapsed_push_reduce']['us']:.1f} us (or residual difference "
        f"{resid['collapsed_push_difference']['us']:.1f} us) per full step")
    achieved = res["bytes_per_step"] / (res["launch_us_avg"] * 1e3)
    traffic = measured_traffic(cfg.name)
    # the ceiling is the faster of the trivial 6:1 interleaved stream's
    # launch shapes
    own = max(ceilings[k]["gbps_median"] for k in ceilings
              if k.startswith("mix_6_1_interleaved") and "stores_in" not in k) if ceilings else None
    line = {
        "metric": METRIC,
        "value": res["gbps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["us_per_step"] / 1e3,
        "us_per_step": res["us_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic: seeded per-element random polynomial in the time variable plus "
                "Gaussian noise, stored in the cache dtype",
        "config": {"workload": cfg.name, "elements_per_entry": cfg.numel,
                   "history_entries": cfg.n_hist, "segments": len(cfg.segments),
                   "bytes_per_step": res["bytes_per_step"], "launch": shape,
                   "layout": LAYOUT, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": achieved / PEAK_HBM_GBPS, "traffic": traffic,
                     "layout": LAYOUT,
                     "ceiling": ceilings,
                     "frac_of_ceiling": achieved / own if own else None,
                     "ceiling_note": "trivial-body streams (XOR, the prediction's access "
                                     "pattern, in its launch shapes) over entry-sized streams of "
                                     "this workload, timed in this run; frac_of_ceiling is "
                                     "against the fastest shape of the 6-read:1-write stream "
                                     "over the same interleaved layout"},
        "layouts": {
            LAYOUT: {"us_per_step": res["us_per_step"], "gbps": res["gbps"],
                     "launch_us_avg": res["launch_us_avg"], "push_us_median": res["push_us_median"]},
            "slots": None if res_sl is None else {
                "us_per_step": res_sl["us_per_step"], "gbps": res_sl["gbps"],
                "launch_us_avg": res_sl["launch_us_avg"], "push_us_median": res_sl["push_us_median"],
                "note": "contiguous entries (the layout a fused push writes into)"}},
        "launch_us": {"median": res["launch_us_median"], "p10": res["launch_us_p10"],
                      "p90": res["launch_us_p90"], "avg": res["launch_us_avg"]},
        "push": {"us_median": res["push_us_median"], "gbps": res["push_gbps"],
                 "note": "full-step copy into the ring, once per full step (not in value)"},
        "device": device_summary(torch),
        "multi_target": multi,
        "residual": resid,
        "online_run": online,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] oracle CPU baseline (~{args.cpu_seconds:.0f} s)")
        line["cpu_baseline"] = cpu_baseline(torch, cfg, entries, cfg.targets, args.cpu_seconds)
        log(f"[bench] oracle: {line['cpu_baseline']['value']:.2f} GB/s on "
            f"{line['cpu_baseline']['cores']} threads")
        par = oracle_parity_sample(torch, cfg, entries, cache, out, cfg.targets[-1])
        line["cpu_baseline"]["parity_sample"] = par
        log(f"[bench] oracle parity sample: floored error {par['floored_rel_err']:.3e}")
    cache.close()
    del entries, cache, out
    torch.cuda.empty_cache()
    if args.other_configs:
        from dataclasses import replace
        from synth import CONFIGS
        per = []
        f16 = replace(by_name("pixart_sigma_1024"), name="pixart_sigma_1024_f16", dtype="f16")
        for c in CONFIGS + [f16]:
            if c.name == cfg.name:
                continue
            steps = max(10, args.steps // 2)
            # as for the headline: both caches filled, a short untimed settle
            # on both, then each layout timed
            e, ch, pm = setup_workload(torch, cheb, c, LAYOUT)
            o = ch.new_output()
            if args.slots:
                _, chs, pms = setup_workload(torch, cheb, c, "slots", e)
                os_ = chs.new_output()
            for _ in range(10):
                ch.extrapolate_at(c.targets[0], o)
                if args.slots:
                    chs.extrapolate_at(c.targets[0], os_)
            torch.cuda.synchronize()
            r = measure_cache(torch, cheb, c, ch, o, pm, e, steps, args.warmup, LAYOUT)
            log(f"[bench] {c.name}: {r['us_per_step']:.1f} us/step, {r['gbps']:.0f} GB/s")
            ch.close()
            del ch, o
            if args.slots:
                rs = measure_cache(torch, cheb, c, chs, os_, pms, e, steps, args.warmup, "slots")
                log(f"[bench] {c.name} (slots): {rs['us_per_step']:.1f} us/step, "
                    f"{rs['gbps']:.0f} GB/s")
                r["slots"] = {"us_per_step": rs["us_per_step"], "gbps": rs["gbps"],
                              "launch_us_avg": rs["launch_us_avg"]}
                chs.close()
                del chs, os_
            per.append(r)
            del e
            torch.cuda.empty_cache()
        line["per_config"] = per
        shares = []
        for g in (2, 4, 8):
            c = cfg.scaled_blocks(g, 1 << 30)
            r, e, ch, o = measure_config(torch, cheb, c, max(10, args.steps // 2), args.warmup)
            log(f"[bench] {cfg.name} 1/{g} token share: {r['us_per_step']:.1f} us/step, "
                f"{r['gbps']:.0f} GB/s")
            shares.append({"share": f"1/{g}", "elements": r["elements"],
                           "bytes_per_step": r["bytes_per_step"], "us_per_step": r["us_per_step"],
                           "gbps": r["gbps"], "launch_us_median": r["launch_us_median"]})
            ch.close()
            del e, ch, o
            torch.cuda.empty_cache()
        line["token_shares"] = {
            "workload": cfg.name, "shares": shares,
            "note": "one GPU's part of the cache when the model is split G ways along the token "
                    "axis (every cached tensor's token dimension divided by G); not in value"}
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
