#!/usr/bin/env python3
"""Fragments/s routed + aggregated on one MI355X, with the dominant kernel's
achieved HBM bandwidth against the 8 TB/s peak.

Workload (default): skewed Zipf(1.2) depth-6 tree of 2^26 fragments, keys packed
before timing, 128-d float32 payload per fragment, route by the level-4 prefix to
256 destinations, mean-pool at level 4, completion mask at level 2. One step =
one alto_aggregate call over the whole batch (routing outputs perm, dest_offsets,
dest, plus groups, means and mask). Inputs are resident in HBM before timing.

Prints one JSON line. --gpus N > 1 is refused: this build runs on one GPU.

--workload picks another of the synthetic workloads (one JSON line each, "all" for
every one): tiny (64-query depth-4 tree, token concat), factool (1,024-query
FacTool-shaped batch, 768-d mean per document then document-id concat per claim),
tokens (256-generator token stream in 4,096-fragment steps), factool_stream
(10,000 steps of 4,096 fragments, both stages per step, per-step latency), join
(pcombine of level-4 group objects with the Zipf tree's fragments), split
(split_text of 16,384 generator token streams into sentences at a pmap entry),
route_load (sticky least-loaded routing of flows, against hash routing).
"""
import argparse
import gc
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
PHASES = ["prep", "sort", "segment", "groups", "gather", "mean_kernel", "total"]
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "k_mean_zipf64M_traffic.json")
MEAN_SRC = os.path.join(ROOT, "paper_2403_04311_amd", "csrc", "aggregate.hip")
MEAN_KERNEL = "k_mean<4, 1, BatchSrc>"


def mean_kernel_source_sha():
    """sha256 of the mean-gather kernel's source text (its template through the
    closing brace): the traffic measured by hardware counters is reported only
    while this text is unchanged."""
    import hashlib
    src = open(MEAN_SRC).read()
    a = src.index("template <int VEC, int CPL, typename Src>\n__global__ __launch_bounds__(256) void k_mean(")
    b = src.index("\n}\n", a)
    return hashlib.sha256(src[a:b].encode()).hexdigest()


def derive_traffic(fetch_csv, write_csv, command):
    """HBM bytes per launch of every kernel from two rocprofv3 --pmc runs of
    `bench.py --steps 1 --warmup 1 --copy-calibration-mib M` (FETCH_SIZE, then
    WRITE_SIZE, KiB per dispatch), each scaled by what the same counter reads for
    the calibration copy of known size. Writes the summary next to the profiles."""
    import csv
    import collections
    per = {}
    calib = {}
    for name, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == name]
        cal = [r for r in rows if "copyBuffer" in r["Kernel_Name"]]
        big = max(cal, key=lambda r: int(r["Grid_Size"]))
        calib[name] = float(big["Counter_Value"]) * 1024.0
        acc = collections.defaultdict(list)
        for r in rows:
            k = r["Kernel_Name"].replace("(anonymous namespace)::", "").split("(")[0]
            k = k[5:] if k.startswith("void ") else k
            acc[k].append(float(r["Counter_Value"]) * 1024.0)
        per[name] = acc
    return calib, per


def write_traffic_summary(fetch_csv, write_csv, copy_mib, command):
    calib, per = derive_traffic(fetch_csv, write_csv, command)
    known = copy_mib * 1024.0 * 1024.0
    fs, ws = known / calib["FETCH_SIZE"], known / calib["WRITE_SIZE"]
    kernels = {}
    for k in sorted(set(per["FETCH_SIZE"]) | set(per["WRITE_SIZE"])):
        f = per["FETCH_SIZE"].get(k, [])
        w = per["WRITE_SIZE"].get(k, [])
        if not f or not w:
            continue
        fb, wb = max(f) * fs, max(w) * ws   # the largest dispatch of each kernel (the full-size launch)
        kernels[k] = {"fetch_bytes": fb, "write_bytes": wb, "dispatches": len(f)}
    mk = kernels[MEAN_KERNEL]
    out = {"kernel": MEAN_KERNEL, "source_sha256": mean_kernel_source_sha(),
           "traffic_bytes_per_launch": mk["fetch_bytes"] + mk["write_bytes"],
           "fetch_bytes_per_launch": mk["fetch_bytes"], "write_bytes_per_launch": mk["write_bytes"],
           "calibration": {"copy_bytes": known, "FETCH_SIZE_scale": fs, "WRITE_SIZE_scale": ws},
           "command": command, "kernels": kernels}
    with open(TRAFFIC_SUMMARY, "w") as fh:
        json.dump(out, fh, indent=1)
    return out


def measured_traffic():
    """Traffic of the mean kernel per launch from the committed counter summary,
    or None when there is none or the kernel's source changed since."""
    try:
        t = json.load(open(TRAFFIC_SUMMARY))
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != mean_kernel_source_sha():
        return None
    return t["traffic_bytes_per_launch"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(leaves_log2: int):
    """The oracle, as it stands, on a smaller draw of the same generator."""
    import numpy as np
    from oracle import alto_oracle as O
    from paper_2403_04311_amd import workloads as W
    w = W.zipf_tree("cpu", leaves=1 << leaves_log2)
    path, fan, x = w.path.numpy(), w.fan.numpy(), w.payload_f32.numpy()
    # one core: the process is pinned to one CPU for the timed run (numpy's own
    # threads, if any, then share it), and the affinity is restored afterwards
    pinned = None
    try:
        before = os.sched_getaffinity(0)
        cpu = min(before)
        os.sched_setaffinity(0, {cpu})
        pinned = (before, cpu)
    except (AttributeError, OSError):
        pass
    try:
        t0 = time.perf_counter()
        keys = O.pack_keys(path, w.bits)
        O.aggregate(keys, fan, w.bits, w.agg_level, w.op, w.dim, w.mask_level, w.route_level, w.num_dest,
                    None, x)
        dt = time.perf_counter() - t0
    finally:
        if pinned:
            os.sched_setaffinity(0, pinned[0])
    return {"value": (1 << leaves_log2) / dt, "unit": "fragments/s", "cores": 1, "kind": "oracle",
            "sample": f"same generator at 2^{leaves_log2} leaves (1/{1 << (26 - leaves_log2)} of the "
                      f"workload): pack + route + aggregate, {dt:.1f} s of numpy on one pinned CPU"
                      + (f" (cpu {pinned[1]})" if pinned else " (affinity not settable: unpinned)"),
            "host": host_info()}


def host_info():
    """CPU model, hardware threads and RAM of the machine the oracle ran on."""
    info = {"cpu_model": None, "threads": os.cpu_count(), "ram_gib": None}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["cpu_model"] = line.split(":", 1)[1].strip()
                    break
        with open("/proc/meminfo") as f:
            for line in f:
                if line.startswith("MemTotal"):
                    info["ram_gib"] = round(int(line.split()[1]) / (1 << 20), 1)
                    break
    except OSError:
        pass
    return info


def read_ceiling_gbps(dev, gib: int = 16, reps: int = 5):
    """Attainable streaming read on this GPU: alto_read_probe (16-byte non-temporal
    loads, XOR-reduced) over a resident array, bytes read per rep over the time."""
    import ctypes as C
    import torch
    from paper_2403_04311_amd import alto
    lib = alto.load()
    lib.alto_read_probe.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
    x = torch.ones(gib << 30, dtype=torch.uint8, device=dev)
    out = torch.zeros(16384, dtype=torch.int64, device=dev)
    st = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert lib.alto_read_probe(C.c_void_p(x.data_ptr()), x.numel(), C.c_void_p(out.data_ptr()), st) == 0
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        lib.alto_read_probe(C.c_void_p(x.data_ptr()), x.numel(), C.c_void_p(out.data_ptr()), st)
    e1.record()
    torch.cuda.synchronize()
    gbps = x.numel() * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del x
    torch.cuda.empty_cache()
    return gbps


def _timed(fn, steps, warmup):
    """Runs fn warmup + steps times; returns ms per call of the timed calls
    (HIP events on the current stream around all of them)."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def _line(workload, n, ms, steps, warmup, path_bytes, extra=None):
    res = {
        "metric": "fragments/sec routed+aggregated at 1 MI355X; achieved HBM GB/s vs peak",
        "value": n / (ms * 1e-3), "unit": "fragments/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic", "config": {"workload": workload, "fragments": n},
        "path_roofline": {"algorithmic_bytes_per_step": path_bytes, "achieved": path_bytes / (ms * 1e-3) / 1e9,
                          "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                          "frac": path_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS},
    }
    if extra:
        res.update(extra)
    return res


def bench_tiny(args):
    """64-query depth-4 tree: one alto_aggregate (route by query to 8 destinations,
    token concat per sentence); launch-latency bound."""
    import torch
    from paper_2403_04311_amd import alto, workloads as W
    w = W.tiny_tree("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    n = w.n
    ws = alto.new_workspace(alto.workspace_bytes(w.bits, n, w.num_dest, w.agg_level, "concat"))
    perm = torch.empty(n, dtype=torch.int32, device="cuda")
    offs = torch.empty(w.num_dest + 1, dtype=torch.int64, device="cuda")
    dest = torch.empty(n, dtype=torch.int32, device="cuda")
    out = alto.new_groups(n, w.agg_level, "concat", cap_tokens=n)
    status = alto.new_status()

    def step():
        alto.aggregate(keys, w.fan, w.bits, w.agg_level, "concat", 1, 0, w.route_level, w.num_dest,
                       w.payload_i32, None, ws=ws, perm=perm, dest_offsets=offs, dest=dest, out=out,
                       status=status, n=n)
    ms = _timed(step, args.steps * 20, args.warmup)
    assert int(status.item()) == 0
    E = int(out.counts[0])
    nl = w.depth - 1 - w.agg_level + 1
    path_bytes = n * (8 + 4 * nl + 4 + 4 + 4 + 4) + E * (8 + 4 + 8 + 4 * (w.agg_level - 1) + 8)
    return _line("64-query depth-4 tree (query/doc/sentence/token), token concat per sentence, 8 destinations "
                 "by query, one batch", n, ms, args.steps * 20, args.warmup, path_bytes,
                 {"groups": E, "us_per_call": ms * 1e3})


def bench_factool(args):
    """FacTool-shaped batch, both stages per step: 768-d mean per document (route by
    claim to 32 destinations), then concat of the documents' corpus ids per claim
    over the first stage's records."""
    import torch
    from paper_2403_04311_amd import alto, workloads as W
    w = W.factool_batch("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    n, dim = w.n, w.dim
    sb = W.FACTOOL_CLAIM_STAGE
    ws = alto.new_workspace(alto.workspace_bytes(w.bits, n, 32, 4, "mean", dim))
    perm = torch.empty(n, dtype=torch.int32, device="cuda")
    offs = torch.empty(33, dtype=torch.int64, device="cuda")
    dest = torch.empty(n, dtype=torch.int32, device="cuda")
    gA = alto.new_groups(n // 4 + 1024, 4, "mean", dim)
    stA, stB = alto.new_status(), alto.new_status()
    alto.aggregate(keys, w.fan, w.bits, 4, "mean", dim, 0, 2, 32, w.payload_i32, w.payload_f32, ws=ws,
                   perm=perm, dest_offsets=offs, dest=dest, out=gA, status=stA, n=n)
    torch.cuda.synchronize()
    E = int(gA.counts[0])
    assert int(stA.item()) == 0 and E > 0
    wsB = alto.new_workspace(alto.workspace_bytes(sb["bits"], E, 32, 2, "concat"))
    permB = torch.empty(E, dtype=torch.int32, device="cuda")
    destB = torch.empty(E, dtype=torch.int32, device="cuda")
    gB = alto.new_groups(E, 2, "concat", cap_tokens=E)
    fanB = gA.fan_up.view(3, -1)[:, :E]
    prof = {}

    offsB = torch.empty(33, dtype=torch.int64, device="cuda")

    def step():
        alto.aggregate(keys, w.fan, w.bits, 4, "mean", dim, 0, 2, 32, w.payload_i32, w.payload_f32, ws=ws,
                       perm=perm, dest_offsets=offs, dest=dest, out=gA, status=stA, n=n)
        alto.aggregate(gA.key, fanB, sb["bits"], 2, "concat", 1, 0, 2, 32, gA.first_i32, None, ws=wsB,
                       perm=permB, dest_offsets=offsB, dest=destB, out=gB, status=stB, n=E)

    # stage B of a step on a second HIP stream beside stage A of the next: stage A's
    # records in one of two buffers, an event each way
    side = torch.cuda.Stream()
    gAs = [gA, alto.new_groups(n // 4 + 1024, 4, "mean", dim)]
    fanBs = [g.fan_up.view(3, -1)[:, :E] for g in gAs]
    a_done = [torch.cuda.Event(), torch.cuda.Event()]
    b_done = [torch.cuda.Event(), torch.cuda.Event()]
    used = [False, False]
    cnt = [0]

    def step_pipe():
        k = cnt[0] & 1
        cnt[0] += 1
        main = torch.cuda.current_stream()
        if used[k]:
            main.wait_event(b_done[k])
        g = gAs[k]
        alto.aggregate(keys, w.fan, w.bits, 4, "mean", dim, 0, 2, 32, w.payload_i32, w.payload_f32, ws=ws,
                       perm=perm, dest_offsets=offs, dest=dest, out=g, status=stA, n=n, stream=main)
        a_done[k].record(main)
        side.wait_event(a_done[k])
        with torch.cuda.stream(side):
            alto.aggregate(g.key, fanBs[k], sb["bits"], 2, "concat", 1, 0, 2, 32, g.first_i32, None, ws=wsB,
                           perm=permB, dest_offsets=offsB, dest=destB, out=gB, status=stB, n=E, stream=side)
        b_done[k].record(side)
        used[k] = True
    lib = alto.load()
    import ctypes as C
    lib.alto_profile_begin.argtypes = [C.c_int32]
    lib.alto_profile_end.argtypes = [C.POINTER(C.c_float), C.POINTER(C.c_int32), C.c_int32]
    pipe = not args.no_stage_overlap
    run = step_pipe if pipe else step
    for _ in range(args.warmup):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    lib.alto_profile_phases.argtypes = [C.c_uint32]
    assert lib.alto_profile_phases(1 << PHASES.index("mean_kernel")) == 0
    assert lib.alto_profile_begin(4 * args.steps + 4) == 0
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    side.wait_stream(torch.cuda.current_stream())
    for _ in range(args.steps):
        run()
    torch.cuda.current_stream().wait_stream(side)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    msp = (C.c_float * len(PHASES))()
    calls = (C.c_int32 * len(PHASES))()
    assert lib.alto_profile_end(msp, calls, len(PHASES)) == 0
    assert lib.alto_profile_phases(0xFFFFFFFF) == 0
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    seq_ms = _timed(step, args.steps, 0) if pipe else ms   # both stages one after the other on one stream
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    C2 = int(gB.counts[0])
    # mean gather of stage A: one launch per step (stage B has no mean)
    mean_ms = msp[PHASES.index("mean_kernel")] / max(calls[PHASES.index("mean_kernel")], 1)
    kern_bytes = (n + E) * dim * 4
    path_bytes = (n * (8 + 4 + 4 + 4 * dim + 4 + 4) + E * (8 + 4 + 8 + 4 + 12 + 4 * dim)
                  + E * (8 + 8 + 4 + 4 + 4 + 4) + C2 * (8 + 4 + 8 + 4 + 8))
    return _line("FacTool-shaped batch: 1,024 queries, depth 5, 768-d mean per document (route by claim to 32 "
                 "destinations), then document-id concat per claim"
                 + (" (the claim stage of a batch on a second HIP stream beside the document stage of the next)"
                    if pipe else ""), n, ms, args.steps, args.warmup, path_bytes,
                 {"documents": E, "claims": C2, "sequential_ms_per_step": seq_ms,
                  "roofline": {"bound": "hbm", "kernel": "k_mean (first stage)", "achieved":
                               kern_bytes / (mean_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                               "frac": kern_bytes / (mean_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                               "algorithmic_bytes_per_launch": kern_bytes, "avg_launch_ms": mean_ms}})


class _CollectorPaused:
    """Python's garbage collector paused over a timed stream loop, the objects alive
    at its start frozen out of later collections: a collection that scans the tens
    of thousands of tensor views and events of a long stream stalls the host for
    milliseconds, and a host that enqueues the steps then lets the GPU run dry (the
    FacTool stream measured 119 us per step with the collector paused, 149-223 us
    with it running after other work in the same process). Collects first, outside
    the timed region; restores the collector's state afterwards."""

    def __enter__(self):
        self.was = gc.isenabled()
        gc.collect()
        gc.freeze()
        gc.disable()
        return self

    def __exit__(self, *exc):
        gc.unfreeze()
        if self.was:
            gc.enable()
        return False


def _stream_run(steps, step_of, after=None):
    """Runs every step of a stream (stage callables per step); returns total ms
    (events around all steps) and per-step device ms (events per step). after(s),
    if given, runs after step s's closing event (bookkeeping outside the steps)."""
    import torch
    e0 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    e1 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    with _CollectorPaused():
        for s in range(steps):
            e0[s].record()
            step_of(s)
            e1[s].record()
            if after:
                after(s)
        torch.cuda.synchronize()
    per = [e0[s].elapsed_time(e1[s]) for s in range(steps)]
    return e0[0].elapsed_time(e1[steps - 1]), per


class _LightEvents:
    """Timing events recorded without the system-scope fence that a default event's
    completion carries (hipEventDisableSystemFence: no cache write-back and
    invalidation at the marker), for per-step stamps inside a pipeline of short
    steps, where a default event pair costs the stream it is recorded on a few
    microseconds. Created, recorded and read through the HIP runtime that torch
    loaded; released by close()."""

    FLAG = 0x20000000   # hipEventDisableSystemFence (timing stays enabled)

    def __init__(self, count):
        import ctypes as C
        self.C = C
        self.hip = C.CDLL("libamdhip64.so")
        self.ev = [C.c_void_p() for _ in range(count)]
        for e in self.ev:
            if self.hip.hipEventCreateWithFlags(C.byref(e), C.c_uint(self.FLAG)) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, i, stream):
        if self.hip.hipEventRecord(self.ev[i], self.C.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, i, j):
        ms = self.C.c_float()
        if self.hip.hipEventElapsedTime(self.C.byref(ms), self.ev[i], self.ev[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def close(self):
        for e in self.ev:
            self.hip.hipEventDestroy(e)
        self.ev = []


def _pct(xs, q):
    import numpy as np
    return float(np.percentile(np.asarray(xs), q))


def bench_tokens(args):
    """Token stream: 256 generators, round-robin arrival, 4,096-fragment steps,
    sentences carried across steps and emitted when their last token arrives."""
    import torch
    from paper_2403_04311_amd import alto, workloads as W
    w = W.token_stream("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    n, step = w.n, w.step
    nsteps = (n + step - 1) // step
    out = alto.new_groups(step, 2, "concat", cap_tokens=(1 << 16) + step)
    status = alto.new_status()

    def run():
        s = alto.Stream(w.bits, 2, 64, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 16, step_max=step,
                        release=args.release)

        def one(i):
            a, b = i * step, min(n, (i + 1) * step)
            s.step(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b], None, out=out, status=status)
        tot, per = _stream_run(nsteps, one)
        s.close()
        return tot, per
    def run_overlapped(ends=True, starts=True):
        # each step's routing on a second HIP stream, beside the previous step's merge
        # and emission (alto_stream_step_overlap). ends: an event at every step's end
        # (on the merge stream), starts: one at every step's start (on the routing
        # stream); each event itself costs a few microseconds on its stream, so the
        # period is taken with ends only, the latency with both, the rate with neither
        s = alto.Stream(w.bits, 2, 64, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 16, step_max=step,
                        release=args.release)
        main = torch.cuda.current_stream()
        route = route_stream
        route.wait_stream(main)
        ev = _LightEvents(2 * nsteps)   # t0[i] = i, t1[i] = nsteps + i
        one = s.prepare(out, status, stream=main, route_stream=route)   # fixed arguments checked once
        with _CollectorPaused():
            h0 = time.perf_counter()
            for i in range(nsteps):
                if (ends and starts) or i == 0:
                    ev.record(i, route)
                one(*step_views[i])
                if ends or i == nsteps - 1:
                    ev.record(nsteps + i, main)
            host_us[0] = (time.perf_counter() - h0) * 1e6 / nsteps
            main.wait_stream(route)
            torch.cuda.synchronize()
        s.close()
        lat = [ev.elapsed_ms(i, nsteps + i) for i in range(nsteps)] if (ends and starts) else []
        period = [ev.elapsed_ms(nsteps + i - 1, nsteps + i) for i in range(1, nsteps)] if ends else []
        tot = ev.elapsed_ms(0, 2 * nsteps - 1)
        ev.close()
        return tot, lat, period
    route_stream = torch.cuda.Stream()
    host_us = [0.0]   # the host's time to enqueue a step (the last run)
    # each step's inputs as views of the stream's arrays, made once (no copies)
    step_views = [(keys[i * step:min(n, (i + 1) * step)], w.fan[:, i * step:min(n, (i + 1) * step)],
                   w.payload_i32[i * step:min(n, (i + 1) * step)]) for i in range(nsteps)]
    # the stream is short (96 steps, a few ms): many runs, so that the GPU clock
    # settles first and the percentiles pool enough steps
    reps, warm = 10, max(args.warmup, 20)
    for _ in range(warm):
        run()
    seq_per = []
    seq_tot = 0.0
    for _ in range(reps):
        t, p = run()
        seq_tot += t / reps
        seq_per += p
    assert int(status.item()) == 0
    for _ in range(warm):
        run_overlapped()
    tot, lat, period = 0.0, [], []
    for _ in range(reps):
        t, _, p = run_overlapped(starts=False)
        tot += t / reps
        period += p
        lat += run_overlapped()[1]
    bare_runs = sorted(run_overlapped(ends=False, starts=False)[0] / nsteps for _ in range(reps))
    host_bare = host_us[0]
    assert int(status.item()) == 0
    ms = tot / nsteps
    path_bytes = (n * (8 + 4 + 4 + 4 + 4 + 4) + 16384 * (8 + 4 + 8 + 4 + 8)) / nsteps
    return _line(f"token stream: 256 generators x 64 sentences, geometric(1/24) tokens, round-robin, "
                 f"{step}-fragment steps, concat per sentence, 64 destinations, release {args.release}; "
                 f"each step's routing on a second HIP stream beside the previous step's merge",
                 n / nsteps, ms, nsteps, 1,
                 path_bytes, {"stream_fragments": n, "stream_ms": tot,
                              "step_ms_p50": _pct(period, 50), "step_ms_p99": _pct(period, 99),
                              "step_ms_max": max(period),
                              "step_ms_note": "p50/p99/max of the period between consecutive steps' ends, "
                                              f"{reps} runs of {nsteps} steps pooled, an event at each step's end; "
                                              "latency from runs with an event at each step's start as well",
                              "uninstrumented_ms_per_step": _pct(bare_runs, 50),
                              "uninstrumented_ms_per_step_min_max": [bare_runs[0], bare_runs[-1]],
                              "host_enqueue_us_per_step": host_bare,
                              "step_latency_ms_p50": _pct(lat, 50), "step_latency_ms_p99": _pct(lat, 99),
                              "sequential_ms_per_step": seq_tot / nsteps, "sequential_step_ms_p50": _pct(seq_per, 50),
                              "sequential_step_ms_p99": _pct(seq_per, 99)})


def bench_factool_stream(args):
    """FacTool-shaped windowed stream, 10,000 steps of 4,096 fragments; per step the
    document stage (768-d mean) and the claim stage over its emitted records, which
    reads the first stage's emitted count on the device (no host read per step)."""
    import torch
    from paper_2403_04311_amd import alto, workloads as W
    w = W.factool_stream("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    step, steps = w.step, min(w.info["steps"], args.stream_steps)
    ring, ring_rows = w.payload_f32, w.payload_f32.shape[0]
    sbB = W.FACTOOL_CLAIM_STAGE
    gA = alto.new_groups(step, 4, "mean", 768)
    gB = alto.new_groups(step, 2, "concat", cap_tokens=(1 << 16) + step)
    stA, stB = alto.new_status(), alto.new_status()
    fanA = gA.fan_up.view(3, -1)
    emitted = torch.zeros(1, dtype=torch.int64, device="cuda")

    def run(nsteps):
        sA = alto.Stream(w.bits, 2, 32, 4, "mean", 768, max_live_leaves=1 << 17, max_groups=1 << 22,
                         step_max=step, release=args.release)
        sB = alto.Stream(sbB["bits"], 2, 32, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 20,
                         step_max=step, release=args.release)
        emitted.zero_()

        def one(s):
            a, b = s * step, (s + 1) * step
            r0 = (s * step) % ring_rows
            sA.step(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b], ring[r0:r0 + step], out=gA, status=stA)
            sB.step(gA.key, fanA, gA.first_i32, None, out=gB, status=stB, n=step, n_dev=gA.counts[0:1])

        def count(s):
            emitted.add_(gA.counts[0:1])   # documents emitted, for the byte count
        tot, per = _stream_run(nsteps, one, count)
        sA.close()
        sB.close()
        return tot, per
    def run_pipelined(nsteps, count=False):
        # stage B of step s on a second HIP stream, beside stage A of step s + 1:
        # stage A writes its records into one of two buffers, stage B waits for them
        # (an event), stage A waits before reusing a buffer until stage B has read it.
        # count: also add up the emitted documents (a torch kernel per step on the
        # second stream, and its launch on the host: bookkeeping, so not in timed runs)
        sA = alto.Stream(w.bits, 2, 32, 4, "mean", 768, max_live_leaves=1 << 17, max_groups=1 << 22,
                         step_max=step, release=args.release)
        sB = alto.Stream(sbB["bits"], 2, 32, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 20,
                         step_max=step, release=args.release)
        emitted.zero_()
        main = torch.cuda.current_stream()
        side, rA, rB = side_stream, route_a, route_b
        a_done = [torch.cuda.Event() for _ in range(2)]
        b_done = [torch.cuda.Event() for _ in range(2)]
        ev = _LightEvents(2 * nsteps)   # step s: start s, end nsteps + s
        for x in (side, rA, rB):
            x.wait_stream(main)
        # the per-step calls with their fixed arguments checked once (Stream.prepare)
        stepA = [sA.prepare(gAs[k], stA, stream=main, route_stream=rA if route_sa else None) for k in range(2)]
        stepB = sB.prepare(gB, stB, stream=side, route_stream=rB if route_sb else None)
        nA = [g.counts[0:1] for g in gAs]
        with _CollectorPaused():
            h0 = time.perf_counter()
            for s in range(nsteps):
                k = s & 1
                ev.record(s, rA if route_sa else main)
                if s >= 2:
                    main.wait_event(b_done[k])
                # stage A: routing on rA (beside the previous step), the rest on main
                stepA[k](*views_a[s])
                a_done[k].record(main)
                # stage B over stage A's records: routing on rB, the rest on side (which
                # reads them only after the routing's signal when the routing is on rB)
                rB.wait_event(a_done[k])
                if not route_sb:
                    side.wait_event(a_done[k])
                stepB(gAs[k].key, fanAs[k], gAs[k].first_i32, None, n=step, n_dev=nA[k])
                if count:
                    with torch.cuda.stream(side):
                        emitted.add_(nA[k])
                b_done[k].record(side)
                ev.record(nsteps + s, side)
            host_us[0] = (time.perf_counter() - h0) * 1e6 / nsteps
            for x in (side, rA, rB):
                main.wait_stream(x)
            torch.cuda.synchronize()
        sA.close()
        sB.close()
        lat = [ev.elapsed_ms(s, nsteps + s) for s in range(nsteps)]
        period = [ev.elapsed_ms(nsteps + s - 1, nsteps + s) for s in range(1, nsteps)]
        tot = ev.elapsed_ms(0, 2 * nsteps - 1)
        ev.close()
        return tot, lat, period
    side_stream, route_a, route_b = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    host_us = [0.0]   # the host's time to enqueue a step (the last run)
    # each step's inputs as views of the stream's arrays, made once (no copies)
    views_a = [(keys[s * step:(s + 1) * step], w.fan[:, s * step:(s + 1) * step],
                w.payload_i32[s * step:(s + 1) * step], ring[(s * step) % ring_rows:(s * step) % ring_rows + step])
               for s in range(steps)]
    route_sa = args.stream_overlap in ("a", "ab")
    route_sb = args.stream_overlap in ("b", "ab")
    gAs = [gA, alto.new_groups(step, 4, "mean", 768)]
    fanAs = [g.fan_up.view(3, -1) for g in gAs]
    run(max(args.warmup, 1) * 50)
    seq_total, seq_dev = run(steps)
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    E_seq = int(emitted.item())
    run_pipelined(max(args.warmup, 1) * 50)
    total, lat, period = run_pipelined(steps)
    host_timed = host_us[0]
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    run_pipelined(steps, count=True)   # untimed: the same documents as on one stream
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    E = int(emitted.item())
    assert E == E_seq
    n = steps * step
    # inputs read once (key, 3 count columns, doc id, 768-d row), perm/dest, emitted document
    # records and their means; the carried partial state is not counted
    path_bytes = (n * (8 + 12 + 4 + 3072 + 8) + E * (8 + 4 + 8 + 4 + 12 + 3072)) / steps
    ms = total / steps
    return _line(f"FacTool-shaped windowed stream: {steps} steps x {step} fragments, 768-d mean per document "
                 f"then document-id concat per claim (both stages each step, the claim stage reading the "
                 f"document stage's emitted count on the device; the claim stage of a step on a second HIP "
                 f"stream beside the document stage of the next"
                 + {"ab": ", each stage's routing on a stream of its own", "a": ", the document stage's routing on "
                    "a stream of its own", "b": ", the claim stage's routing on a stream of its own",
                    "none": ""}[args.stream_overlap] + "), "
                 f"release {args.release}",
                 step, ms, steps, 50, path_bytes,
                 {"stream_fragments": n, "documents_emitted": E, "window_fragments": w.info["window"],
                  "long_lived_fraction": w.info["calibrated_frac"],
                  "step_ms_p50": _pct(period, 50), "step_ms_p99": _pct(period, 99), "step_ms_max": max(period),
                  "step_ms_note": "p50/p99/max of the period between consecutive steps' ends (two stages in flight)",
                  "step_latency_ms_p50": _pct(lat, 50), "step_latency_ms_p99": _pct(lat, 99),
                  "host_enqueue_us_per_step": host_timed,
                  "sequential_ms_per_step": seq_total / steps, "sequential_step_ms_p50": _pct(seq_dev, 50),
                  "sequential_step_ms_p99": _pct(seq_dev, 99)})


def bench_join(args):
    """pcombine by ancestry: left objects of one level joined with every fragment below
    them. Timed: the 2^26-fragment Zipf tree (1,452 level-4 group objects); also
    reported: the FacTool-shaped tree (search-query objects with their sentences)."""
    import ctypes
    import torch
    from paper_2403_04311_amd import alto, workloads as W

    def one(keys, bits, level, steps, warmup):
        shift = sum(bits[level:])
        left = torch.unique(keys >> shift)
        g = torch.Generator(device="cuda")
        g.manual_seed(11)
        left = left[torch.randperm(left.numel(), generator=g, device="cuda")].contiguous()
        nl, nr = left.numel(), keys.numel()
        L = alto.layout(bits)
        ws = alto.new_workspace(alto.load().alto_join_workspace_bytes(ctypes.byref(L), nl))
        match = torch.empty(nr, dtype=torch.int32, device="cuda")
        hits = torch.empty(nl, dtype=torch.int32, device="cuda")
        counts = torch.zeros(2, dtype=torch.int64, device="cuda")
        st = alto.new_status()
        ms = _timed(lambda: alto.join(left, keys, bits, level, match=match, hits=hits, counts=counts, status=st,
                                      ws=ws), steps, warmup)
        assert int(st.item()) == 0 and int(counts[0]) == nr
        return nl, nr, ms

    w2 = W.factool_batch("cuda")
    k2, _ = alto.pack_keys(w2.path, w2.bits)
    nl2, nr2, ms2 = one(k2, w2.bits, 3, args.steps * 10, args.warmup)
    del w2, k2
    w5 = W.zipf_tree("cuda", leaves=1 << args.leaves_log2)
    k5, _ = alto.pack_keys(w5.path, w5.bits)
    del w5
    torch.cuda.empty_cache()
    nl5, nr5, ms5 = one(k5, (3, 12, 12, 12, 12, 12), 4, args.steps, args.warmup)
    path_bytes = nr5 * (8 + 4) + nl5 * (8 + 4)
    return _line(f"pcombine join: {nl5} level-4 group objects with all 2^{args.leaves_log2} fragments of the Zipf "
                 f"depth-6 tree", nr5, ms5, args.steps, args.warmup, path_bytes,
                 {"left_objects": nl5,
                  "factool": {"left_objects": nl2, "right_fragments": nr2, "ms": ms2,
                              "fragments_per_s": nr2 / (ms2 * 1e-3),
                              "hbm_frac": (nr2 * 12 + nl2 * 12) / (ms2 * 1e-3) / 1e9 / HBM_PEAK_GBPS}})


def bench_split(args):
    """split_text at a pmap entry: generator token streams cut at sentence delimiters
    into (request, sentence, token) keys with their declared counts. Timed: 16,384
    generator streams (64x the token-stream workload, 26.2M positions); also
    reported: the 256 streams of the token-stream workload itself (408,190)."""
    import torch
    from paper_2403_04311_amd import alto, workloads as W

    def one(t, steps, warmup):
        keys, st = alto.pack_keys(t.path, t.bits)
        n = t.n
        L = alto.layout(t.bits)
        import ctypes
        ws = alto.new_workspace(alto.load().alto_split_workspace_bytes(ctypes.byref(L), n))
        ok = torch.empty(n, dtype=torch.int64, device="cuda")
        of = torch.empty((len(t.bits), n), dtype=torch.int32, device="cuda")
        otok = torch.empty(n, dtype=torch.int32, device="cuda")
        oidx = torch.empty(n, dtype=torch.int32, device="cuda")
        rest = torch.empty(n, dtype=torch.int32, device="cuda")
        counts = torch.zeros(4, dtype=torch.int64, device="cuda")
        ms = _timed(lambda: alto.split(keys, t.fan, t.tokens, t.bits, t.delim, t.seg_bits, t.tok_bits, out_keys=ok,
                                       out_fan=of, out_tokens=otok, out_idx=oidx, rest_idx=rest, counts=counts,
                                       status=st, ws=ws), steps, warmup)
        assert int(st.item()) == 0 and int(counts[2]) == 0
        return n, ms

    t3 = W.token_stream_text("cuda")
    n3, ms3 = one(t3, args.steps * 10, args.warmup)
    del t3
    t = W.token_stream_text("cuda", generators=16384)
    n, ms = one(t, args.steps, args.warmup)
    # in: key, stream length, token; out per placed token: key, two counts, token, input index
    per = 8 + 4 + 4 + 8 + 4 + 4 + 4 + 4
    return _line("split_text: 16,384 generator streams x 64 sentences, geometric(1/24) tokens + delimiter "
                 "per sentence, round-robin arrival, cut into (request, sentence, token)", n, ms, args.steps,
                 args.warmup, n * per,
                 {"token_stream_256": {"positions": n3, "ms": ms3, "fragments_per_s": n3 / (ms3 * 1e-3),
                                       "hbm_frac": n3 * per / (ms3 * 1e-3) / 1e9 / HBM_PEAK_GBPS}})


def bench_route_load(args):
    """Load-aware routing (flows keep their first destination; new flows take the
    shortest queue). Timed: the 2^26-fragment Zipf tree routed by its level-4 prefix
    (1,452 flows) to 256 destinations with every flow known (steady state; the
    queues are emptied between calls). Also: the first call (every flow new, the
    greedy assignment included), hash routing (alto_route) of the same keys, the
    queue balance of both, and the FacTool-shaped stream routed by claim to 32
    destinations step by step, each destination draining 128 fragments per step."""
    import time as T
    import torch
    from paper_2403_04311_amd import alto, workloads as W
    w5 = W.zipf_tree("cuda", leaves=1 << args.leaves_log2)
    keys, _ = alto.pack_keys(w5.path, w5.bits)
    bits = w5.bits
    del w5
    torch.cuda.empty_cache()
    n, D = keys.numel(), 256
    rt = alto.LoadRouter(bits, 4, D, 1 << 16, n)
    load = torch.zeros(D, dtype=torch.int64, device="cuda")
    perm = torch.empty(n, dtype=torch.int32, device="cuda")
    offs = torch.empty(D + 1, dtype=torch.int64, device="cuda")
    dest = torch.empty(n, dtype=torch.int32, device="cuda")
    counts = torch.zeros(2, dtype=torch.int64, device="cuda")
    st = alto.new_status()
    first = []
    for _ in range(3):
        rt.reset()
        load.zero_()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rt.route(keys, load, perm=perm, dest_offsets=offs, dest=dest, counts=counts, status=st)
        e1.record()
        torch.cuda.synchronize()
        first.append(e0.elapsed_time(e1))
    assert int(st.item()) == 0 and int(counts[0]) > 0
    flows = int(counts[0])
    bal_load = float(load.max()) / float(load.double().mean())

    def steady():
        load.zero_()
        rt.route(keys, load, perm=perm, dest_offsets=offs, dest=dest, counts=counts, status=st)
    ms = _timed(steady, args.steps, args.warmup)
    assert int(st.item()) == 0 and int(counts[0]) == 0 and int(counts[1]) == flows
    hws = alto.new_workspace(alto.workspace_bytes(bits, n, D))
    hoffs = torch.empty(D + 1, dtype=torch.int64, device="cuda")
    hst = alto.new_status()
    ms_hash = _timed(lambda: alto.route(keys, bits, 4, D, ws=hws, perm=perm, dest_offsets=hoffs, dest=dest,
                                        status=hst), args.steps, args.warmup)
    hc = (hoffs[1:] - hoffs[:-1]).double()
    bal_hash = float(hc.max()) / float(hc.mean())
    del hws, perm, dest, keys, rt
    torch.cuda.empty_cache()

    # the FacTool-shaped stream: claims as flows, 32 destinations, 128 fragments drained per step
    w = W.factool_stream("cuda")
    skeys, _ = alto.pack_keys(w.path, w.bits)
    step, steps = w.step, min(w.info["steps"], args.stream_steps)
    Ds, service = 32, 128
    srt = alto.LoadRouter(w.bits, 2, Ds, 1 << 20, step)
    sload = torch.zeros(Ds, dtype=torch.int64, device="cuda")
    hload = torch.zeros(Ds, dtype=torch.int64, device="cuda")
    sp = torch.empty(step, dtype=torch.int32, device="cuda")
    so = torch.empty(Ds + 1, dtype=torch.int64, device="cuda")
    sd = torch.empty(step, dtype=torch.int32, device="cuda")
    sc = torch.zeros(2, dtype=torch.int64, device="cuda")
    sst = alto.new_status()
    hws = alto.new_workspace(alto.workspace_bytes(w.bits, step, Ds))
    hso = torch.empty(Ds + 1, dtype=torch.int64, device="cuda")
    maxq = torch.zeros(steps, dtype=torch.int64, device="cuda")
    hmaxq = torch.zeros(steps, dtype=torch.int64, device="cuda")
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = T.perf_counter()
    for s in range(steps):
        k = skeys[s * step:(s + 1) * step]
        evs[s][0].record()
        srt.route(k, sload, perm=sp, dest_offsets=so, dest=sd, counts=sc, status=sst)
        evs[s][1].record()
        maxq[s] = sload.max()
        sload.sub_(service).clamp_(min=0)
        alto.route(k, w.bits, 2, Ds, ws=hws, perm=sp, dest_offsets=hso, dest=sd, status=hst)
        hload.add_(hso[1:] - hso[:-1])
        hmaxq[s] = hload.max()
        hload.sub_(service).clamp_(min=0)
    torch.cuda.synchronize()
    wall = (T.perf_counter() - t0) * 1e3
    assert int(sst.item()) == 0 and int(hst.item()) == 0
    dev = [a.elapsed_time(b) for a, b in evs]
    stream = {"steps": steps, "step_fragments": step, "destinations": Ds, "drain_per_step": service,
              "route_load_ms_p50": _pct(dev, 50), "route_load_ms_p99": _pct(dev, 99),
              "loop_ms_per_step_both_routers": wall / steps,
              "mean_longest_queue_load_aware": float(maxq.double().mean()),
              "mean_longest_queue_hash": float(hmaxq.double().mean())}
    return _line(f"load-aware routing: 2^{args.leaves_log2}-fragment Zipf depth-6 tree, {flows} level-4 flows known, "
                 f"256 destinations", n, ms, args.steps, args.warmup, n * (8 + 4 + 4),
                 {"first_call_ms": min(first), "hash_route_ms": ms_hash,
                  "longest_over_mean_queue": {"load_aware": bal_load, "hash": bal_hash},
                  "factool_stream": stream})


def bench_live_scaling(args):
    """Per-step cost of a stream step against the size of the carried state. A token
    stream in the token stream's layout (31, 6, 12) whose 256 sentences stay open (each
    declares 4,095 tokens): every 4,096-fragment step adds 16 tokens to each, so the
    live set grows by 4,096 leaves a step, to 1,044,480 after 255 steps. Reports the
    device time per step at several live-set sizes and the least-squares slope."""
    import numpy as np
    import torch
    from paper_2403_04311_amd import alto
    bits, G, per, steps = (31, 6, 12), 256, 16, 255
    step = G * per
    rng = np.random.default_rng(20240307)
    roots = rng.choice(1 << 31, size=G, replace=False).astype(np.int64)
    # step s: tokens s*16 .. s*16+15 of every generator's sentence 0, generator-major
    # within a tick (round robin), as the token stream arrives
    t = np.arange(steps * per, dtype=np.int64)
    tick, gen = np.meshgrid(t, np.arange(G), indexing="ij")
    path = np.stack([roots[gen.ravel()], np.zeros(gen.size, np.int64), tick.ravel()]).astype(np.int32)
    keys, st = alto.pack_keys(torch.from_numpy(path).cuda(), bits)
    n = keys.numel()
    fan = torch.empty((2, n), dtype=torch.int32, device="cuda")
    fan[0].fill_(64)
    fan[1].fill_(4095)
    p32 = torch.arange(n, dtype=torch.int32, device="cuda")
    out = alto.new_groups(step, 2, "concat", cap_tokens=step)
    status = alto.new_status()

    def run():
        s = alto.Stream(bits, 2, 64, 2, "concat", 1, max_live_leaves=steps * step, max_groups=1 << 12,
                        step_max=step)

        def one(i):
            s.step(keys[i * step:(i + 1) * step], fan[:, i * step:(i + 1) * step], p32[i * step:(i + 1) * step],
                   None, out=out, status=status)
        tot, per_ms = _stream_run(steps, one)
        s.close()
        return tot, per_ms
    run()   # one untimed pass (255 steps)
    tot, per_ms = run()
    assert int(status.item()) == 0 and int(out.counts[0]) == 0
    live = np.arange(steps) * step           # carried leaves before each step
    slope, icpt = np.polyfit(live, np.asarray(per_ms) * 1e3, 1)
    at = {}
    for lo in (0, 1 << 16, 1 << 18, 1 << 19, 1 << 20):
        sel = (live >= lo) & (live < lo + (1 << 16))
        if sel.any():
            at[str(lo)] = float(np.median(np.asarray(per_ms)[sel]) * 1e3)
    return _line("open token stream (live set growing 4,096 leaves a step to 1,044,480), token-stream layout, "
                 "concat per sentence, 64 destinations", step, tot / steps, steps, 1, 0,
                 {"step_us_p50_at_live": at, "step_us_per_1k_live": float(slope * 1e3), "step_us_at_live_0": float(icpt)})


WORKLOADS = {"tiny": bench_tiny, "factool": bench_factool, "tokens": bench_tokens, "live_scaling": bench_live_scaling,
             "factool_stream": bench_factool_stream, "join": bench_join, "split": bench_split,
             "route_load": bench_route_load}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=30,
                    help="untimed steps first (the GPU settles at its steady clock after ~20 steps "
                         "of the 2^26-fragment call)")
    ap.add_argument("--leaves-log2", type=int, default=26)
    ap.add_argument("--cpu-sample-log2", type=int, default=24)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stream-steps", type=int, default=10000,
                    help="route_load, factool_stream: steps of the FacTool-shaped stream (at most 10,000)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB before the workload (untimed), the "
                         "reference for scaling hardware byte counters")
    ap.add_argument("--derive-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the mean kernel's HBM traffic summary from two rocprofv3 --pmc "
                         "counter_collection.csv files (FETCH_SIZE, WRITE_SIZE) and exit")
    ap.add_argument("--pmc-command", default="", help="the rocprofv3 commands, recorded in the summary")
    ap.add_argument("--stream-overlap", default="ab", choices=["none", "a", "b", "ab"],
                    help="factool_stream: which stages (document a, claim b) route each step on a HIP stream of "
                         "their own (the stages always run on two streams)")
    ap.add_argument("--no-stage-overlap", action="store_true",
                    help="factool: run the claim stage after the document stage on one stream (by default the "
                         "claim stage of a batch runs on a second HIP stream beside the next batch's first stage)")
    ap.add_argument("--batch-overlap", action="store_true",
                    help="zipf64M: run each batch's gathers on a second HIP stream beside the next batch's routing "
                         "(measured slower: the persistent mean gather fills every CU)")
    ap.add_argument("--release", default="complete", choices=["complete", "in_order"],
                    help="streams: a group leaves when complete, or in child order within its parent")
    ap.add_argument("--workload", default="zipf64M", choices=["zipf64M", "all"] + sorted(WORKLOADS),
                    help="zipf64M (default): the 2^26-fragment Zipf batch")
    args = ap.parse_args()
    if args.derive_traffic:
        out = write_traffic_summary(args.derive_traffic[0], args.derive_traffic[1],
                                    args.copy_calibration_mib or 1024, args.pmc_command)
        print(json.dumps({k: out[k] for k in ("kernel", "traffic_bytes_per_launch", "calibration")}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)

    if args.workload != "zipf64M":
        names = sorted(WORKLOADS) if args.workload == "all" else [args.workload]
        for name in names:
            log(f"workload {name}")
            print(json.dumps(WORKLOADS[name](args)), flush=True)
        if args.workload != "all":
            return

    import ctypes as C
    import numpy as np
    import torch
    from paper_2403_04311_amd import alto, workloads as W

    dev = "cuda"
    lib = alto.load()
    if args.copy_calibration_mib:
        nb = args.copy_calibration_mib << 20
        a = torch.empty(nb, dtype=torch.uint8, device=dev)
        b = torch.empty(nb, dtype=torch.uint8, device=dev)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
        log(f"calibration copy of {args.copy_calibration_mib} MiB done")
    n = 1 << args.leaves_log2
    log(f"generating workload: 2^{args.leaves_log2} fragments")
    t0 = time.time()
    w = W.zipf_tree(dev, leaves=n)
    keys, st = alto.pack_keys(w.path, w.bits)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    w.path = None
    torch.cuda.empty_cache()
    log(f"workload ready in {time.time() - t0:.1f}s; level node counts {w.info['level_nodes']}")

    bits, La, Lm, Lr, D, dim = w.bits, w.agg_level, w.mask_level, w.route_level, w.num_dest, w.dim
    ws = alto.new_workspace(alto.workspace_bytes(bits, n, D, La, "mean", dim, Lm), dev)
    perm = torch.empty(n, dtype=torch.int32, device=dev)
    offs = torch.empty(D + 1, dtype=torch.int64, device=dev)
    dest = torch.empty(n, dtype=torch.int32, device=dev)
    cap = 1 << 16
    out = alto.new_groups(cap, La, "mean", dim, cap_mask=cap, device=dev, with_first=False)
    status = alto.new_status(dev)
    fan, pf = w.fan, w.payload_f32

    def step():
        alto.aggregate(keys, fan, bits, La, "mean", dim, Lm, Lr, D, None, pf, ws=ws, perm=perm,
                       dest_offsets=offs, dest=dest, out=out, status=status, n=n)

    # batches in flight on two HIP streams: a batch's gathers (bandwidth bound) on the
    # gather stream beside the next batch's routing, order and completion (mostly
    # latency bound) on the call's stream; two sets of workspace and outputs, and a
    # batch waits until the gathers of the batch two before it, which used the same
    # set, have ended
    overlap = args.batch_overlap
    gather = torch.cuda.Stream()
    if overlap:
        sets = [(ws, perm, offs, dest, out),
                (alto.new_workspace(alto.workspace_bytes(bits, n, D, La, "mean", dim, Lm), dev),
                 torch.empty(n, dtype=torch.int32, device=dev), torch.empty(D + 1, dtype=torch.int64, device=dev),
                 torch.empty(n, dtype=torch.int32, device=dev),
                 alto.new_groups(cap, La, "mean", dim, cap_mask=cap, device=dev, with_first=False))]
        gathered = [torch.cuda.Event(), torch.cuda.Event()]
        used = [False, False]
    calls = [0]

    def step_timed():
        if not overlap:
            step()
            return
        k = calls[0] & 1
        calls[0] += 1
        main = torch.cuda.current_stream()
        if used[k]:
            main.wait_event(gathered[k])
        w_, p_, o_, d_, g_ = sets[k]
        alto.aggregate(keys, fan, bits, La, "mean", dim, Lm, Lr, D, None, pf, ws=w_, perm=p_,
                       dest_offsets=o_, dest=d_, out=g_, status=status, n=n, stream=main, gather_stream=gather)
        gathered[k].record(gather)
        used[k] = True

    def settle():
        torch.cuda.current_stream().wait_stream(gather)
        torch.cuda.synchronize()

    for _ in range(args.warmup):
        step_timed()
    settle()
    if int(status.item()) != 0:
        raise SystemExit(f"status {int(status.item())} from alto_aggregate")
    E, T, M, P = [int(x) for x in out.counts.cpu()]
    log(f"warmup done: {E} groups emitted, {P} pending, mask nodes {M}")

    lib.alto_profile_begin.argtypes = [C.c_int32]
    lib.alto_profile_phases.argtypes = [C.c_uint32]
    lib.alto_profile_end.argtypes = [C.POINTER(C.c_float), C.POINTER(C.c_int32), C.c_int32]
    # timed region: only the mean kernel's event pair is recorded (each event pair
    # between two kernels idles the GPU for a few microseconds)
    assert lib.alto_profile_phases(1 << PHASES.index("mean_kernel")) == 0
    rc = lib.alto_profile_begin(4 * args.steps + 4)
    assert rc == 0
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    gather.wait_stream(torch.cuda.current_stream())
    for k in range(args.steps):
        step_timed()
        evs[k + 1].record(gather if overlap else torch.cuda.current_stream())   # the step's end
    settle()
    ms_total = evs[0].elapsed_time(evs[-1])
    per_step = sorted(evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps))
    ms = (C.c_float * len(PHASES))()
    calls = (C.c_int32 * len(PHASES))()
    rc = lib.alto_profile_end(ms, calls, len(PHASES))
    assert rc == 0
    kern_ms = ms[PHASES.index("mean_kernel")] / max(calls[PHASES.index("mean_kernel")], 1)
    assert int(status.item()) == 0
    ms_step = ms_total / args.steps
    seq_ms = None
    if overlap:
        # the same steps one after the other on one stream, for comparison
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for k in range(args.steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        seq_ms = e0.elapsed_time(e1) / args.steps
        assert int(status.item()) == 0
    # one more call, untimed, with every phase recorded (diagnostics)
    assert lib.alto_profile_phases(0xFFFFFFFF) == 0
    assert lib.alto_profile_begin(32) == 0
    step()
    torch.cuda.synchronize()
    assert lib.alto_profile_end(ms, calls, len(PHASES)) == 0
    phase_ms = {p: (ms[i] / calls[i] if calls[i] else None) for i, p in enumerate(PHASES)}

    # algorithmic bytes: inputs read once, outputs written once
    nfan_levels = (w.depth - 1) - min(La, Lm) + 1
    per_frag = 8 + 4 * nfan_levels + 4 * dim + 4 + 4
    per_group = 8 + 4 + 8 + 4 * (La - 1) + 4 * dim
    path_bytes = n * per_frag + E * per_group + M * 9 + (D + 1) * 8
    kern_bytes = n * dim * 4 + E * dim * 4
    achieved = kern_bytes / (kern_ms * 1e-3) / 1e9
    path_gbps = path_bytes / (ms_step * 1e-3) / 1e9
    res = {
        "metric": "fragments/sec routed+aggregated at 1 MI355X; achieved HBM GB/s vs peak",
        "value": n / (ms_step * 1e-3),
        "unit": "fragments/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_median": per_step[len(per_step) // 2],
        "ms_per_step_min": per_step[0],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"zipf depth-6 tree, 2^{args.leaves_log2} fragments, 128-d f32 mean at level 4, "
                               "mask at level 2, 256 destinations by level-4 prefix, one batch per step"
                               + (" (a batch's gathers on a second HIP stream beside the next batch's routing)"
                                  if overlap else ""),
                   "fragments": n, "groups": E, "mask_nodes": M, "dim": dim, "num_dest": D},
        "batch_overlap": overlap,
        "sequential_ms_per_step": seq_ms,
        "roofline": {"bound": "hbm", "kernel": "k_mean (fp64-accumulating row gather)",
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": measured_traffic(),
                     "algorithmic_bytes_per_launch": kern_bytes, "avg_launch_ms": kern_ms},
        "path_roofline": {"algorithmic_bytes_per_step": path_bytes, "bytes_per_fragment": per_frag,
                          "achieved": path_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                          "frac": path_gbps / HBM_PEAK_GBPS},
        "phase_ms_one_call": phase_ms,
        "read_ceiling_gbps": read_ceiling_gbps(dev),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        res["cpu_baseline"] = cpu_baseline(args.cpu_sample_log2)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
