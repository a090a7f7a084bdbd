#!/usr/bin/env python3
"""Fragments/s routed + aggregated on one MI355X, with the dominant kernel's
achieved HBM bandwidth against the 8 TB/s peak.

Workload (default): skewed Zipf(1.2) depth-6 tree of 2^26 fragments, keys packed
before timing, 128-d float32 payload per fragment, route by the level-4 prefix to
256 destinations, mean-pool at level 4, completion mask at level 2. One step =
one alto_aggregate call over the whole batch (routing outputs perm, dest_offsets,
dest, plus groups, means and mask). Inputs are resident in HBM before timing.

Prints one JSON line. --gpus N > 1 is refused: this build runs on one GPU.
"""
import argparse
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
    w = W.config5("cpu", leaves=1 << leaves_log2)
    path, fan, x = w.path.numpy(), w.fan.numpy(), w.payload_f32.numpy()
    t0 = time.perf_counter()
    keys = O.pack_keys(path, w.bits)
    O.aggregate(keys, fan, w.bits, w.agg_level, w.op, w.dim, w.mask_level, w.route_level, w.num_dest,
                None, x)
    dt = time.perf_counter() - t0
    return {"value": (1 << leaves_log2) / dt, "unit": "fragments/s", "cores": 1, "kind": "oracle",
            "sample": f"same generator at 2^{leaves_log2} leaves (1/{1 << (26 - leaves_log2)} of the "
                      f"workload): pack + route + aggregate, {dt:.1f} s single-threaded numpy"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--leaves-log2", type=int, default=26)
    ap.add_argument("--cpu-sample-log2", type=int, default=24)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB before the workload (untimed), the "
                         "reference for scaling hardware byte counters")
    ap.add_argument("--derive-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the mean kernel's HBM traffic summary from two rocprofv3 --pmc "
                         "counter_collection.csv files (FETCH_SIZE, WRITE_SIZE) and exit")
    ap.add_argument("--pmc-command", default="", help="the rocprofv3 commands, recorded in the summary")
    args = ap.parse_args()
    if args.derive_traffic:
        out = write_traffic_summary(args.derive_traffic[0], args.derive_traffic[1],
                                    args.copy_calibration_mib or 1024, args.pmc_command)
        print(json.dumps({k: out[k] for k in ("kernel", "traffic_bytes_per_launch", "calibration")}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)

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
    w = W.config5(dev, leaves=n)
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

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if int(status.item()) != 0:
        raise SystemExit(f"status {int(status.item())} from alto_aggregate")
    E, T, M, P = [int(x) for x in out.counts.cpu()]
    log(f"warmup done: {E} groups emitted, {P} pending, mask nodes {M}")

    lib.alto_profile_begin.argtypes = [C.c_int32]
    lib.alto_profile_end.argtypes = [C.POINTER(C.c_float), C.POINTER(C.c_int32), C.c_int32]
    rc = lib.alto_profile_begin(16 * args.steps + 16)
    assert rc == 0
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_total = e0.elapsed_time(e1)
    ms = (C.c_float * len(PHASES))()
    calls = (C.c_int32 * len(PHASES))()
    rc = lib.alto_profile_end(ms, calls, len(PHASES))
    assert rc == 0
    phase_ms = {p: (ms[i] / calls[i] if calls[i] else None) for i, p in enumerate(PHASES)}
    assert int(status.item()) == 0
    ms_step = ms_total / args.steps

    # algorithmic bytes: inputs read once, outputs written once
    nfan_levels = (w.depth - 1) - min(La, Lm) + 1
    per_frag = 8 + 4 * nfan_levels + 4 * dim + 4 + 4
    per_group = 8 + 4 + 8 + 4 * (La - 1) + 4 * dim
    path_bytes = n * per_frag + E * per_group + M * 9 + (D + 1) * 8
    kern_bytes = n * dim * 4 + E * dim * 4
    kern_ms = phase_ms["mean_kernel"]
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
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"zipf depth-6 tree, 2^{args.leaves_log2} fragments, 128-d f32 mean at level 4, "
                               "mask at level 2, 256 destinations by level-4 prefix, one batch",
                   "fragments": n, "groups": E, "mask_nodes": M, "dim": dim, "num_dest": D},
        "roofline": {"bound": "hbm", "kernel": "k_mean (fp64-accumulating row gather)",
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": measured_traffic(),
                     "algorithmic_bytes_per_launch": kern_bytes, "avg_launch_ms": kern_ms},
        "path_roofline": {"algorithmic_bytes_per_step": path_bytes, "bytes_per_fragment": per_frag,
                          "achieved": path_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                          "frac": path_gbps / HBM_PEAK_GBPS},
        "phase_ms": phase_ms,
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        res["cpu_baseline"] = cpu_baseline(args.cpu_sample_log2)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
