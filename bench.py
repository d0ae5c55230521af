#!/usr/bin/env python3
"""Prof-K top-k throughput on one MI355X.

Workload: one vector of N = 2^28 standard-normal fp32 values (seed 1), exact
top-k with k = 1024 and eps = 1e-6 -- the large-N, small-k regime of the
paper's synthetic study (Sec. 5), synthetic data.  One step is one
profk_topk call: sampling, threshold, the filter-and-compact pass and the
exact refinement, with the input already resident in HBM.

Prints one JSON line.  `value` is effective GB/s (N * 4 bytes / step time);
`roofline` times the filter kernel alone with HIP events recorded by the
library around each launch on its own stream; `cpu_baseline` times the CPU
oracle (exact stable-sort top-k) on a prefix of the same input.
"""

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBPS = 8000.0
N_DEFAULT = 2**28
K_DEFAULT = 1024
COUNTERS = os.path.join(ROOT, "profiles", "filter_counters.json")
CSRC = os.path.join(ROOT, "paper_2608_12573_amd", "csrc")
# Every source the filter kernel is compiled from: the committed counters
# stand for this exact code and are dropped once any of these changes.
FILTER_SRCS = ("kernels_flat.hip", "filter_tile.h", "device_common.h", "launch.h", "topk_block.h")


def filter_source_sha256():
    h = hashlib.sha256()
    for name in FILTER_SRCS:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


class HipEvents:
    """Minimal hipEvent_t access for timing on the library's stream."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        if self.hip.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def destroy(self, ev):
        self.hip.hipEventDestroy(ev)


def counters_traffic(n_launch_bytes):
    """HBM bytes per filter launch from the committed rocprofv3 counter
    summary, or None when it is missing or the kernel source changed since."""
    try:
        with open(COUNTERS) as f:
            c = json.load(f)
        sha = filter_source_sha256()
    except OSError:
        return None
    if c.get("kernel_source_sha256") != sha:
        return None
    return c.get("traffic_bytes_per_launch")


def cpu_baseline(x_np, k, budget_s=10.0):
    """The oracle's exact top-k (full stable sort, oracle.exact) on a 2^24
    prefix of the workload, repeated for about budget_s seconds."""
    sys.path.insert(0, ROOT)
    from oracle import exact, keys
    n_s = min(x_np.size, 2**24)
    bits = keys.f32_bits(x_np[:n_s])
    reps, t0 = 0, time.perf_counter()
    while True:
        exact.topk(bits, "f32", k)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    per = el / reps
    return {"value": round(n_s * 4 / per / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"oracle.exact.topk (numpy stable argsort, one thread) on the first 2^24 of the "
                      f"2^28 values, k={k}, {reps} runs, {per * 1e3:.0f} ms each",
            "elements_per_s": round(n_s / per, 1)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--k", type=int, default=K_DEFAULT)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-torch-baseline", action="store_true")
    ap.add_argument("--no-copy-probe", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    sys.path.insert(0, ROOT)
    import paper_2608_12573_amd as pk
    import workloads

    N, k = N_DEFAULT, args.k
    x_np = workloads.normal_f32(N, seed=1)
    x = torch.from_numpy(x_np).cuda()
    p = pk.plan(N, k, 1e-6, 1.0)
    ws = pk.workspace(p, pk.F32)
    out = (torch.empty(k, dtype=torch.float32, device="cuda"),
           torch.empty(k, dtype=torch.int64, device="cuda"))
    info = torch.empty(pk.INFO_BYTES, dtype=torch.uint8, device="cuda")
    lib = pk.lib()

    def step():
        pk.topk(x, k, p=p, ws=ws, out=out, info=info, seed=0)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    ev = HipEvents()
    pairs = [(ev.create(), ev.create()) for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for a, b in pairs:
        lib.profk_set_trace_events(a, b)
        step()
    stop.record()
    torch.cuda.synchronize()
    lib.profk_set_trace_events(None, None)
    total_ms = start.elapsed_time(stop)
    filt_ms = [ev.elapsed_ms(a, b) for a, b in pairs]
    for a, b in pairs:
        ev.destroy(a)
        ev.destroy(b)

    rec = pk.read_info(info)[0]
    ms_per_step = total_ms / args.steps
    filt_avg_ms = float(np.mean(filt_ms))
    in_bytes = N * 4
    value = in_bytes / (ms_per_step * 1e-3) / 1e9
    filt_bytes = in_bytes + int(rec["count"]) * 8
    achieved = filt_bytes / (filt_avg_ms * 1e-3) / 1e9

    line = {
        "metric": "effective GB/s and elements/s at N=2^28 fp32, k=1024; % of HBM peak",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": f"one fp32 vector, N=2^28 standard normal (seed 1), exact top-k k={k}, "
                               f"eps=1e-6, sample seed 0", "N": N, "k": k, "eps": 1e-6,
                   "plan": {"S": p.S, "t": p.t, "M": p.M}},
        "elements_per_s": round(N / (ms_per_step * 1e-3), 1),
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "filter_ms": round(filt_avg_ms, 5),
        "filter_pct_hbm_peak": round(100 * in_bytes / (filt_avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
        "count": int(rec["count"]),
        "status": int(rec["status"]),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": counters_traffic(filt_bytes), "kernel": "k_filter<f32>",
                     "algorithmic_bytes_per_launch": filt_bytes},
    }

    if not args.no_torch_baseline:
        for _ in range(3):
            torch.topk(x, k, sorted=True)
        torch.cuda.synchronize()
        reps = 10
        start.record()
        for _ in range(reps):
            tv, ti = torch.topk(x, k, sorted=True)
        stop.record()
        torch.cuda.synchronize()
        t_ms = start.elapsed_time(stop) / reps
        same_vals = bool(torch.equal(tv, out[0]))
        line["torch_topk"] = {"ms": round(t_ms, 4), "GB/s": round(in_bytes / (t_ms * 1e-3) / 1e9, 1),
                              "values_equal": same_vals, "speedup_vs_torch": round(t_ms / ms_per_step, 3)}

    if not args.no_copy_probe:
        # A plain device-to-device copy of the same 1 GiB: the practical
        # streaming ceiling on this GPU, and the reference kernel that scales
        # the FETCH_SIZE / WRITE_SIZE counters into bytes.
        dst = torch.empty_like(x)
        for _ in range(2):
            dst.copy_(x)
        torch.cuda.synchronize()
        reps = 5
        start.record()
        for _ in range(reps):
            dst.copy_(x)
        stop.record()
        torch.cuda.synchronize()
        c_ms = start.elapsed_time(stop) / reps
        line["copy_probe"] = {"bytes_read": in_bytes, "bytes_written": in_bytes, "ms": round(c_ms, 4),
                              "GB/s": round(2 * in_bytes / (c_ms * 1e-3) / 1e9, 1)}
        del dst

    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(x_np, k)

    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
