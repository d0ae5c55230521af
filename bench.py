#!/usr/bin/env python3
"""Prof-K top-k throughput on one MI355X.

Default workload: one vector of N = 2^28 standard-normal fp32 values
(seed 1), exact top-k with k = 1024 and eps = 1e-6 -- the large-N, small-k
regime of the paper's synthetic study (Sec. 5), synthetic data.  One step
is one profk_topk call: sampling, threshold, the filter-and-compact pass
and the exact refinement, with the input already resident in HBM.

--workload picks one of the other shapes the parity tests cover (the small
uniform vector, the adversarial 2^26 vectors, the per-row bf16 batch and
the flattened BatchTopK select); the printed line then describes that one.

Prints one JSON line.  `value` is effective GB/s (input bytes / step time);
`roofline` times the dominant kernel -- the filter, or for the per-row
path its single fused kernel -- with HIP events recorded by the library
around the launch on its own stream; `cpu_baseline` times the CPU oracle
(exact stable-sort top-k) on a bounded prefix of the same input.
"""

import argparse
import csv
import ctypes
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBPS = 8000.0
COUNTERS = os.path.join(ROOT, "profiles", "filter_counters.json")
CSRC = os.path.join(ROOT, "paper_2608_12573_amd", "csrc")
# Every source the filter kernel is compiled from: the committed counters
# stand for this exact code and are dropped once any of these changes.
FILTER_SRCS = ("kernels_filter.hip", "filter_tile.h", "device_common.h", "launch.h")
WORKLOADS = ("c2", "c1", "c3a", "c3b", "c3c", "c3d", "c3d2", "c4", "c5", "c5r", "c5p", "sae")
MFMA_BF16_PEAK_TFLOPS = 2500.0
FLUSH_BYTES = 512 << 20


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


def counters_traffic(workload_key):
    """HBM bytes per filter launch from the committed rocprofv3 counter
    summary, or None when it covers another workload or the kernel source
    changed since it was taken."""
    try:
        with open(COUNTERS) as f:
            c = json.load(f)
        sha = filter_source_sha256()
    except OSError:
        return None
    if c.get("kernel_source_sha256") != sha or c.get("workload_key") != workload_key:
        return None
    return c.get("traffic_bytes_per_launch")


def write_counters(fetch_dir, write_dir, bench_json):
    """profiles/filter_counters.json from two rocprofv3 --pmc runs of the
    default workload (FETCH_SIZE, then WRITE_SIZE) and the JSON line one of
    them printed.  The counters' units are calibrated on the 1 GiB device
    copy bench.py's copy probe makes in the same runs."""
    def per_dispatch(d, counter):
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            sys.exit(f"no counter_collection.csv under {d}")
        disp = {}
        for f in files:
            with open(f) as fh:
                for r in csv.DictReader(fh):
                    if r["Counter_Name"] != counter:
                        continue
                    key = (r["Kernel_Name"], int(r["Grid_Size"]), r["Dispatch_Id"])
                    disp[key] = disp.get(key, 0.0) + float(r["Counter_Value"])
        kern = {}
        for (name, grid, _), v in disp.items():
            kern.setdefault((name, grid), []).append(v)
        return {key: (sum(v) / len(v), len(v)) for key, v in kern.items()}

    fetch, write = per_dispatch(fetch_dir, "FETCH_SIZE"), per_dispatch(write_dir, "WRITE_SIZE")
    with open(bench_json) as fh:
        line = json.loads(fh.read().strip().splitlines()[-1])

    def pick(table, pred, biggest=False):
        keys = [key for key in table if pred(key[0])]
        if not keys:
            sys.exit("kernel not found in the counter files")
        return max(keys, key=lambda key: table[key][0]) if biggest else keys[0]

    is_filter = lambda n: "k_filter<0, false," in n
    is_copy = lambda n: "copyBuffer" in n
    fk, ck = pick(fetch, is_filter), pick(fetch, is_copy, biggest=True)
    wk, cwk = pick(write, is_filter), pick(write, is_copy, biggest=True)
    gib = float(1 << 30)
    fpu, wpu = gib / fetch[ck][0], gib / write[cwk][0]
    fb, wb = fetch[fk][0] * fpu, write[wk][0] * wpu
    algo = line["roofline"]["algorithmic_bytes_per_launch"]
    out = {
        "kernel": "profk::k_filter<0, false, U> (fp32 filter-and-compact)",
        "workload_key": "c2-k1024",
        "workload": line["config"]["workload"] + f"; {line['count']} survivors",
        "commands": [
            "rocprofv3 --pmc FETCH_SIZE -d gpurun_out/pmc_fetch -o fetch --output-format csv -- "
            "python bench.py --steps 3 --warmup 1 --no-cpu-baseline --no-torch-baseline",
            "rocprofv3 --pmc WRITE_SIZE -d gpurun_out/pmc_write -o write --output-format csv -- "
            "python bench.py --steps 3 --warmup 1 --no-cpu-baseline --no-torch-baseline",
            "python bench.py --write-counters gpurun_out/pmc_fetch gpurun_out/pmc_write "
            "gpurun_out/pmc_fetch.json",
        ],
        "fetch_size_kib_per_dispatch": round(fetch[fk][0], 2),
        "write_size_kib_per_dispatch": round(write[wk][0], 2),
        "dispatches": [fetch[fk][1], write[wk][1]],
        "calibration": {
            "kernel": "__amd_rocclr_copyBuffer (the copy probe: torch copy_ of the same 1 GiB tensor, "
                      "in the same runs)",
            "bytes_read": 1 << 30, "bytes_written": 1 << 30,
            "fetch_size_kib": round(fetch[ck][0], 2), "write_size_kib": round(write[cwk][0], 2),
            "fetch_bytes_per_kib_unit": round(fpu, 3), "write_bytes_per_kib_unit": round(wpu, 3),
        },
        "fetch_bytes_per_launch": int(round(fb)),
        "write_bytes_per_launch": int(round(wb)),
        "traffic_bytes_per_launch": int(round(fb + wb)),
        "algorithmic_bytes_per_launch": algo,
        "traffic_over_algorithmic": round((fb + wb) / algo, 5),
        "kernel_source_sha256": filter_source_sha256(),
        "kernel_sources": list(FILTER_SRCS),
    }
    with open(COUNTERS, "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    print(json.dumps(out, indent=1))


class Workload:
    """Input, preallocated outputs and one step of the path for one shape."""

    def __init__(self, name, k_arg, torch, pk, wl, lex=False):
        self.name = name
        self.lex = lex
        self.flops = None   # set for a matrix-core workload
        rule = dict(lexicographic=1) if lex else {}
        self.rows = False
        self.es = 4
        self.recall = 1.0

        def f32(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()

        if name in ("c1", "c2") or name.startswith("c3"):
            if name == "c1":
                N, k, host, what = 2**20, 64, wl.uniform_f32(2**20, seed=0), "Uniform(0,1) (seed 0)"
            elif name == "c2":
                N, k = 2**28, k_arg
                host, what = wl.normal_f32(N, seed=1), "standard normal (seed 1)"
            else:
                N, k = 2**26, 512
                host, what = {
                    "c3a": lambda: (wl.pareto_f32(N, seed=2), "Pareto alpha=1.1 (seed 2)"),
                    "c3b": lambda: (wl.zeros90_f32(N, seed=2), "90% +0.0, 10% Uniform(0,1) (seed 2)"),
                    "c3c": lambda: (wl.ramp_f32(N), "ascending ramp float32(i)"),
                    "c3d": lambda: (wl.plateau_f32(N, seed=2, first_rank=257, width=10_000),
                                    "Uniform(0,1) with a 1e4-wide plateau at ranks 257..10256 (seed 2)"),
                    "c3d2": lambda: (wl.plateau_f32(N, seed=2, first_rank=257, width=200_000),
                                     "Uniform(0,1) with a 2e5-wide plateau at ranks 257..200256 (seed 2)"),
                }[name]()
            self.desc = (f"one fp32 vector, N=2^{N.bit_length() - 1} {what}, exact top-k k={k}, "
                         f"eps=1e-6, sample seed 0")
            self.host = host
            self.x = f32(host)
            self.p = pk.plan(N, k, 1e-6, 1.0, **rule)
            self.kernel = "k_filter<f32>"
            self.ws = pk.workspace(self.p, pk.F32)
            self.out = (torch.empty(k, dtype=torch.float32, device="cuda"),
                        torch.empty(k, dtype=torch.int64, device="cuda"))
            self.info = torch.empty(pk.INFO_BYTES, dtype=torch.uint8, device="cuda")
            self.step = lambda: pk.topk(self.x, k, p=self.p, ws=self.ws, out=self.out, info=self.info,
                                        seed=0)
            self.torch_ref = lambda: torch.topk(self.x, k, sorted=True)
            self.N, self.k = N, k
        elif name == "c4":
            B, D, k = 4096, 131072, 32
            bits = wl.relu_normal_bf16((B, D), seed=3)
            self.host = bits
            self.x = torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)
            self.rows, self.es = True, 2
            self.p = pk.plan_rows(D, k, 1e-6, 1.0, **rule)
            self.kernel = "k_rows<bf16>"
            self.desc = (f"bf16 rows [4096, 131072] of ReLU(N(0,1)) (seed 3), per-row top-k k={k}, "
                         f"eps=1e-6, one row plan, sample seed 0")
            self.ws = pk.workspace(self.p, pk.BF16, B)
            self.out = (torch.empty((B, k), dtype=torch.bfloat16, device="cuda"),
                        torch.empty((B, k), dtype=torch.int64, device="cuda"))
            self.info = torch.empty(B * pk.INFO_BYTES, dtype=torch.uint8, device="cuda")
            self.step = lambda: pk.topk_rows(self.x, k, p=self.p, ws=self.ws, out=self.out,
                                             info=self.info, seed=0)
            self.torch_ref = lambda: torch.topk(self.x, k, dim=1, sorted=True)
            self.N, self.k, self.B, self.D = B * D, k, B, D
        elif name in ("c5", "c5r", "c5p"):
            # c5p: the paper's SAE shape, [4096, 12288] with k = 32 per row
            B, D, k_row = (4096, 12288, 32) if name == "c5p" else (4096, 65536, 64)
            self.recall = 0.95 if name == "c5r" else 1.0
            host = wl.sae_preacts_f32(B=B, D=D, seed=4)
            self.host = host.reshape(-1)
            self.x = f32(host).view(B, D)
            K = B * k_row
            self.p = pk.plan(B * D, K, 1e-6, self.recall, **rule)
            self.kernel = "k_filter<f32>"
            self.desc = (f"BatchTopK select over fp32 [{B}, {D}] N(-0.5,1) pre-activations with 1% "
                         f"hot columns +3 (seed 4), K={B}*{k_row}={B * k_row}, eps=1e-6, recall {self.recall}, "
                         f"sample seed 0")
            self.ws = pk.workspace(self.p, pk.F32)
            self.out = (torch.empty(K, dtype=torch.float32, device="cuda"),
                        torch.empty(K, dtype=torch.int64, device="cuda"))
            self.info = torch.empty(pk.INFO_BYTES, dtype=torch.uint8, device="cuda")
            self.step = lambda: pk.batchtopk(self.x, k_row, recall=self.recall, p=self.p, ws=self.ws,
                                             out=self.out, info=self.info, seed=0)
            self.torch_ref = lambda: torch.topk(self.x.view(-1), K, sorted=True)
            self.N, self.k = B * D, K
        elif name == "sae":
            # the paper's BatchTopK SAE shape, with the selection fused into
            # the encoder GEMM: the B x d_dict latents are never written
            B, d_model, d_dict, k_row = 4096, 512, 12288, 32
            m = wl.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=6)
            bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
            self.sx, self.sw, self.sb = bf(m["x"]), bf(m["w_enc"]), torch.from_numpy(m["b_enc"]).cuda()
            self.host = None
            self.x = self.sx
            K = B * k_row
            self.p = pk.plan_sae(B, d_dict, k_row, 1e-6, 1.0, **rule)
            self.kernel = "k_sae_filter (bf16 MFMA GEMM + filter epilogue)"
            self.desc = (f"BatchTopK SAE encoder: bf16 x [{B}, {d_model}] (N(0,1)) times W_enc [{d_dict}, {d_model}] "
                         f"(N(0,1/d_model)), fp32 bias -0.5 (+1.5 on every 100th latent), ReLU, top K={B}*{k_row}="
                         f"{K} of the flattened latents, eps=1e-6, sample seed 0 (seed 6 model)")
            self.ws = pk.sae_workspace(self.p, B, d_dict)
            self.out = (torch.empty(K, dtype=torch.float32, device="cuda"),
                        torch.empty(K, dtype=torch.int64, device="cuda"))
            self.info = torch.empty(pk.INFO_BYTES, dtype=torch.uint8, device="cuda")
            self.step = lambda: pk.sae_encode_topk(self.sx, self.sw, self.sb, k_row, p=self.p, ws=self.ws,
                                                   out=self.out, info=self.info, seed=0)
            self.dense = torch.empty((B, d_dict), dtype=torch.float32, device="cuda")
            self.p_flat = pk.plan(B * d_dict, K)
            self.ws_flat = pk.workspace(self.p_flat, pk.F32)
            self.out_flat = (torch.empty(K, dtype=torch.float32, device="cuda"),
                             torch.empty(K, dtype=torch.int64, device="cuda"))

            def unfused():
                pk.sae_encode_dense(self.sx, self.sw, self.sb, out=self.dense)
                return pk.batchtopk(self.dense, k_row, p=self.p_flat, ws=self.ws_flat, out=self.out_flat, seed=0)
            self.unfused = unfused

            def torch_ref():
                z = torch.relu(torch.matmul(self.sx, self.sw.t()).float() + self.sb)
                return torch.topk(z.view(-1), K, sorted=True)
            self.torch_ref = torch_ref
            self.N, self.k, self.es = B * d_dict, K, 4
            self.flops = 2 * B * d_model * d_dict
        else:
            raise SystemExit(f"unknown workload {name}; choose from {', '.join(WORKLOADS)}")
        self.in_bytes = self.N * self.es
        if lex:
            self.desc += "; tie-exact filter on (key, -index) pairs"

    def key(self):
        return f"{self.name}-k{self.k}" + ("-lex" if self.lex else "")


def cpu_baseline(w, budget_s=10.0):
    """The oracle's exact top-k (full stable sort, oracle.exact) on a bounded
    prefix of the workload -- 2^24 values, or 128 rows of the per-row batch --
    repeated for about budget_s seconds."""
    sys.path.insert(0, ROOT)
    from oracle import exact, keys
    if w.rows:
        R = 128
        bits = w.host[:R]
        run = lambda: exact.topk_rows(bits, "bf16", w.k)
        n_s, what = R * w.D, f"oracle.exact.topk_rows on the first {R} of the {w.B} rows"
    else:
        n_s = min(w.N, 2**24)
        bits = keys.f32_bits(w.host[:n_s])
        kk = min(w.k, n_s)
        run = lambda: exact.topk(bits, "f32", kk)
        what = f"oracle.exact.topk on the first 2^{n_s.bit_length() - 1} of the {w.N} values, k={kk}"
    reps, t0 = 0, time.perf_counter()
    while True:
        run()
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    per = el / reps
    return {"value": round(n_s * w.es / per / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{what} (numpy stable argsort, one thread), {reps} runs, {per * 1e3:.0f} ms each",
            "elements_per_s": round(n_s / per, 1)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    # A GPU idle during input generation needs a few milliseconds of work to
    # reach its steady clocks: after 5 steps the per-row workload still reads
    # 7 % slower than after 50.
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="c2", choices=WORKLOADS)
    ap.add_argument("--k", type=int, default=1024, help="k of the default N=2^28 workload")
    ap.add_argument("--cold", action="store_true",
                    help="also time each step after overwriting 512 MiB (flushes the last-level cache)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-torch-baseline", action="store_true")
    ap.add_argument("--no-copy-probe", action="store_true")
    ap.add_argument("--lexicographic", action="store_true",
                    help="plan with the tie-exact filter rule on (key, -index) pairs")
    ap.add_argument("--write-counters", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "BENCH_JSON"),
                    help="write profiles/filter_counters.json from two rocprofv3 --pmc runs and exit")
    args = ap.parse_args()
    if args.write_counters:
        write_counters(*args.write_counters)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    sys.path.insert(0, ROOT)
    import paper_2608_12573_amd as pk
    import workloads

    w = Workload(args.workload, args.k, torch, pk, workloads, lex=args.lexicographic)
    lib = pk.lib()
    for _ in range(args.warmup):
        w.step()
    torch.cuda.synchronize()

    # The timed steps: nothing but the calls themselves on the stream.
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        w.step()
    stop.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(stop) / args.steps

    # The dominant kernel alone: the library records HIP events right before
    # and after the filter launch on its stream (a separate pass, since the
    # extra events add gaps between the launches).
    if w.rows:
        kern_ms = ms_per_step  # the per-row path is one kernel
    else:
        ev = HipEvents()
        pairs = [(ev.create(), ev.create()) for _ in range(args.steps)]
        for a, b in pairs:
            lib.profk_set_trace_events(a, b)
            w.step()
        torch.cuda.synchronize()
        lib.profk_set_trace_events(None, None)
        kern_ms = float(np.mean([ev.elapsed_ms(a, b) for a, b in pairs]))
        for a, b in pairs:
            ev.destroy(a)
            ev.destroy(b)

    recs = pk.read_info(w.info)
    if w.rows:
        count = int(recs["count"].sum())
        status = {str(int(s)): int((recs["status"] == s).sum()) for s in np.unique(recs["status"])}
        # one read of the batch, the outputs and the per-row reports
        kern_bytes = w.in_bytes + w.B * w.k * (w.es + 8) + w.B * pk.INFO_BYTES
    else:
        count = int(recs[0]["count"])
        status = int(recs[0]["status"])
        kern_bytes = w.in_bytes + count * 8  # one read of the input, (key, index) per survivor
    value = w.in_bytes / (ms_per_step * 1e-3) / 1e9
    achieved = kern_bytes / (kern_ms * 1e-3) / 1e9
    if w.flops:
        roofline = {"bound": "mfma", "achieved": round(w.flops / (kern_ms * 1e-3) / 1e12, 1),
                    "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(w.flops / (kern_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                    "traffic": None, "kernel": w.kernel, "algorithmic_flops_per_launch": w.flops}
    else:
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                    "traffic": counters_traffic(w.key()), "kernel": w.kernel,
                    "algorithmic_bytes_per_launch": kern_bytes}

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
        "dtype": "u16" if w.es == 2 else "u32",
        "data": "synthetic",
        "config": {"workload": w.desc, "N": w.N, "k": w.k, "eps": 1e-6, "recall": w.recall,
                   "plan": {"S": w.p.S, "t": w.p.t, "M": w.p.M, "mode": w.p.mode,
                            "lexicographic": int(w.p.lexicographic)}},
        "elements_per_s": round(w.N / (ms_per_step * 1e-3), 1),
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "kernel_ms": round(kern_ms, 5),
        "kernel_pct_hbm_peak": round(100 * w.in_bytes / (kern_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
        "count": count,
        "status": status,
        "roofline": roofline,
    }
    if w.flops:
        # the latent matrix a dense pipeline would write and then read
        line["metric"] = "BatchTopK SAE encoder + selection: effective GB/s of fp32 latents; MFMA roofline"
        line["dtype"] = "bf16"
        for key in ("pct_hbm_peak", "kernel_pct_hbm_peak"):
            line.pop(key)
        line["step_tflops"] = round(w.flops / (ms_per_step * 1e-3) / 1e12, 1)
        for _ in range(2):
            w.unfused()
        torch.cuda.synchronize()
        start.record()
        for _ in range(5):
            w.unfused()
        stop.record()
        torch.cuda.synchronize()
        u_ms = start.elapsed_time(stop) / 5
        line["unfused"] = {"what": "profk_sae_encode_dense (the same GEMM, latents written) + profk_batchtopk",
                           "ms": round(u_ms, 4), "values_equal": bool(torch.equal(w.out_flat[0], w.out[0])),
                           "indices_equal": bool(torch.equal(w.out_flat[1], w.out[1])),
                           "speedup_of_fused": round(u_ms / ms_per_step, 3)}

    if args.cold:
        flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        cold = []
        for i in range(args.steps):
            flush.fill_(float(i))
            start.record()
            w.step()
            stop.record()
            torch.cuda.synchronize()
            cold.append(start.elapsed_time(stop))
        line["cold_ms_per_step"] = round(float(np.median(cold)), 5)
        del flush

    if not args.no_torch_baseline:
        for _ in range(2):
            w.torch_ref()
        torch.cuda.synchronize()
        reps = 5
        start.record()
        for _ in range(reps):
            tv, ti = w.torch_ref()
        stop.record()
        torch.cuda.synchronize()
        t_ms = start.elapsed_time(stop) / reps
        line["torch_topk"] = {"ms": round(t_ms, 4), "GB/s": round(w.in_bytes / (t_ms * 1e-3) / 1e9, 1),
                              "values_equal": bool(torch.equal(tv, w.out[0])),
                              "speedup_vs_torch": round(t_ms / ms_per_step, 3)}
        if w.flops:
            line["torch_topk"]["what"] = ("torch.matmul (bf16 output) + bias + relu + torch.topk; its latents "
                                          "are rounded to bf16, so values differ")
        del tv, ti

    if not args.no_copy_probe and not w.flops:
        # A plain device-to-device copy of the same input: the practical
        # streaming ceiling on this GPU, and the reference kernel that scales
        # the FETCH_SIZE / WRITE_SIZE counters into bytes.
        dst = torch.empty_like(w.x)
        for _ in range(2):
            dst.copy_(w.x)
        torch.cuda.synchronize()
        reps = 5
        start.record()
        for _ in range(reps):
            dst.copy_(w.x)
        stop.record()
        torch.cuda.synchronize()
        c_ms = start.elapsed_time(stop) / reps
        line["copy_probe"] = {"bytes_read": w.in_bytes, "bytes_written": w.in_bytes, "ms": round(c_ms, 4),
                              "GB/s": round(2 * w.in_bytes / (c_ms * 1e-3) / 1e9, 1)}
        del dst

    if not args.no_cpu_baseline and not w.flops:
        line["cpu_baseline"] = cpu_baseline(w)

    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
