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
around the launch on its own stream; `read_probe` times the library's
read-only stream over the same bytes; `cpu_baseline` times the CPU oracle:
its Prof-K stages on the whole input with the filter split over the host
threads (O2), and the exact stable-sort top-k on a bounded prefix (O1).
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
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2608_12573_amd", "csrc")
WORKLOADS = ("c2", "c1", "c3a", "c3b", "c3c", "c3d", "c3d2", "c4", "c5", "c5r", "c5p", "sae")
MFMA_BF16_PEAK_TFLOPS = 2500.0
FLUSH_BYTES = 512 << 20

# The dominant kernel of each workload family: the name it has in rocprofv3
# output, and every source it is compiled from (committed counters stand
# for this exact code and are dropped once any of these changes).
KERNELS = {
    "filter": {"match": "k_filter<0, false,", "what": "profk::k_filter<0, false, U> (fp32 filter-and-compact)",
               "sources": ("kernels_filter.hip", "filter_tile.h", "device_common.h", "launch.h")},
    "rows": {"match": "k_rows<1, false>", "what": "profk::k_rows<1, false> (bf16 per-row Prof-K, one workgroup per row)",
             "sources": ("kernels_rows.hip", "filter_tile.h", "topk_block.h", "device_common.h", "launch.h")},
    "sae": {"match": "k_sae_filter", "what": "profk::k_sae_filter (bf16 MFMA encoder GEMM + filter epilogue)",
            "sources": ("kernels_sae.hip", "sample_union.h", "device_common.h", "launch.h")},
}


def kernel_family(workload):
    return "rows" if workload == "c4" else "sae" if workload == "sae" else "filter"


def counters_path(workload_key):
    return os.path.join(PROFILES, f"counters_{workload_key}.json")


def source_sha256(family):
    h = hashlib.sha256()
    for name in KERNELS[family]["sources"]:
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


def counters_traffic(workload_key, family):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 counter summary of this workload, or None when there is none
    or the kernel's sources changed since it was taken."""
    try:
        with open(counters_path(workload_key)) as f:
            c = json.load(f)
        sha = source_sha256(family)
    except OSError:
        return None
    if c.get("kernel_source_sha256") != sha:
        return None
    return c.get("traffic_bytes_per_launch")


def write_counters(fetch_dir, write_dir, bench_json):
    """profiles/counters_<workload>.json from two rocprofv3 --pmc runs of one
    bench.py workload (FETCH_SIZE with TA_FLAT_ATOMIC_WAVEFRONTS_sum, then
    WRITE_SIZE with TCC_ATOMIC_sum) and the JSON line one of them printed.
    The byte counters' units are calibrated on the device copy bench.py's
    copy probe makes in the same runs."""
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
        # the median dispatch: one launch of the same kernel and grid but
        # another size (a small staging copy among the copy probe's) does
        # not move it
        return {key: (sorted(v)[len(v) // 2], len(v)) for key, v in kern.items()}

    with open(bench_json) as fh:
        line = json.loads(fh.read().strip().splitlines()[-1])
    wl = line["config"]["workload_key"]
    family = kernel_family(wl.split("-")[0])
    spec = KERNELS[family]
    fetch, write = per_dispatch(fetch_dir, "FETCH_SIZE"), per_dispatch(write_dir, "WRITE_SIZE")
    atom_w = per_dispatch(fetch_dir, "TA_FLAT_ATOMIC_WAVEFRONTS_sum")
    atom_l2 = per_dispatch(write_dir, "TCC_ATOMIC_sum")

    def pick(table, pred, biggest=False):
        keys = [key for key in table if pred(key[0])]
        if not keys:
            sys.exit("kernel not found in the counter files")
        return max(keys, key=lambda key: table[key][0]) if biggest else keys[0]

    is_kernel = lambda n: spec["match"] in n
    is_copy = lambda n: "copyBuffer" in n
    fk, ck = pick(fetch, is_kernel), pick(fetch, is_copy, biggest=True)
    wk, cwk = pick(write, is_kernel), pick(write, is_copy, biggest=True)
    copy_bytes = line["copy_probe"]["bytes_read"]
    fpu, wpu = copy_bytes / fetch[ck][0], copy_bytes / write[cwk][0]
    fb, wb = fetch[fk][0] * fpu, write[wk][0] * wpu
    algo = line["roofline"].get("algorithmic_bytes_per_launch")
    base = "python bench.py --workload {} --steps 3 --warmup 1 --no-cpu-baseline --no-torch-baseline --no-read-probe"
    wl_args = base.format(wl.split("-")[0]) + (f" --k {line['config']['k']}" if wl.startswith("c2") else "")
    out = {
        "kernel": spec["what"],
        "workload_key": wl,
        "workload": line["config"]["workload"] + f"; {line['count']} survivors",
        "commands": [
            f"rocprofv3 --pmc FETCH_SIZE TA_FLAT_ATOMIC_WAVEFRONTS_sum -d {fetch_dir} -o fetch --output-format csv -- "
            + wl_args,
            f"rocprofv3 --pmc WRITE_SIZE TCC_ATOMIC_sum -d {write_dir} -o write --output-format csv -- " + wl_args,
            f"python bench.py --write-counters {fetch_dir} {write_dir} <the JSON line the first run printed>",
        ],
        "fetch_size_kib_per_dispatch": round(fetch[fk][0], 2),
        "write_size_kib_per_dispatch": round(write[wk][0], 2),
        "dispatches": [fetch[fk][1], write[wk][1]],
        "calibration": {
            "kernel": "__amd_rocclr_copyBuffer (the copy probe: torch copy_ of a device buffer, in the same runs)",
            "bytes_read": copy_bytes, "bytes_written": copy_bytes,
            "fetch_size_kib": round(fetch[ck][0], 2), "write_size_kib": round(write[cwk][0], 2),
            "fetch_bytes_per_kib_unit": round(fpu, 3), "write_bytes_per_kib_unit": round(wpu, 3),
        },
        "fetch_bytes_per_launch": int(round(fb)),
        "write_bytes_per_launch": int(round(wb)),
        "traffic_bytes_per_launch": int(round(fb + wb)),
        "atomic_wave_instructions_per_launch": round(atom_w[pick(atom_w, is_kernel)][0], 1),
        "l2_atomic_requests_per_launch": round(atom_l2[pick(atom_l2, is_kernel)][0], 1),
        "kernel_source_sha256": source_sha256(family),
        "kernel_sources": list(spec["sources"]),
    }
    if algo:
        out["algorithmic_bytes_per_launch"] = algo
        out["traffic_over_algorithmic"] = round((fb + wb) / algo, 5)
    with open(counters_path(wl), "w") as fh:
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


def _o2_flat(bits, dtype, k, plan, seed, workers):
    """The oracle's Prof-K stages on one vector, with stage 3 (the filter)
    split into `workers` contiguous chunks run on a thread pool: sample
    (oracle.philox), threshold (oracle.profk.threshold), survivors per chunk
    (oracle.keys.keys_of, key >= tau), then the status and the sorted top-k
    of the survivors (or O1 on a failure), as oracle.profk.run composes them.
    Returns (indices, count, tau)."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import exact, keys, philox, profk
    n = bits.size
    sidx = philox.sample_indices(seed, 0, plan.S, n)
    tau = profk.threshold(keys.keys_of(bits[sidx], dtype), plan.t)
    bounds = np.linspace(0, n, workers + 1).astype(np.int64)

    def part(c):
        lo, hi = int(bounds[c]), int(bounds[c + 1])
        return np.flatnonzero(keys.keys_of(bits[lo:hi], dtype) >= tau) + lo

    with ThreadPoolExecutor(workers) as ex:
        surv = np.concatenate(list(ex.map(part, range(workers))))
    count = int(surv.size)
    if count < plan.k_req or count > plan.M:
        return exact.topk(bits, dtype, k)[1], count, tau
    order = surv[np.argsort(-keys.keys_of(bits[surv], dtype), kind="stable")]
    return order[:k].astype(np.int64), count, tau


def cpu_baseline(w, gpu_idx, budget_s=10.0):
    """The oracle timed on the host.

    O2 (the reported value): the CPU Prof-K of oracle.profk on the whole
    workload, with its filter stage split over the host threads (for the
    per-row batch: 256 rows, one oracle.profk.run per row on the same pool),
    the sample seed of the GPU steps; its indices are compared with the GPU
    result.  O1: the exact top-k by a full stable sort (oracle.exact) on one
    thread, on a bounded prefix (2^24 values or 128 rows)."""
    sys.path.insert(0, ROOT)
    from concurrent.futures import ThreadPoolExecutor
    from oracle import exact, keys, plan as oplan, profk
    host_cpus = os.cpu_count() or 1
    workers = max(1, min(host_cpus, int(os.environ.get("OMP_NUM_THREADS") or host_cpus)))
    dt = "bf16" if w.es == 2 else "f32"
    out = {"kind": "oracle", "unit": "GB/s", "cores": workers, "host_cpu_count": host_cpus}
    if w.lex:
        out.update(value=None, sample="O2 not timed for the lexicographic rule")
    elif w.rows:
        R = 256
        bits = w.host[:R]
        q = oplan.plan_rows(w.D, w.k)
        t0 = time.perf_counter()
        with ThreadPoolExecutor(workers) as ex:
            res = list(ex.map(lambda r: profk.run(bits[r], dt, w.k, q, 0, row=r), range(R)))
        el = time.perf_counter() - t0
        same = all(np.array_equal(res[r].idx, gpu_idx[r]) for r in range(R))
        out.update(value=round(R * w.D * w.es / el / 1e9, 4),
                   sample=(f"O2: oracle.profk.run on the first {R} of the {w.B} rows, one row per task on "
                           f"{workers} threads, {el:.2f} s"),
                   elements_per_s=round(R * w.D / el, 1), matches_gpu=bool(same))
    else:
        bits = keys.f32_bits(w.host) if dt == "f32" else w.host
        q = oplan.plan(w.N, w.k, 1e-6, w.recall)
        reps, t0 = 0, time.perf_counter()
        while True:
            idx, count, tau = _o2_flat(bits, dt, w.k, q, 0, workers)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s or reps >= 3:
                break
        per = el / reps
        n_valid = min(w.k, count) if count >= q.k_req else w.k
        same = bool(np.array_equal(idx[:n_valid], gpu_idx[:n_valid]))
        out.update(value=round(w.N * w.es / per / 1e9, 4),
                   sample=(f"O2: oracle Prof-K stages on all {w.N} values, filter split over {workers} threads, "
                           f"{reps} runs, {per:.2f} s each ({count} survivors)"),
                   elements_per_s=round(w.N / per, 1), matches_gpu=same)
    # O1 on one thread, bounded
    if w.rows:
        R = 128
        b1 = w.host[:R]
        run = lambda: exact.topk_rows(b1, dt, w.k)
        n_s, what = R * w.D, f"oracle.exact.topk_rows on the first {R} of the {w.B} rows"
    else:
        n_s = min(w.N, 2**24)
        b1 = keys.f32_bits(w.host[:n_s]) if dt == "f32" else w.host[:n_s]
        kk = min(w.k, n_s)
        run = lambda: exact.topk(b1, dt, kk)
        what = f"oracle.exact.topk on the first 2^{n_s.bit_length() - 1} of the {w.N} values, k={kk}"
    reps, t0 = 0, time.perf_counter()
    while True:
        run()
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    per = el / reps
    out["o1"] = {"value": round(n_s * w.es / per / 1e9, 4), "unit": "GB/s", "cores": 1,
                 "sample": f"{what} (numpy stable argsort, one thread), {reps} runs, {per * 1e3:.0f} ms each",
                 "elements_per_s": round(n_s / per, 1)}
    return out


def read_probe(pk, torch, x, per_cu, loads, reps=10):
    """The library's read-only stream probe over x's bytes: (ms, GB/s)."""
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = torch.empty(1024, dtype=torch.int32, device=x.device)
    for _ in range(2):
        pk.debug_read_probe(x, per_cu, loads, out=out)
    torch.cuda.synchronize()
    start.record()
    for _ in range(reps):
        pk.debug_read_probe(x, per_cu, loads, out=out)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / reps
    return ms, x.numel() * x.element_size() / (ms * 1e-3) / 1e9


def graph_leg(w, torch, steps, warmup):
    """The same step captured once in a HIP graph and replayed: per-step time
    without the host's launch overhead between the kernels, and whether every
    replay left the eager step's outputs (values, indices, reports)."""
    outs = [w.out[0], w.out[1], w.info]
    ref = [o.clone() for o in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        w.step()  # the capture stream's first use, outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        w.step()
    for o in outs:  # eager work between the capture and the replays
        o.fill_(-7 if o.dtype == torch.int64 else 0)
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    equal = all(bool(torch.equal(a, b)) for a, b in zip(outs, ref))
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        g.replay()
    stop.record()
    torch.cuda.synchronize()
    equal = equal and all(bool(torch.equal(a, b)) for a, b in zip(outs, ref))
    del g
    return start.elapsed_time(stop) / steps, equal


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
    ap.add_argument("--no-read-probe", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the graph-replay leg (the step captured once in a HIP graph)")
    ap.add_argument("--lexicographic", action="store_true",
                    help="plan with the tie-exact filter rule on (key, -index) pairs")
    ap.add_argument("--write-counters", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "BENCH_JSON"),
                    help="write profiles/counters_<workload>.json from two rocprofv3 --pmc runs of one workload and exit")
    args = ap.parse_args()
    if args.write_counters:
        write_counters(*args.write_counters)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
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
                    "traffic": counters_traffic(w.key(), kernel_family(w.name)), "kernel": w.kernel,
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
        "config": {"workload": w.desc, "workload_key": w.key(), "N": w.N, "k": w.k, "eps": 1e-6, "recall": w.recall,
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

    if not args.no_graph:
        g_ms, g_equal = graph_leg(w, torch, args.steps, max(5, args.warmup))
        line["graph"] = {"what": "the same step captured once in a HIP graph and replayed",
                         "ms_per_step": round(g_ms, 5), "value": round(w.in_bytes / (g_ms * 1e-3) / 1e9, 2),
                         "outputs_equal_eager": g_equal}

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

    if not args.no_copy_probe:
        # A plain device-to-device copy of the input (of the latent buffer
        # for the SAE layer, whose input is small): the reference kernel that
        # scales the FETCH_SIZE / WRITE_SIZE counters into bytes.
        src = w.dense if w.flops else w.x
        src_bytes = src.numel() * src.element_size()
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        reps = 5
        start.record()
        for _ in range(reps):
            dst.copy_(src)
        stop.record()
        torch.cuda.synchronize()
        c_ms = start.elapsed_time(stop) / reps
        line["copy_probe"] = {"bytes_read": src_bytes, "bytes_written": src_bytes, "ms": round(c_ms, 4),
                              "GB/s": round(2 * src_bytes / (c_ms * 1e-3) / 1e9, 1)}
        del dst

    if not args.no_read_probe and not w.flops and (w.in_bytes % 16 == 0):
        # The library's read-only stream with the filter's access pattern:
        # the practical ceiling of a single read of the input.  First the
        # launch shape the filter uses for this size, then the best of a
        # small sweep.
        big = w.in_bytes >= (512 << 20)
        shape = (2, 4) if big else (4, 8)
        ms, gbps = read_probe(pk, torch, w.x, *shape)
        sweep = {f"{pc}x{u}": round(read_probe(pk, torch, w.x, pc, u)[1], 1)
                 for pc in (1, 2, 4) for u in (4, 8)}
        line["read_probe"] = {"bytes_read": w.in_bytes, "workgroups_per_cu": shape[0], "loads_per_lane": shape[1],
                              "ms": round(ms, 4), "GB/s": round(gbps, 1),
                              "sweep_GB/s (workgroups per CU x loads per lane)": sweep}

    if not args.no_cpu_baseline and not w.flops:
        line["cpu_baseline"] = cpu_baseline(w, w.out[1].cpu().numpy())

    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
