"""Measured plan tuning (Sec. 4, "Optimal Sample Size").

The cost model C = tau_A S + tau_B M log k leaves the ratio tau_B / tau_A
to the hardware, to be estimated by a small benchmark.  Each ratio gives a
plan (S from Algorithm 1, t and M from the exact failure tails, so every
plan keeps the eps guarantee); `sweep_rows` / `sweep_flat` time the path
for a range of ratios on the caller's tensor, `fit` estimates tau_A and
tau_B from those times by least squares, and `best` picks the fastest plan.
The fit assumes the linear model; a larger M also lowers occupancy in steps
(LDS per workgroup), so the fastest measured plan is the better guide.

    python -m paper_2608_12573_amd.tune rows --B 4096 --D 131072 --k 32 --dtype bf16
    python -m paper_2608_12573_amd.tune flat --N 268435456 --k 1024 --dtype f32

The command line builds a synthetic input on the GPU (rows: bf16/fp32
max(N(0,1), 0) as in a ReLU SAE latent; flat: N(0,1)) and prints a table.
"""

import argparse
import json
import math

import numpy as np

from . import (BF16, F32, INFO_BYTES, MODE_FILTER, ProfkError, plan, plan_rows, topk, topk_rows,
               workspace)

RATIOS = (2.0, 1.0, 0.8, 0.65, 0.5, 0.4, 0.3, 0.2)


def _time_us(fn, iters, reps):
    import torch
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = math.inf
    for _ in range(reps):
        s.record()
        for _ in range(iters):
            fn()
        e.record()
        torch.cuda.synchronize()
        best = min(best, s.elapsed_time(e) / iters * 1e3)
    return best


def _dtype_code(x):
    import torch
    if x.dtype == torch.float32:
        return F32
    if x.dtype == torch.bfloat16:
        return BF16
    raise ProfkError("x must be float32 or bfloat16")


def sweep_rows(x, k, ratios=RATIOS, eps=1e-6, recall=1.0, iters=10, reps=3):
    """Time topk_rows on the [B, D] tensor x for each cost ratio.  Returns
    one dict per distinct filtering plan: ratio, S, t, M, us (best of reps)."""
    import torch
    B, D = x.shape
    dt = _dtype_code(x)
    out = (torch.empty((B, k), dtype=x.dtype, device=x.device),
           torch.empty((B, k), dtype=torch.int64, device=x.device))
    info = torch.empty(B * INFO_BYTES, dtype=torch.uint8, device=x.device)
    res, seen = [], set()
    for r in ratios:
        p = plan_rows(D, k, eps, recall, cost_ratio=r)
        if p.mode != MODE_FILTER or p.S in seen:
            continue
        seen.add(p.S)
        ws = workspace(p, dt, B, x.device)
        us = _time_us(lambda: topk_rows(x, k, p=p, ws=ws, out=out, info=info), iters, reps)
        res.append(dict(ratio=r, S=int(p.S), t=int(p.t), M=int(p.M), us=us))
    return res


def sweep_flat(x, k, ratios=RATIOS, eps=1e-6, recall=1.0, iters=10, reps=3, S_min=None):
    """Time topk on the 1-D tensor x for each cost ratio (S_min lowers the
    sample floor so that the ratio can move S at all)."""
    import torch
    N = x.numel()
    dt = _dtype_code(x)
    out = (torch.empty(k, dtype=x.dtype, device=x.device),
           torch.empty(k, dtype=torch.int64, device=x.device))
    info = torch.empty(INFO_BYTES, dtype=torch.uint8, device=x.device)
    kw = {} if S_min is None else dict(S_min=S_min)
    res, seen = [], set()
    for r in ratios:
        p = plan(N, k, eps, recall, cost_ratio=r, **kw)
        if p.mode != MODE_FILTER or p.S in seen:
            continue
        seen.add(p.S)
        ws = workspace(p, dt, 1, x.device)
        us = _time_us(lambda: topk(x, k, p=p, ws=ws, out=out, info=info), iters, reps)
        res.append(dict(ratio=r, S=int(p.S), t=int(p.t), M=int(p.M), us=us))
    return res


def fit(res, k):
    """Least-squares fit of us = c + tau_A S + tau_B M log2 k over a sweep.
    Returns (c, tau_A, tau_B, tau_B / tau_A or None when a coefficient is
    not positive or the sweep has fewer than four plans)."""
    if len(res) < 4:
        return None
    A = np.array([[1.0, r["S"], r["M"] * math.log2(max(k, 2))] for r in res])
    y = np.array([r["us"] for r in res])
    (c, ta, tb), *_ = np.linalg.lstsq(A, y, rcond=None)
    ratio = tb / ta if ta > 0 and tb > 0 else None
    return float(c), float(ta), float(tb), (None if ratio is None else float(ratio))


def best(res):
    return min(res, key=lambda r: r["us"]) if res else None


def _table(res, k):
    lines = ["| tau_B/tau_A | S | t | M | us per call |", "|---|---|---|---|---|"]
    b = best(res)
    for r in res:
        mark = " **(best)**" if r is b else ""
        lines.append(f"| {r['ratio']:g} | {r['S']} | {r['t']} | {r['M']} | {r['us']:.1f}{mark} |")
    f = fit(res, k)
    if f is not None:
        c, ta, tb, ratio = f
        lines.append("")
        lines.append(f"least-squares fit: us = {c:.1f} + {ta:.4f} S + {tb:.5f} M log2 k"
                     + (f"  (tau_B/tau_A = {ratio:.2f})" if ratio is not None else ""))
    return "\n".join(lines)


def main(argv=None):
    import torch
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("mode", choices=("rows", "flat"))
    ap.add_argument("--B", type=int, default=4096)
    ap.add_argument("--D", type=int, default=131072)
    ap.add_argument("--N", type=int, default=1 << 28)
    ap.add_argument("--k", type=int, default=32)
    ap.add_argument("--dtype", choices=("f32", "bf16"), default="bf16")
    ap.add_argument("--eps", type=float, default=1e-6)
    ap.add_argument("--recall", type=float, default=1.0)
    ap.add_argument("--ratios", type=str, default=",".join(f"{r:g}" for r in RATIOS))
    ap.add_argument("--S-min", type=int, default=None, help="flat: lower the sample floor")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--json", action="store_true")
    a = ap.parse_args(argv)
    dtype = torch.bfloat16 if a.dtype == "bf16" else torch.float32
    ratios = tuple(float(s) for s in a.ratios.split(","))
    g = torch.Generator(device="cuda").manual_seed(a.seed)
    if a.mode == "rows":
        x = torch.randn((a.B, a.D), generator=g, device="cuda").clamp_min_(0.0).to(dtype)
        res = sweep_rows(x, a.k, ratios, a.eps, a.recall)
        what = f"rows [{a.B}, {a.D}] {a.dtype}, k = {a.k}"
    else:
        x = torch.randn(a.N, generator=g, device="cuda").to(dtype)
        res = sweep_flat(x, a.k, ratios, a.eps, a.recall, S_min=a.S_min)
        what = f"flat N = {a.N} {a.dtype}, k = {a.k}"
    if a.json:
        print(json.dumps(dict(workload=what, sweep=res, best=best(res), fit=fit(res, a.k))))
    else:
        print(f"plan sweep, {what}, eps = {a.eps:g}, recall = {a.recall:g}\n")
        print(_table(res, a.k))
        b = best(res)
        if b is not None:
            print(f"\nfastest: tau_B/tau_A = {b['ratio']:g} (S = {b['S']}, t = {b['t']}, M = {b['M']}), "
                  f"{b['us']:.1f} us")


if __name__ == "__main__":
    main()
