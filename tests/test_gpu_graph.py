"""The library's calls captured in a HIP graph: every replay must equal the
eager call, with eager work (clobbering the outputs) and synchronisations
between replays.  No kernel of the library clears memory with a memset
node; the kernels reset their own counters."""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, profk as oprofk
from gpu_util import compare, gpu_bf16, gpu_f32, note, oracle_plan_of, torch

pytestmark = pytest.mark.gpu


def _replays_equal_eager(call, outs, reps=3):
    t = torch()
    ref = [o.clone() for o in outs]
    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(side):
        call()                       # warm-up on the capture stream
    t.cuda.current_stream().wait_stream(side)
    t.cuda.synchronize()
    g = t.cuda.CUDAGraph()
    with t.cuda.graph(g):
        call()
    for rep in range(reps):
        for o in outs:
            o.fill_(-7 if o.dtype == t.int64 else 0)   # eager work between replays
        t.cuda.synchronize()
        g.replay()
        t.cuda.synchronize()
        for a, b in zip(outs, ref):
            assert t.equal(a, b), f"replay {rep} differs from the eager call"


def test_graph_batchtopk_big_k():
    t = torch()
    B, D, k_row = 64, 4096, 32
    x = workloads.sae_preacts_f32(B=B, D=D, seed=4)
    p = pk.plan(B * D, B * k_row)
    note(f"graph batchtopk B={B} D={D} K={B * k_row} S={p.S} t={p.t} M={p.M}")
    g = gpu_f32(x.reshape(-1)).view(B, D)
    ws = pk.workspace(p, pk.F32)
    out = (t.empty(B * k_row, dtype=t.float32, device="cuda"),
           t.empty(B * k_row, dtype=t.int64, device="cuda"))
    info = t.empty(pk.INFO_BYTES, dtype=t.uint8, device="cuda")
    call = lambda: pk.batchtopk(g, k_row, seed=0, p=p, ws=ws, out=out, info=info)
    call()
    ref = oprofk.run_batchtopk(okeys.f32_bits(x.reshape(-1)).reshape(B, D), "f32", k_row,
                               oracle_plan_of(p), 0)
    compare(out[0], out[1], info, ref, "f32")
    _replays_equal_eager(call, [out[0], out[1], info])


@pytest.mark.parametrize("case", ["bucket", "radix"])
def test_graph_flat_k_above_4096(case):
    # k > 4096: the bucket refinement, and the radix refinement (whose first
    # two digit passes run in the scatter and sort launches), each inside the
    # capture; a plateau of 20000 equal keys at rank 3000 puts more
    # candidates in one bucket than the bucket path takes, so that the radix
    # path works (its plan, t = 164, also takes the capped sample lists)
    t = torch()
    if case == "bucket":
        x, k, eps = workloads.normal_f32(2**21 + 7, seed=21), 20000, 1e-6
    else:
        x, k, eps = workloads.plateau_f32(2**21, seed=5, first_rank=3000, width=20_000), 8000, 1e-3
    p = pk.plan(x.size, k, eps)
    note(f"graph flat {case} N={x.size} k={k} S={p.S} t={p.t} M={p.M}")
    g = gpu_f32(x)
    ws = pk.workspace(p, pk.F32)
    out = (t.empty(k, dtype=t.float32, device="cuda"), t.empty(k, dtype=t.int64, device="cuda"))
    info = t.empty(pk.INFO_BYTES, dtype=t.uint8, device="cuda")
    call = lambda: pk.topk(g, k, seed=1, p=p, ws=ws, out=out, info=info)
    call()
    ref = oprofk.run(okeys.f32_bits(x), "f32", k, oracle_plan_of(p), 1)
    compare(out[0], out[1], info, ref, "f32")
    _replays_equal_eager(call, [out[0], out[1], info])


def test_graph_flat_small_k():
    t = torch()
    x = workloads.normal_f32(2**20 + 3, seed=5)
    p = pk.plan(x.size, 64)
    note(f"graph flat N={x.size} k=64")
    g = gpu_f32(x)
    ws = pk.workspace(p, pk.F32)
    out = (t.empty(64, dtype=t.float32, device="cuda"), t.empty(64, dtype=t.int64, device="cuda"))
    info = t.empty(pk.INFO_BYTES, dtype=t.uint8, device="cuda")
    call = lambda: pk.topk(g, 64, seed=1, p=p, ws=ws, out=out, info=info)
    call()
    _replays_equal_eager(call, [out[0], out[1], info])


def test_graph_rows_bf16():
    t = torch()
    B, D, k = 32, 8192, 16
    bits = workloads.relu_normal_bf16((B, D), seed=6)
    note(f"graph rows bf16 B={B} D={D} k={k}")
    g = gpu_bf16(bits.reshape(-1)).view(B, D)
    p = pk.plan_rows(D, k)
    ws = pk.workspace(p, pk.BF16, B)
    out = (t.empty((B, k), dtype=t.bfloat16, device="cuda"), t.empty((B, k), dtype=t.int64, device="cuda"))
    info = t.empty(B * pk.INFO_BYTES, dtype=t.uint8, device="cuda")
    call = lambda: pk.topk_rows(g, k, seed=2, p=p, ws=ws, out=out, info=info)
    call()
    _replays_equal_eager(call, [out[0].view(t.int16), out[1], info])


def test_graph_sae_encode_topk():
    # the fused SAE layer: sample, tau, thresholds, the GEMM with the filter
    # in its epilogue, the fallback check and the refinement, all captured
    t = torch()
    B, d_model, d_dict, k_row = 512, 128, 2048, 16
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=29)
    bf = lambda a: t.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(t.bfloat16)
    x, w, b = bf(m["x"]), bf(m["w_enc"]), t.from_numpy(m["b_enc"]).cuda()
    p = pk.plan_sae(B, d_dict, k_row)
    note(f"graph sae B={B} d_model={d_model} d_dict={d_dict} K={B * k_row} S={p.S} t={p.t} M={p.M}")
    ws = pk.sae_workspace(p, B, d_dict)
    out = (t.empty(B * k_row, dtype=t.float32, device="cuda"),
           t.empty(B * k_row, dtype=t.int64, device="cuda"))
    info = t.empty(pk.INFO_BYTES, dtype=t.uint8, device="cuda")
    call = lambda: pk.sae_encode_topk(x, w, b, k_row, seed=0, p=p, ws=ws, out=out, info=info)
    call()
    assert int(pk.read_info(info)[0]["status"]) == 0
    _replays_equal_eager(call, [out[0], out[1], info])
