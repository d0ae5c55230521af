"""GPU parity of the multi-block refinement (k > 4096) against the CPU
oracle: the BatchTopK workload, relaxed recall, forced fallbacks, ties."""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, plan as oplan, profk as oprofk
from gpu_util import (compare, gpu_bf16, gpu_f32, host_bits, note, oracle_plan_of,
                      plan_from_lib, torch)

pytestmark = pytest.mark.gpu


def _f32(x, k, seed, eps=1e-6, recall=1.0, **kw):
    p = pk.plan(x.size, k, eps, recall, **kw)
    q = oracle_plan_of(p, **kw)
    note(f"big f32 N={x.size} k={k} seed={seed} S={p.S} t={p.t} M={p.M} mode={p.mode}")
    vals, idx, info = pk.topk(gpu_f32(x), k, seed=seed, p=p)
    ref = oprofk.run(okeys.f32_bits(x), "f32", k, q, seed)
    return compare(vals, idx, info, ref, "f32"), ref


@pytest.mark.parametrize("k", [4097, 5000, 20000, 65536])
def test_big_k_normal(k):
    x = workloads.normal_f32(2**21 + 7, seed=21)
    rec, ref = _f32(x, k, 0)
    assert ref.status == oprofk.STATUS_FILTERED


def test_big_k_ties_cut_by_index():
    x = workloads.plateau_f32(2**21, seed=5, first_rank=3000, width=20_000)
    rec, ref = _f32(x, 8000, 1, eps=1e-3)


def test_big_k_bf16_ties():
    b = workloads.relu_normal_bf16(2**21, seed=22)
    p = pk.plan(b.size, 10000)
    q = oracle_plan_of(p)
    note("big bf16")
    vals, idx, info = pk.topk(gpu_bf16(b), 10000, seed=2, p=p)
    ref = oprofk.run(b, "bf16", 10000, q, 2)
    compare(vals, idx, info, ref, "bf16")


def test_big_k_direct():
    x = workloads.special_f32(40_000, seed=23)
    rec, ref = _f32(x, 6000, 0)
    assert ref.status == oprofk.STATUS_DIRECT


@pytest.mark.parametrize("which", ["max", "min"])
def test_big_k_forced_fallback(which):
    x = workloads.uniform_f32(2**20, seed=24)
    bits = okeys.f32_bits(x)
    key = okeys.key_u32(bits).astype(np.int64)
    k = 10000
    p = pk.plan(x.size, k, 1e-6, 1.0, S_min=8192, S_max=8192, force_mode=pk.FORCE_FILTER)
    q = plan_from_lib(p)
    tau = int(key.max()) if which == "max" else int(key.min())
    note(f"big topk_tau {which}")
    vals, idx, info = pk.topk_tau(gpu_f32(x), k, tau, p)
    ref = oprofk.run(bits, "f32", k, q, 0, tau_override=tau)
    assert ref.status in (oprofk.STATUS_UNDERFLOW, oprofk.STATUS_OVERFLOW)
    compare(vals, idx, info, ref, "f32")


def test_big_k_relaxed_partial_output():
    x = workloads.normal_f32(2**20, seed=25)
    bits = okeys.f32_bits(x)
    key = np.sort(okeys.key_u32(bits).astype(np.int64))
    k = 20000
    p = pk.plan(x.size, k, 1e-3, 0.9, S_min=8192, S_max=8192, force_mode=pk.FORCE_FILTER)
    q = plan_from_lib(p)
    tau = int(key[-19000])                       # 19000 survivors: k_req <= count < k
    note("big relaxed partial")
    vals, idx, info = pk.topk_tau(gpu_f32(x), k, tau, p)
    ref = oprofk.run(bits, "f32", k, q, 0, tau_override=tau)
    assert ref.status == oprofk.STATUS_FILTERED and ref.n_valid == 19000
    compare(vals, idx, info, ref, "f32")


def test_batchtopk_small():
    x = workloads.sae_preacts_f32(B=64, D=4096, seed=4)
    p = pk.plan(64 * 4096, 64 * 32)
    q = oracle_plan_of(p)
    note("batchtopk small")
    vals, idx, info = pk.batchtopk(gpu_f32(x.reshape(-1)).view(64, 4096), 32, seed=0, p=p)
    ref = oprofk.run_batchtopk(okeys.f32_bits(x.reshape(-1)).reshape(64, 4096), "f32", 32, q, 0)
    compare(vals, idx, info, ref, "f32")


@pytest.mark.parametrize("recall", [1.0, 0.95])
def test_config5_batchtopk_4096x65536(recall):
    B, D, k_row = 4096, 65536, 64
    x = workloads.sae_preacts_f32(B=B, D=D, seed=4)
    p = pk.plan(B * D, B * k_row, 1e-6, recall)
    q = oracle_plan_of(p)
    note(f"config5 recall={recall} S={p.S} t={p.t} M={p.M}")
    g = gpu_f32(x.reshape(-1)).view(B, D)
    vals, idx, info = pk.batchtopk(g, k_row, seed=0, p=p)
    ref = oprofk.run_batchtopk(okeys.f32_bits(x.reshape(-1)).reshape(B, D), "f32", k_row, q, 0)
    compare(vals, idx, info, ref, "f32")
    assert ref.status == oprofk.STATUS_FILTERED
