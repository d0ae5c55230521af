"""GPU parity of the per-row path (profk_topk_rows) against the CPU oracle,
row by row, bit-exact, including each row's threshold, count and status."""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, plan as oplan, profk as oprofk
from gpu_util import check_rows as _check_rows, oracle_plan_of, plan_from_lib

pytestmark = pytest.mark.gpu


def _bits(dtype, B, D, seed):
    if dtype == "bf16":
        return workloads.relu_normal_bf16((B, D), seed=seed)
    return okeys.f32_bits(workloads.normal_f32(B * D, seed=seed)).reshape(B, D)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("D,k", [(4096, 1), (4096, 32), (4099, 7), (20_000, 100), (131072, 32)])
def test_rows_small_batches(dtype, D, k):
    b = _bits(dtype, 24, D, seed=D + k)
    p = pk.plan_rows(D, k, 1e-3, 1.0, S_min=512, S_max=512, force_mode=pk.FORCE_FILTER)
    q = oracle_plan_of(p, S_min=512, S_max=512, force_mode=oplan.FORCE_FILTER)
    for seed in (0, 3):
        _check_rows(b, dtype, k, p, q, seed)


@pytest.mark.parametrize("offset,extra", [(1, 0), (3, 5), (0, 13)])
def test_rows_unaligned_and_strided(offset, extra):
    b = _bits("bf16", 16, 30_001, seed=9)
    p = pk.plan_rows(30_001, 16)
    q = oracle_plan_of(p, rows=True)
    _check_rows(b, "bf16", 16, p, q, 1, offset=offset, stride=30_001 + extra)


def test_rows_fallback_per_row():
    b = _bits("f32", 32, 8192, seed=4)
    b[5, :] = okeys.f32_bits(np.full(8192, 1.5, np.float32))  # all ties: overflow
    p = pk.plan_rows(8192, 16, 1e-2, 1.0, S_min=256, S_max=256, force_mode=pk.FORCE_FILTER)
    p.M = 64
    q = plan_from_lib(p)
    st = _check_rows(b, "f32", 16, p, q, 0)
    assert oprofk.STATUS_OVERFLOW in st


def test_rows_direct_mode():
    b = _bits("bf16", 12, 300, seed=5)
    p = pk.plan_rows(300, 20)
    assert p.mode == pk.MODE_DIRECT
    q = oracle_plan_of(p, rows=True)
    st = _check_rows(b, "bf16", 20, p, q, 0)
    assert set(st) == {oprofk.STATUS_DIRECT}


def test_rows_special_values():
    x = workloads.special_f32(16 * 5000, seed=8).reshape(16, 5000)
    b = okeys.f32_bits(x.reshape(-1)).reshape(16, 5000)
    p = pk.plan_rows(5000, 50, 1e-3, 1.0, S_min=600, S_max=600, force_mode=pk.FORCE_FILTER)
    q = oracle_plan_of(p, S_min=600, S_max=600, force_mode=oplan.FORCE_FILTER)
    _check_rows(b, "f32", 50, p, q, 2)


def test_rows_large_k():
    b = _bits("f32", 8, 65536, seed=6)
    p = pk.plan_rows(65536, 1024)
    q = oracle_plan_of(p, rows=True)
    _check_rows(b, "f32", 1024, p, q, 0)


def test_config4_bf16_4096x131072_k32():
    B, D, k = 4096, 131072, 32
    b = workloads.relu_normal_bf16((B, D), seed=3)
    p = pk.plan_rows(D, k)
    q = oracle_plan_of(p, rows=True)
    st = _check_rows(b, "bf16", k, p, q, 0)
    assert st.count(oprofk.STATUS_FILTERED) >= B - 2


def test_rows_relaxed_recall_partial_rows():
    # recall 0.5 of k = 64 with t forced low: rows whose count falls in
    # [k_req, k) return their count survivors padded, rows below k_req fall
    # back, the rest are exact top-k
    b = _bits("f32", 64, 4096, seed=11)
    p = pk.plan_rows(4096, 64, 1e-2, 0.5, S_min=256, S_max=256, force_mode=pk.FORCE_FILTER)
    p.t = 3
    q = plan_from_lib(p)
    st = _check_rows(b, "f32", 64, p, q, 0)
    assert oprofk.STATUS_FILTERED in st
