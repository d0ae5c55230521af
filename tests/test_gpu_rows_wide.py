"""GPU parity of profk_topk_rows for row plans outside the one-workgroup
row kernel's envelope (k > 1024, or a sample and buffer beyond its LDS):
those rows run the vector path one row after another, each with its own
Philox stream (counter word 1 = row), and must equal the oracle row by row,
bit-exact, with every row's threshold, count, status and n_valid."""

import dataclasses

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, plan as oplan, profk as oprofk
from gpu_util import check_rows, oracle_plan_of

pytestmark = pytest.mark.gpu


def _bits(dtype, B, D, seed):
    if dtype == "bf16":
        return workloads.relu_normal_bf16((B, D), seed=seed)
    return okeys.f32_bits(workloads.normal_f32(B * D, seed=seed)).reshape(B, D)


def _wide(p, dtype, B):
    """The plan is outside the row kernel's envelope: the library asks for
    a real workspace instead of the row kernel's token 256 bytes."""
    return pk.workspace_size(p, pk.F32 if dtype == "f32" else pk.BF16, B) > 256


@pytest.mark.parametrize("seed", [0, 5])
def test_wide_rows_fp32_D2p22_k32(seed):
    B, D, k = 8, 2**22, 32
    b = _bits("f32", B, D, seed=31)
    p = pk.plan_rows(D, k)
    assert _wide(p, "f32", B) and p.M > 32768
    st = check_rows(b, "f32", k, p, oracle_plan_of(p, rows=True), seed)
    assert st.count(oprofk.STATUS_FILTERED) >= B - 1


def test_wide_rows_bf16_k2048():
    B, D, k = 16, 65536, 2048
    b = _bits("bf16", B, D, seed=32)
    p = pk.plan_rows(D, k)
    assert _wide(p, "bf16", B)
    check_rows(b, "bf16", k, p, oracle_plan_of(p, rows=True), 1)


def test_wide_rows_bf16_ragged_strided_unaligned():
    """Odd width, odd row stride (so row starts are not 16-byte aligned) and
    a base offset, on rows far wider than the row kernel holds."""
    B, D, k = 3, 2**23 + 5, 48
    b = _bits("bf16", B, D, seed=33)
    p = pk.plan_rows(D, k)
    assert _wide(p, "bf16", B)
    check_rows(b, "bf16", k, p, oracle_plan_of(p, rows=True), 2, offset=1, stride=D + 3)


def test_wide_rows_relaxed_recall():
    B, D, k = 4, 2**20, 2000
    b = _bits("f32", B, D, seed=34)
    p = pk.plan_rows(D, k, 1e-6, 0.9)
    assert _wide(p, "f32", B) and p.k_req == 1800
    check_rows(b, "f32", k, p, oracle_plan_of(p, rows=True), 3)


def test_wide_rows_lexicographic_with_ties():
    """bf16 ReLU rows: half the values are +0.0 and the rest repeat often,
    so the threshold pair usually sits inside a tie class."""
    B, D, k = 4, 65536, 1500
    b = _bits("bf16", B, D, seed=35)
    p = pk.plan_rows(D, k, lexicographic=1)
    assert _wide(p, "bf16", B) and p.lexicographic
    q = oracle_plan_of(p, opts=dataclasses.replace(oplan.ROW_OPTS, lexicographic=True))
    check_rows(b, "bf16", k, p, q, 4)


def test_wide_rows_direct_mode():
    B, D, k = 3, 20000, 3000
    b = _bits("f32", B, D, seed=36)
    p = pk.plan_rows(D, k)
    assert p.mode == pk.MODE_DIRECT and _wide(p, "f32", B)
    st = check_rows(b, "f32", k, p, oracle_plan_of(p, rows=True), 0)
    assert set(st) == {oprofk.STATUS_DIRECT}


@pytest.mark.parametrize("k", [1024, 1025])
def test_rows_either_side_of_the_k_limit(k):
    """k = 1024 runs the row kernel, k = 1025 the vector path per row; both
    give the oracle's rows."""
    B, D = 6, 131072
    b = _bits("bf16", B, D, seed=37)
    p = pk.plan_rows(D, k)
    assert _wide(p, "bf16", B) == (k > 1024)
    check_rows(b, "bf16", k, p, oracle_plan_of(p, rows=True), 6)


def test_wide_rows_overflow_fallback_per_row():
    """One row of all-equal values overflows the buffer and falls back on
    its own; the others are filtered."""
    B, D, k = 4, 2**21, 1100
    b = _bits("f32", B, D, seed=38)
    b[2, :] = okeys.f32_bits(np.full(D, 0.75, np.float32))
    p = pk.plan_rows(D, k)
    assert _wide(p, "f32", B)
    st = check_rows(b, "f32", k, p, oracle_plan_of(p, rows=True), 7)
    assert st[2] == oprofk.STATUS_OVERFLOW and st.count(oprofk.STATUS_FILTERED) >= 2
