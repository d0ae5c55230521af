"""GPU parity of the per-row kernel on rows of 128 KiB to 256 KiB (bf16 D in
[65536, 131072], fp32 D in [32768, 65536]), row by row against the
oracle, bit-exact, with every row's threshold, count, status and n_valid.
Covers batches smaller and larger than the number of compute units and not
a multiple of it, unaligned and strided rows, ragged widths, the
lexicographic rule, relaxed recall, per-row fallback, k from 1 to 1024 and
thresholds above the wave-level top-t limit."""

import dataclasses

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, plan as oplan, profk as oprofk
from gpu_util import check_rows, oracle_plan_of, plan_from_lib

pytestmark = pytest.mark.gpu


def _bits(dtype, B, D, seed):
    if dtype == "bf16":
        return workloads.relu_normal_bf16((B, D), seed=seed)
    return okeys.f32_bits(workloads.normal_f32(B * D, seed=seed)).reshape(B, D)


def _row_kernel_plan(p, dtype, D):
    """The plan runs the one-workgroup row kernel (no vector workspace) with
    a sample of at most 2048 draws, rows of 128-256 KiB."""
    es = 4 if dtype == "f32" else 2
    return (p.mode == pk.MODE_FILTER and p.S <= 2048 and p.k <= 1024 and 128 * 1024 <= D * es <= 256 * 1024
            and pk.workspace_size(p, pk.F32 if dtype == "f32" else pk.BF16, 2) == 256)


@pytest.mark.parametrize("dtype,D", [("bf16", 131072), ("bf16", 65536), ("bf16", 100_003), ("f32", 65536),
                                     ("f32", 32768), ("f32", 50_001)])
@pytest.mark.parametrize("B", [7, 300])
def test_register_rows_widths_and_batches(dtype, D, B):
    b = _bits(dtype, B, D, seed=D % 997 + B)
    p = pk.plan_rows(D, 32)
    assert _row_kernel_plan(p, dtype, D)
    st = check_rows(b, dtype, 32, p, oracle_plan_of(p, rows=True), 1)
    assert st.count(oprofk.STATUS_FILTERED) >= B - 1


@pytest.mark.parametrize("offset,extra", [(1, 0), (3, 5), (0, 13)])
def test_register_rows_unaligned_and_strided(offset, extra):
    D = 131072
    b = _bits("bf16", 20, D, seed=41)
    p = pk.plan_rows(D, 16)
    check_rows(b, "bf16", 16, p, oracle_plan_of(p, rows=True), 2, offset=offset, stride=D + extra)


@pytest.mark.parametrize("k", [1, 100, 1024])
def test_register_rows_k(k):
    """k = 1024 plans more than 2048 draws by default: the sample is capped
    at 2048 here."""
    D = 131072
    b = _bits("bf16", 40, D, seed=42 + k)
    kw = dict(S_min=2048, S_max=2048) if k > 500 else {}
    p = pk.plan_rows(D, k, **kw)
    assert _row_kernel_plan(p, "bf16", D)
    q = oracle_plan_of(p, opts=dataclasses.replace(oplan.ROW_OPTS, **kw)) if kw else oracle_plan_of(p, rows=True)
    check_rows(b, "bf16", k, p, q, 3)


def test_register_rows_lexicographic():
    D = 131072
    b = _bits("bf16", 64, D, seed=43)
    p = pk.plan_rows(D, 32, lexicographic=1)
    assert _row_kernel_plan(p, "bf16", D)
    q = oracle_plan_of(p, opts=dataclasses.replace(oplan.ROW_OPTS, lexicographic=True))
    check_rows(b, "bf16", 32, p, q, 4)


def test_register_rows_fallback_and_relaxed():
    """All-equal rows overflow and fall back on their own; a forced low t
    with recall 0.5 gives rows in [k_req, k) (padded), rows below k_req
    (fallback) and exact rows, in one batch."""
    D = 131072
    b = _bits("bf16", 48, D, seed=44)
    b[5, :] = 0x3F80          # 1.0 everywhere
    b[17, :] = 0x0000         # +0.0 everywhere
    p = pk.plan_rows(D, 64, 1e-2, 0.5)
    p.t = 2
    q = plan_from_lib(p)
    st = check_rows(b, "bf16", 64, p, q, 5)
    assert st[5] == oprofk.STATUS_OVERFLOW and st[17] == oprofk.STATUS_OVERFLOW
    assert oprofk.STATUS_FILTERED in st


def test_register_rows_large_t_select():
    """t above the wave top-t limit: the threshold comes from the radix
    select over the sample in LDS."""
    D = 131072
    b = _bits("bf16", 24, D, seed=45)
    p = pk.plan_rows(D, 1000, S_min=2048, S_max=2048)
    assert p.t > 32 and _row_kernel_plan(p, "bf16", D)
    q = oracle_plan_of(p, opts=dataclasses.replace(oplan.ROW_OPTS, S_min=2048, S_max=2048))
    check_rows(b, "bf16", 1000, p, q, 6)
