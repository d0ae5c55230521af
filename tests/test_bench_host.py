"""Host-side pieces of bench.py: the CPU baseline's O2 (the oracle's Prof-K
stages with the filter split over threads) gives oracle.profk.run's result,
so the time it reports is the oracle's."""

import numpy as np
import pytest

import bench
import workloads
from oracle import keys, plan as oplan, profk


@pytest.mark.parametrize("workers", [1, 3, 8])
@pytest.mark.parametrize("case", ["filtered", "relaxed", "fallback"])
def test_o2_threaded_equals_oracle_run(case, workers):
    n, k = 2**20 + 3, 64
    x = workloads.normal_f32(n, seed=40)
    recall = 0.5 if case == "relaxed" else 1.0
    q = oplan.plan(n, k, 1e-6, recall)
    if case == "fallback":
        x[:] = 2.0   # all ties: count = n > M
    if case == "relaxed":
        q = oplan.Plan(**{**q.__dict__, "t": 1})   # a high tau: fewer than k survive
    bits = keys.f32_bits(x)
    idx, count, tau = bench._o2_flat(bits, "f32", k, q, 7, workers)
    ref = profk.run(bits, "f32", k, q, 7)
    assert count == ref.count and tau == ref.tau_key
    assert np.array_equal(idx, ref.idx[:idx.size])
    assert np.all(ref.idx[idx.size:] == -1)
    if case == "fallback":
        assert ref.status == profk.STATUS_OVERFLOW and np.array_equal(idx, np.arange(k))
