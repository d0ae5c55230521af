"""Pins for O2 (oracle.profk): the stage-by-stage CPU Prof-K.

Checks the paper's invariants (Sec. 3 design goal and refinement rule) and
reduces special cases to independently computed results: brute-force
comparators on float semantics, float max of the sample, O1.
"""

import functools

import numpy as np
import pytest

from oracle import exact, keys, philox, plan, profk
import workloads

SMALL = plan.PlanOpts(S_min=48, S_max=48, force_mode=plan.FORCE_FILTER)


def _brute_order(x):
    def cmp(i, j):
        a, b = float(x[i]), float(x[j])
        if a != b:
            return -1 if a > b else 1
        return -1 if i < j else (1 if i > j else 0)
    return sorted(range(len(x)), key=functools.cmp_to_key(cmp))


@pytest.mark.parametrize("seed", range(40))
def test_filtered_result_equals_brute_force(seed):
    g = np.random.default_rng(seed)
    n = int(g.integers(60, 400))
    x = g.integers(1, 40, n).astype(np.float32)   # positive, many ties
    k = int(g.integers(1, 12))
    p = plan.plan(n, k, 0.2, 1.0, SMALL)
    r = profk.run(keys.f32_bits(x), "f32", k, p, seed)
    order = _brute_order(x)
    assert list(r.idx) == order[:k]
    tau_val = keys.bits_from_key_u32(np.uint32(r.tau_key)).view(np.float32)
    assert r.count == int(np.sum(x >= tau_val))
    if r.status == profk.STATUS_FILTERED:
        assert k <= r.count <= p.M
        # I4: every true top-k element survived the filter
        assert np.all(x[order[:k]] >= tau_val)
    else:
        assert (r.count < p.k_req) == (r.status == profk.STATUS_UNDERFLOW)
        assert (r.count > p.M) == (r.status == profk.STATUS_OVERFLOW)


def test_threshold_is_t_th_largest_sampled_value():
    x = workloads.normal_f32(5000, seed=4)
    for t in (1, 2, 7):
        p = plan.Plan(N=5000, k=5, eps=0.1, recall=1.0, k_req=5, S=100, t=t,
                      M=5000, mode=plan.MODE_FILTER, p_underflow=0, p_overflow=0)
        r = profk.run(keys.f32_bits(x), "f32", 5, p, seed=9)
        samp = x[philox.sample_indices(9, 0, 100, 5000)]
        expect = np.sort(samp.astype(np.float64))[::-1][t - 1]
        tau_val = keys.bits_from_key_u32(np.uint32(r.tau_key)).view(np.float32)
        assert float(tau_val) == expect
        if t == 1:
            assert float(tau_val) == float(samp.max())


def test_duplicate_draws_count_with_multiplicity():
    # N = 2 with many draws: the t-th largest of the multiset.
    x = np.array([1.0, 2.0], np.float32)
    p = plan.Plan(N=2, k=1, eps=0.1, recall=1.0, k_req=1, S=16, t=3, M=2,
                  mode=plan.MODE_FILTER, p_underflow=0, p_overflow=0)
    r = profk.run(keys.f32_bits(x), "f32", 1, p, seed=1)
    idx = philox.sample_indices(1, 0, 16, 2)
    n_hi = int(np.sum(idx == 1))
    expect = 2.0 if n_hi >= 3 else 1.0
    tau_val = keys.bits_from_key_u32(np.uint32(r.tau_key)).view(np.float32)
    assert float(tau_val) == expect


def test_forced_underflow_and_overflow_fall_back_to_exact():
    x = workloads.uniform_f32(20_000, seed=0)
    x[:5] = 7.0
    bits = keys.f32_bits(x)
    kk = keys.key_u32(bits)
    p = plan.plan(20_000, 64, 1e-6, 1.0, plan.PlanOpts(S_min=512, S_max=512,
                                                     force_mode=plan.FORCE_FILTER))
    o1v, o1i = exact.topk(bits, "f32", 64)
    r = profk.run(bits, "f32", 64, p, 0, tau_override=int(kk.max()))
    assert r.status == profk.STATUS_UNDERFLOW and r.count == 5
    assert np.array_equal(r.idx, o1i) and np.array_equal(r.vals, o1v)
    r = profk.run(bits, "f32", 64, p, 0, tau_override=int(kk.min()))
    assert r.status == profk.STATUS_OVERFLOW and r.count == 20_000
    assert np.array_equal(r.idx, o1i)


def test_relaxed_recall_returns_true_prefix_and_padding():
    x = workloads.normal_f32(50_000, seed=6)
    bits = keys.f32_bits(x)
    kk = keys.key_u32(bits).astype(np.int64)
    k = 200
    p = plan.plan(50_000, k, 1e-3, 0.9, plan.PlanOpts(S_min=2000, S_max=2000,
                                                    force_mode=plan.FORCE_FILTER))
    tau = int(np.sort(kk)[::-1][189])                 # 190 survivors
    r = profk.run(bits, "f32", k, p, 0, tau_override=tau)
    assert p.k_req == 180
    assert r.status == profk.STATUS_FILTERED and r.count == 190 and r.n_valid == 190
    _, o1i = exact.topk(bits, "f32", k)
    assert np.array_equal(r.idx[:190], o1i[:190])
    assert np.all(r.idx[190:] == -1)
    assert np.all(r.vals[190:] == np.uint32(0xFF800000))


def test_direct_mode_is_o1():
    x = workloads.special_f32(300, seed=2)
    bits = keys.f32_bits(x)
    p = plan.plan(300, 20)
    assert p.mode == plan.MODE_DIRECT
    r = profk.run(bits, "f32", 20, p, 0)
    v, i = exact.topk(bits, "f32", 20)
    assert r.status == profk.STATUS_DIRECT
    assert np.array_equal(r.idx, i) and np.array_equal(r.vals, v)


def test_rows_use_independent_streams_and_match_o1():
    b = workloads.relu_normal_bf16((6, 4096), seed=3)
    rp = plan.plan_rows(4096, 8, 1e-6, 1.0, plan.PlanOpts(S_min=256, S_max=256,
                                                         force_mode=plan.FORCE_FILTER))
    res = profk.run_rows(b, "bf16", 8, rp, seed=0)
    taus = {r.tau_key for r in res}
    assert len(taus) > 1
    for row, r in enumerate(res):
        v, i = exact.topk(b[row], "bf16", 8)
        assert np.array_equal(r.idx, i) and np.array_equal(r.vals, v)


def test_batchtopk_flat_indices():
    x = workloads.sae_preacts_f32(B=16, D=2048, seed=4)
    k_row = 4
    fp = plan.plan(16 * 2048, 16 * k_row, 1e-6, 1.0,
                   plan.PlanOpts(S_min=4096, S_max=4096, force_mode=plan.FORCE_FILTER))
    r = profk.run_batchtopk(keys.f32_bits(x).reshape(16, 2048), "f32", k_row, fp, 0)
    v, i = exact.topk(keys.f32_bits(x).reshape(-1), "f32", 64)
    assert np.array_equal(r.idx, i)
    rows, cols = np.divmod(r.idx, 2048)
    assert np.array_equal(x[rows, cols], v.view(np.float32))


# ---- the tie-exact (lexicographic) filter rule -----------------------------

def _lex(p):
    import dataclasses
    return dataclasses.replace(p, lexicographic=True)


def test_lex_on_a_plateau_equals_the_plain_rule_on_a_descending_ramp():
    # On a constant input the pair order is the index order, which is the
    # value order of the strictly decreasing ramp N-1, ..., 0.  So the same
    # draws must give the same count under the two rules, and the threshold
    # pair's index must be the ramp position of the plain threshold.
    n, k = 3000, 20
    p = plan.plan(n, k, 0.05, 1.0, plan.PlanOpts(S_min=200, S_max=200, force_mode=plan.FORCE_FILTER))
    flat = np.full(n, 2.5, dtype=np.float32)
    ramp = np.arange(n - 1, -1, -1).astype(np.float32)
    for seed in range(12):
        a = profk.run(keys.f32_bits(flat), "f32", k, _lex(p), seed)
        b = profk.run(keys.f32_bits(ramp), "f32", k, p, seed)
        ramp_tau = float(keys.bits_from_key_u32(np.uint32(b.tau_key)).view(np.float32))
        assert a.count == b.count
        assert a.tau_idx == n - 1 - int(ramp_tau)
        assert a.status == b.status
        assert list(a.idx) == list(range(k))      # ties: the smallest indices first


def test_lex_equals_plain_rule_on_distinct_values():
    x = workloads.normal_f32(4000, seed=8)
    assert np.unique(x).size == x.size
    p = plan.plan(4000, 16, 0.05, 1.0, plan.PlanOpts(S_min=300, S_max=300, force_mode=plan.FORCE_FILTER))
    for seed in range(6):
        a = profk.run(keys.f32_bits(x), "f32", 16, _lex(p), seed)
        b = profk.run(keys.f32_bits(x), "f32", 16, p, seed)
        assert (a.count, a.tau_key, a.status) == (b.count, b.tau_key, b.status)
        assert list(a.idx) == list(b.idx)
        # the threshold pair is a drawn element carrying the threshold value
        assert x[a.tau_idx] == keys.bits_from_key_u32(np.uint32(a.tau_key)).view(np.float32)


@pytest.mark.parametrize("seed", range(25))
def test_lex_count_is_the_rank_of_the_threshold_pair(seed):
    # brute force on small inputs with many ties: sort all N pairs by the
    # float value (descending) and then by index, and find the threshold
    # pair's position.
    g = np.random.default_rng(100 + seed)
    n = int(g.integers(80, 300))
    x = g.integers(0, 6, n).astype(np.float32)
    k = int(g.integers(1, 10))
    p = _lex(plan.plan(n, k, 0.3, 1.0, plan.PlanOpts(S_min=40, S_max=40, force_mode=plan.FORCE_FILTER)))
    r = profk.run(keys.f32_bits(x), "f32", k, p, seed)
    order = _brute_order(x)
    assert r.count == order.index(r.tau_idx) + 1
    # the threshold pair is the t-th largest drawn pair, with multiplicity
    drawn = philox.sample_indices(seed, 0, p.S, n)
    ranked = sorted(drawn, key=order.index)
    assert ranked[p.t - 1] == r.tau_idx
    assert list(r.idx) == order[:k]


def test_lex_keeps_a_plateau_inside_the_buffer():
    # 90 % of the mass on one value above the top-k boundary region: under
    # the plain rule every plateau element survives and the buffer overflows;
    # the pair rule keeps rank(tau) elements, within M.
    n, k = 200_000, 64
    x = workloads.normal_f32(n, seed=3)
    x[np.random.default_rng(0).random(n) < 0.5] = 4.0
    p = plan.plan(n, k, 1e-6, 1.0, plan.PlanOpts(S_min=4096, S_max=4096))
    plain = profk.run(keys.f32_bits(x), "f32", k, p, seed=1)
    lex = profk.run(keys.f32_bits(x), "f32", k, _lex(p), seed=1)
    assert plain.status == profk.STATUS_OVERFLOW
    assert lex.status == profk.STATUS_FILTERED and k <= lex.count <= p.M
    ex_v, ex_i = exact.topk(keys.f32_bits(x), "f32", k)
    assert list(lex.idx) == list(ex_i) and list(plain.idx) == list(ex_i)
