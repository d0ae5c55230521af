"""Pins for the sampling reading (i.i.d. draws instead of the paper's draws
without replacement) against Lemma 1, and for the rounding and clamping of
S in Algorithm 1.

  * Lemma 1's pmf (eq. nhg_pmf) against an enumeration of every S-subset on
    tiny inputs, and its total mass at moderate sizes;
  * Lemma 1's mean and variance (eq. nhg_mean_var) against the pmf's own
    moments and against a Monte Carlo run of sampling without replacement;
  * the without-replacement tails as sums of Lemma 1's pmf;
  * the exact binomial tails the planner uses bound the without-replacement
    tails at every workload's plan, so the i.i.d. reading is conservative;
  * S = the clamped nearest integer to the minimiser of the cost model
    (eq. cost_model, Algorithm 1's constants), found numerically.
"""

import itertools
import math

import numpy as np
import pytest
from scipy.optimize import minimize_scalar

from oracle import plan


def _enumerate_wo(N, S, t):
    """Distribution of the rank of the t-th largest over all C(N, S)
    equally likely subsets (element i has rank i + 1)."""
    counts = {}
    total = 0
    for sub in itertools.combinations(range(1, N + 1), S):
        r = sub[t - 1]          # subsets come sorted: t-th smallest rank
        counts[r] = counts.get(r, 0) + 1
        total += 1
    return {r: c / total for r, c in counts.items()}


@pytest.mark.parametrize("N,S", [(7, 3), (8, 4), (9, 5), (6, 6), (10, 2)])
def test_lemma1_pmf_equals_subset_enumeration(N, S):
    for t in range(1, S + 1):
        dist = _enumerate_wo(N, S, t)
        for r in range(1, N + 1):
            assert plan.rank_pmf_wo(r, N, S, t) == pytest.approx(dist.get(r, 0.0), abs=1e-14), (N, S, t, r)


@pytest.mark.parametrize("N,S,t", [(300, 40, 7), (2000, 100, 3), (5000, 64, 64), (1000, 1000, 10)])
def test_lemma1_pmf_mass_and_moments(N, S, t):
    r = np.arange(t, N - S + t + 1)
    p = np.array([plan.rank_pmf_wo(int(x), N, S, t) for x in r])
    assert p.sum() == pytest.approx(1.0, abs=1e-10)
    mean = float((r * p).sum())
    var = float((r * r * p).sum() - mean * mean)
    assert mean == pytest.approx(plan.rank_mean_wo(N, S, t), rel=1e-10)
    assert var == pytest.approx(plan.rank_var_wo(N, S, t), rel=1e-7, abs=1e-9)


def test_lemma1_moments_monte_carlo():
    """R under uniform sampling without replacement, simulated: a random
    subset is the S smallest of N independent uniform keys."""
    N, S, t, trials = 1000, 50, 5, 40000
    rng = np.random.default_rng(12345)
    R = np.empty(trials)
    for lo in range(0, trials, 4000):
        keys = rng.random((4000, N))
        sub = np.argpartition(keys, S, axis=1)[:, :S] + 1   # ranks of the sampled elements
        R[lo:lo + 4000] = np.sort(sub, axis=1)[:, t - 1]
    m, v = plan.rank_mean_wo(N, S, t), plan.rank_var_wo(N, S, t)
    # standard errors of the sample mean and variance
    se_mean = math.sqrt(v / trials)
    mu4 = float(np.mean((R - R.mean()) ** 4))
    se_var = math.sqrt((mu4 - v * v) / trials)
    assert abs(R.mean() - m) < 5 * se_mean, (R.mean(), m)
    assert abs(R.var(ddof=1) - v) < 5 * se_var, (R.var(ddof=1), v)
    # with replacement the variance is larger (no finite-population correction)
    assert v < t * (S - t + 1) * (N + 1) ** 2 / ((S + 1) ** 2 * (S + 2))


@pytest.mark.parametrize("N,S,t", [(200, 30, 4), (500, 120, 1), (64, 64, 20)])
def test_without_replacement_tails_are_sums_of_the_pmf(N, S, t):
    pmf = {r: plan.rank_pmf_wo(r, N, S, t) for r in range(1, N + 1)}
    for k_req in range(1, N + 1, 7):
        below = sum(p for r, p in pmf.items() if r < k_req)
        assert plan.p_underflow_wo(S, t, N, k_req) == pytest.approx(below, abs=1e-12)
    for M in range(1, N + 1, 5):
        above = sum(p for r, p in pmf.items() if r > M)
        assert plan.p_overflow_wo(S, t, N, M) == pytest.approx(above, abs=1e-12)


WORKLOAD_PLANS = [
    ("C1 2^20 k=64", 2**20, 64, 1.0, plan.PlanOpts()),
    ("C2 2^28 k=16", 2**28, 16, 1.0, plan.PlanOpts()),
    ("C2 2^28 k=256", 2**28, 256, 1.0, plan.PlanOpts()),
    ("C2 2^28 k=1024", 2**28, 1024, 1.0, plan.PlanOpts()),
    ("C2 2^28 k=4096", 2**28, 4096, 1.0, plan.PlanOpts()),
    ("C3 2^26 k=512", 2**26, 512, 1.0, plan.PlanOpts()),
    ("C4 row 131072 k=32", 131072, 32, 1.0, plan.ROW_OPTS),
    ("C4 row, ratio 1", 131072, 32, 1.0, plan.PlanOpts(S_min=256)),
    ("C5 2^28 K=262144", 2**28, 262144, 1.0, plan.PlanOpts()),
    ("C5 recall 0.95", 2**28, 262144, 0.95, plan.PlanOpts()),
    ("SAE 4096x12288 K=131072", 4096 * 12288, 131072, 1.0, plan.SAE_OPTS),
]


@pytest.mark.parametrize("name,N,k,rho,opts", WORKLOAD_PLANS, ids=[w[0] for w in WORKLOAD_PLANS])
def test_binomial_tails_bound_the_without_replacement_tails(name, N, k, rho, opts):
    p = plan.plan(N, k, 1e-6, rho, opts)
    assert p.mode == plan.MODE_FILTER
    wo_u = plan.p_underflow_wo(p.S, p.t, N, p.k_req)
    wo_o = plan.p_overflow_wo(p.S, p.t, N, p.M)
    assert wo_u <= p.p_underflow and wo_o <= p.p_overflow, (wo_u, p.p_underflow, wo_o, p.p_overflow)
    assert wo_u + wo_o <= 1e-6


def _cost_minimiser(N, k, eps, ratio):
    """argmin over real S of tau_A S + tau_B M(S) log2 k with
    M(S) = k + z sqrt(k (N - k) / S), z = z_A + z_B (Algorithm 1's
    constants; f ~ 1 as Theorem 2 assumes), tau_A = 1, tau_B = ratio."""
    z = 2 * plan.z_upper(eps / 2)

    def cost(S):
        return S + ratio * (k + z * math.sqrt(k * (N - k) / S)) * math.log2(k)

    res = minimize_scalar(cost, bounds=(1.0, 1e7), method="bounded", options={"xatol": 1e-7})
    return res.x


@pytest.mark.parametrize("name,N,k,rho,opts", WORKLOAD_PLANS, ids=[w[0] for w in WORKLOAD_PLANS])
def test_sample_size_is_the_clamped_nearest_integer_to_the_cost_minimum(name, N, k, rho, opts):
    s_real = _cost_minimiser(N, k, 1e-6, opts.cost_ratio)
    frac = s_real - math.floor(s_real)
    assert abs(frac - 0.5) > 1e-3, "too close to a rounding tie to decide"
    nearest = math.floor(s_real) + (1 if frac > 0.5 else 0)
    assert plan.plan(N, k, 1e-6, rho, opts).S == min(opts.S_max, max(opts.S_min, nearest))


def test_rounding_cases_cover_both_directions():
    """Among the unclamped workload plans, S* rounds up in one and down in
    another, so flooring and ceiling both fail a case above."""
    ups = downs = 0
    for _, N, k, rho, opts in WORKLOAD_PLANS:
        s_real = _cost_minimiser(N, k, 1e-6, opts.cost_ratio)
        if opts.S_min <= s_real <= opts.S_max:
            if s_real - math.floor(s_real) > 0.5:
                ups += 1
            else:
                downs += 1
    assert ups >= 1 and downs >= 1
