"""Pins for oracle.plan.

  * the paper's worked examples (tests/golden/worked_examples.json);
  * Theorem 2 against a numerical minimisation of the cost model;
  * Corollary 1 against the buffer multiplier c of eqs. (c_0) and (c);
  * the exact binomial failure tails against exhaustive enumeration of every
    i.i.d. sample tuple on tiny inputs;
  * the planned failure rate against a Monte Carlo run of the sampling and
    threshold stages (Clopper-Pearson interval).
"""

import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy.optimize import minimize_scalar
from scipy.stats import binomtest

from oracle import philox, plan

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_worked_example_z():
    g = _golden()["z_eps_1e-3"]
    z = 2 * plan.z_upper(g["eps"] / 2)
    assert abs(z - g["value"]) <= g["abs_tol"]


def test_worked_example_s_star_scaling_factor():
    g = _golden()["s_star_N1e9_k100"]
    N, k = g["N"], g["k"]
    # The printed example is the (k(N-k))^(1/3) factor of Theorem 2: the
    # ratio S*/(that factor) is the prefactor alone.
    factor = (k * (N - k)) ** (1 / 3)
    assert abs(factor - g["value"]) <= g["rel_tol"] * g["value"]
    z = 2 * plan.z_upper(5e-4)
    pref = (z * math.log2(k) / 2) ** (2 / 3)
    assert plan.s_star(N, k, 1e-3) == pytest.approx(pref * factor, rel=1e-12)


def test_worked_example_buffer_size():
    g = _golden()["buffer_N2p29_k64"]
    opts = plan.PlanOpts(S_min=g["S"], S_max=g["S"], paper_literal=True,
                         force_mode=plan.FORCE_FILTER)
    p = plan.plan(g["N"], g["k"], g["eps"], 1.0, opts)
    assert p.S == g["S"]
    assert abs(p.M - g["value"]) <= g["rel_tol"] * g["value"]


@pytest.mark.parametrize("N,k,eps", [(1e9, 100, 1e-3), (2**28, 1024, 1e-6),
                                     (2**24, 32, 1e-2), (2**30, 2**19, 1e-6)])
def test_theorem2_minimises_cost_model(N, k, eps):
    # C(S) = tau_A S + tau_B M(S) log2 k with M(S) = k + z sqrt(k(N-k)/S)
    # (Sec. 4, "Optimal Sample Size", f ~ 1 as Theorem 2 assumes).
    z = 2 * plan.z_upper(eps / 2)
    ratio = 1.0

    def cost(S):
        return S + ratio * (k + z * math.sqrt(k * (N - k) / S)) * math.log2(k)

    res = minimize_scalar(cost, bounds=(1.0, 1e8), method="bounded",
                          options={"xatol": 1e-6})
    assert plan.s_star(N, k, eps, ratio) == pytest.approx(res.x, rel=1e-5)


@pytest.mark.parametrize("N,k,S,eps", [(2**20, 64, 32768, 1e-6),
                                       (2**28, 1024, 86966, 1e-6),
                                       (10**7, 5000, 40000, 1e-3)])
def test_corollary1_equals_multiplier_form(N, k, S, eps):
    # eq. (c_0): c0 = 1 + z_A/sqrt(S) sqrt((1-alpha)/alpha f)
    # eq. (c):   c  = c0 + z_B sqrt((1-alpha) f / (alpha S)),  M = ceil(c k)
    z_a = plan.z_upper(eps / 2)
    z_b = plan.z_upper(eps / 2)
    a = k / N
    f = 1 - S / N
    c0 = 1 + z_a / math.sqrt(S) * math.sqrt((1 - a) / a * f)
    c = c0 + z_b * math.sqrt((1 - a) * f / (a * S))
    opts = plan.PlanOpts(S_min=S, S_max=S, paper_literal=True,
                         force_mode=plan.FORCE_FILTER)
    p = plan.plan(N, k, eps, 1.0, opts)
    assert abs(p.M - c * k) < 1.0 + 1e-6
    assert p.M == math.ceil(c * k - 1e-9) or p.M == math.ceil(c * k)


def _enumerate_rank_distribution(N, S, t):
    """Exact distribution of R = #{x_i >= tau} over all N^S equally likely
    i.i.d. index tuples, for distinct values with element i having rank i+1."""
    dist = {}
    for tup in itertools.product(range(N), repeat=S):
        ranks = sorted(i + 1 for i in tup)          # smaller rank = larger value
        R = ranks[t - 1]                            # t-th largest sampled value
        dist[R] = dist.get(R, 0) + 1
    total = N ** S
    return {r: Fraction(c, total) for r, c in dist.items()}


@pytest.mark.parametrize("N,S", [(6, 4), (7, 3), (5, 5), (8, 2)])
def test_binomial_tails_equal_exhaustive_enumeration(N, S):
    for t in range(1, S + 1):
        dist = _enumerate_rank_distribution(N, S, t)
        for k_req in range(1, N + 1):
            exact = float(sum(p for r, p in dist.items() if r < k_req))
            assert plan.p_underflow(S, t, N, k_req) == pytest.approx(exact, abs=1e-13)
        for M in range(1, N + 1):
            exact = float(sum(p for r, p in dist.items() if r > M))
            assert plan.p_overflow(S, t, N, M) == pytest.approx(exact, abs=1e-13)


@pytest.mark.parametrize("N,k,eps,rho", [(2**20, 64, 1e-6, 1.0),
                                         (2**28, 1024, 1e-6, 1.0),
                                         (2**28, 262144, 1e-6, 0.95),
                                         (131072, 32, 1e-6, 1.0),
                                         (10**6, 10, 1e-3, 1.0)])
def test_exact_plan_is_minimal(N, k, eps, rho):
    p = plan.plan(N, k, eps, rho)
    ea = eb = eps / 2
    assert p.k_req == math.ceil(rho * k)
    assert plan.p_underflow(p.S, p.t, N, p.k_req) <= ea
    if p.t > 1:
        assert plan.p_underflow(p.S, p.t - 1, N, p.k_req) > ea
    assert plan.p_overflow(p.S, p.t, N, p.M) <= eb
    if p.M > k:
        assert plan.p_overflow(p.S, p.t, N, p.M - 1) > eb
    assert p.p_underflow + p.p_overflow <= eps


def test_monte_carlo_failure_rate_within_interval():
    N, k, eps = 4096, 32, 0.05
    opts = plan.PlanOpts(S_min=96, S_max=96, force_mode=plan.FORCE_FILTER)
    p = plan.plan(N, k, eps, 1.0, opts)
    trials = 6000
    fails = 0
    for seed in range(trials):
        idx = philox.sample_indices(seed, 0, p.S, N)
        ranks = np.sort(idx + 1)                   # element i has rank i+1
        R = int(ranks[p.t - 1])
        fails += (R < p.k_req) or (R > p.M)
    ci = binomtest(fails, trials).proportion_ci(confidence_level=0.999)
    expected = p.p_underflow + p.p_overflow
    assert ci.low <= expected <= ci.high
    assert ci.low <= eps


def test_direct_mode_rules():
    assert plan.plan(1000, 10).mode == plan.MODE_DIRECT        # S >= N/2
    assert plan.plan(2**20, 2**18).mode == plan.MODE_DIRECT    # 8k > N
    assert plan.plan(2**20, 64).mode == plan.MODE_FILTER
    forced = plan.plan(1000, 10, opts=plan.PlanOpts(S_min=64, S_max=64,
                                                    force_mode=plan.FORCE_FILTER))
    assert forced.mode == plan.MODE_FILTER and forced.S == 64


def test_paper_literal_t1_rule_is_recall_hostile():
    # The literal Algorithm 1 sets t = 1 in the sparse regime; the exact
    # recall-failure probability of that choice is far above eps.
    opts = plan.PlanOpts(paper_literal=True)
    p = plan.plan(2**20, 64, 1e-6, 1.0, opts)
    assert p.t == 1 and p.p_underflow > 0.5
