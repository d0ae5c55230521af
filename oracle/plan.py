"""Parameter selection (S, t, M) -- Algorithm 1 plus exact binomial tails.

Test infrastructure (see the package docstring).  fp64 throughout.

What the paper fixes
  * Algorithm 1: z = Phi^-1(1 - eps/2) + Phi^-1(1 - eps/2); alpha = k/N;
    S* = (z (tau_B/tau_A) log2 k / 2)^(2/3) (k (N-k))^(1/3)  (Theorem 2);
    S = min(S_max, max(S_min, round(S*))); f = 1 - S/N;
    t = max(1, ceil(S alpha + (z/2) sqrt(S alpha (1-alpha) f)))  (eq. t_choice);
    M = ceil(k + z sqrt(k (N-k) / S * f))                          (Corollary 1);
    t = 1 when alpha S < -ln(eps/2).
  * Defaults: S_min = 32768, S_max = 2^17, tau_B/tau_A = 1 (Sec. 4,
    "Optimal Sample Size"); eps_A = eps_B = eps/2 (Theorem 1).
  * Design goal (Sec. 3): choose (S, t, M) so that k <= R <= M with
    probability at least 1 - eps, where R = #{i : x_i >= tau}.

Readings taken where the paper is silent or inconsistent
  * Sampling is i.i.d. uniform (with replacement).  Then the number of draws
    that land among the m highest-ranked elements is exactly Bin(S, m/N), so
        Pr(R < k_req) = Pr(Bin(S, (k_req-1)/N) >= t)
        Pr(R > M)     = Pr(Bin(S, M/N) <= t-1)
    hold exactly for distinct values (ties only raise R).  Lemma 1's law of
    R under sampling without replacement is kept below (rank_pmf_wo and the
    *_wo tails) to check that these binomial tails bound it.
  * S comes from Algorithm 1.  t and M are the smallest integers that meet
    eps_A and eps_B under those exact tails, because the Gaussian forms of
    eq. t_choice and Corollary 1 under-provision M by orders of magnitude at
    small t, and the t = 1 rule states the success probability (1-alpha)^S as
    the failure probability.  The literal Algorithm 1 is kept as
    paper_literal=True for reporting only.
  * log in S* is log2 (Algorithm 1); round(S*) is round-half-up.
  * Rows: S_min = 256 and tau_B/tau_A = 0.5 (a measured hardware constant;
    the flat default stays at the paper's 1).
  * lexicographic=True selects the tie-exact filter rule of oracle.profk: the
    rank argument behind both tails counts elements above a threshold in a
    total order, and (key, -index) is one with no ties, so the same t and M
    bound Pr(count < k_req) and Pr(count > M) for every input, plateaus
    included.  Under the paper's rule (key >= tau) the tails hold for
    distinct values only.
  * Relaxed recall rho < 1 plans for k_req = ceil(rho k) in the recall tail.
  * mode DIRECT (an exact top-k with no sampling) when S >= N/2, when 8k > N,
    or when no t <= S meets eps_A; it never changes the result.
"""

import math
from dataclasses import dataclass

from scipy.special import gammaln
from scipy.stats import binom, hypergeom, norm

MODE_FILTER = 0
MODE_DIRECT = 1

FORCE_AUTO = 0
FORCE_FILTER = 1
FORCE_DIRECT = 2


@dataclass(frozen=True)
class PlanOpts:
    S_min: int = 32768
    S_max: int = 131072
    cost_ratio: float = 1.0   # tau_B / tau_A
    eps_split: float = 0.5    # eps_A = eps_split * eps
    paper_literal: bool = False
    force_mode: int = FORCE_AUTO
    lexicographic: bool = False  # filter on (key, -index), see the module docstring


ROW_OPTS = PlanOpts(S_min=256, cost_ratio=0.5)
# The fused SAE path: a draw is a d_model-long dot product, not one gathered
# element, so tau_B / tau_A is measured far below 1 (Sec. 4, "Optimal Sample
# Size", leaves the ratio to a benchmark of the hardware).
SAE_OPTS = PlanOpts(cost_ratio=1.0 / 64.0)


@dataclass(frozen=True)
class Plan:
    N: int
    k: int
    eps: float
    recall: float
    k_req: int
    S: int
    t: int
    M: int
    mode: int
    p_underflow: float
    p_overflow: float
    lexicographic: bool = False


def z_upper(eps_tail):
    """Phi^-1(1 - eps_tail), evaluated as the inverse survival function so
    that small tails keep full precision."""
    return float(norm.isf(eps_tail))


def s_star(N, k, eps, cost_ratio=1.0, eps_split=0.5):
    """Theorem 2 with Algorithm 1's constants (log base 2)."""
    z = z_upper(eps_split * eps) + z_upper((1.0 - eps_split) * eps)
    return (z * cost_ratio * math.log2(k) / 2.0) ** (2.0 / 3.0) \
        * (k * (N - k)) ** (1.0 / 3.0)


def sample_size(N, k, eps, opts):
    """Algorithm 1: S* rounded half-up, then clamped to [S_min, S_max]."""
    s = s_star(N, k, eps, opts.cost_ratio, opts.eps_split)
    return int(min(opts.S_max, max(opts.S_min, math.floor(s + 0.5))))


def p_underflow(S, t, N, k_req):
    """Pr(R < k_req) = Pr(Bin(S, (k_req-1)/N) >= t)."""
    return float(binom.sf(t - 1, S, (k_req - 1) / N))


def p_overflow(S, t, N, M):
    """Pr(R > M) = Pr(Bin(S, M/N) <= t-1)."""
    return float(binom.cdf(t - 1, S, M / N))


# ---- Lemma 1: the threshold rank under sampling without replacement ----
# The planner draws i.i.d. (with replacement); these are the paper's own
# distribution, kept to compare the two sampling schemes.

def _log_comb(n, r):
    return gammaln(n + 1) - gammaln(r + 1) - gammaln(n - r + 1)


def rank_pmf_wo(r, N, S, t):
    """Lemma 1, eq. (nhg_pmf): Pr(R = r) for the t-th largest of S indices
    drawn without replacement, rank 1 the largest, r in [t, N - S + t]:
    C(r-1, t-1) C(N-r, S-t) / C(N, S)."""
    if r < t or r > N - S + t:
        return 0.0
    return float(math.exp(_log_comb(r - 1, t - 1) + _log_comb(N - r, S - t) - _log_comb(N, S)))


def rank_mean_wo(N, S, t):
    """Lemma 1, eq. (nhg_mean_var): E[R] = (N + 1) t / (S + 1)."""
    return (N + 1) * t / (S + 1)


def rank_var_wo(N, S, t):
    """Lemma 1, eq. (nhg_mean_var):
    Var(R) = t (S - t + 1) (N + 1) (N - S) / ((S + 1)^2 (S + 2))."""
    return t * (S - t + 1) * (N + 1) * (N - S) / ((S + 1) ** 2 * (S + 2))


def p_underflow_wo(S, t, N, k_req):
    """Pr(R < k_req) without replacement: at least t of the S draws land
    among the k_req - 1 highest ranks (a hypergeometric tail)."""
    return float(hypergeom.sf(t - 1, N, k_req - 1, S))


def p_overflow_wo(S, t, N, M):
    """Pr(R > M) without replacement: fewer than t draws among the M
    highest ranks."""
    return float(hypergeom.cdf(t - 1, N, M, S))


def _min_int(lo, hi, ok):
    """Smallest integer m in [lo, hi] with ok(m), for ok monotone
    (False...False True...True); None when ok(hi) is False."""
    if not ok(hi):
        return None
    while lo < hi:
        mid = (lo + hi) // 2
        if ok(mid):
            hi = mid
        else:
            lo = mid + 1
    return lo


def plan(N, k, eps=1e-6, recall=1.0, opts=PlanOpts()):
    N = int(N)
    k = int(k)
    if N < 1 or k < 1 or k > N:
        raise ValueError("need 1 <= k <= N")
    if not (0.0 < eps < 1.0) or not (0.0 < recall <= 1.0):
        raise ValueError("need 0 < eps < 1 and 0 < recall <= 1")
    eps_a = opts.eps_split * eps
    eps_b = (1.0 - opts.eps_split) * eps
    k_req = max(1, math.ceil(recall * k))
    S = sample_size(N, k, eps, opts)
    alpha = k / N
    t_ok = True
    if opts.paper_literal:
        z_a = z_upper(eps_a)
        z = z_a + z_upper(eps_b)
        f = 1.0 - S / N
        t = max(1, math.ceil(S * alpha + z_a * math.sqrt(S * alpha * (1 - alpha) * f)))
        M = math.ceil(k + z * math.sqrt(k * (N - k) / S * f))
        if alpha * S < -math.log(eps_a):
            t = 1
        t = min(t, S)
        M = min(max(M, k), N)
    else:
        t = _min_int(1, S, lambda tt: p_underflow(S, tt, N, k_req) <= eps_a)
        if t is None:
            t_ok = False
            t = S
        M = _min_int(k, N, lambda mm: p_overflow(S, t, N, mm) <= eps_b)
    mode = MODE_FILTER
    if opts.force_mode == FORCE_DIRECT:
        mode = MODE_DIRECT
    elif opts.force_mode == FORCE_AUTO:
        if 2 * S >= N or 8 * k > N or not t_ok:
            mode = MODE_DIRECT
    return Plan(N=N, k=k, eps=float(eps), recall=float(recall), k_req=k_req,
                S=S, t=t, M=M, mode=mode,
                p_underflow=p_underflow(S, t, N, k_req),
                p_overflow=p_overflow(S, t, N, M),
                lexicographic=bool(opts.lexicographic))


def plan_rows(D, k, eps=1e-6, recall=1.0, opts=ROW_OPTS):
    """Per-row plan: the same selection with N = D, a lower S floor, since
    S_min = 32768 would sample a quarter of a 131072-wide row, and the cost
    ratio tau_B/tau_A = 0.5, which Sec. 4 ("Optimal Sample Size") leaves to a
    measurement of the hardware (the per-row kernel's, on MI355X)."""
    return plan(D, k, eps, recall, opts)
