// Host-side parameter selection for Prof-K (S, t, M).
//
// S follows Algorithm 1 (Theorem 2 with the log2 k cost term, rounded half
// up and clamped to [S_min, S_max]).  t and M are the smallest integers whose
// exact failure tails meet eps_A and eps_B.  With i.i.d. uniform draws the
// number of draws among the m highest-ranked elements is Bin(S, m/N), so
//   Pr(count < k_req) = Pr(Bin(S, (k_req-1)/N) >= t)          (recall failure)
//   Pr(count > M)     = Pr(Bin(S, M/N) <= t-1)                (buffer overflow)
// for distinct values; ties only raise the count.  The Gaussian forms of
// eq. (t_choice) and Corollary 1 are available as paper_literal mode.
#include <cmath>
#include <cstdint>
#include <limits>

#include "profk.h"
#include "plan_internal.h"

namespace profk {
namespace {

constexpr double kPi = 3.14159265358979323846;

// Upper-tail standard normal quantile z with Q(z) = p, 0 < p < 1, by Newton
// steps on log Q(z) (Q(z) = erfc(z / sqrt 2) / 2, Q'(z) = -phi(z)).
double z_upper(double p) {
  if (p >= 0.5) return -z_upper(1.0 - p);
  double z = std::sqrt(-2.0 * std::log(p));  // start above the root
  for (int it = 0; it < 100; ++it) {
    const double q = 0.5 * std::erfc(z / std::sqrt(2.0));
    const double phi = std::exp(-0.5 * z * z) / std::sqrt(2.0 * kPi);
    const double step = (std::log(q) - std::log(p)) * q / phi;  // g / (-g')
    z += step;
    if (std::fabs(step) <= 1e-15 * std::fmax(1.0, std::fabs(z))) break;
  }
  return z;
}

// Loader's saddle-point form of the binomial pmf ("Fast and accurate
// computation of binomial probabilities", 2000): stirlerr is the remainder
// of Stirling's formula and bd0 the deviance term.
double stirlerr(double n) {
  if (n <= 15.0) {
    if (n == 0.0) return 0.0;
    return std::lgamma(n + 1.0) - (n + 0.5) * std::log(n) + n - 0.5 * std::log(2.0 * kPi);
  }
  const double n2 = n * n;
  return (1.0 / 12 - (1.0 / 360 - (1.0 / 1260 - (1.0 / 1680 - (1.0 / 1188) / n2) / n2) / n2) / n2) / n;
}

double bd0(double x, double np) {
  if (std::fabs(x - np) < 0.1 * (x + np)) {
    const double v = (x - np) / (x + np);
    double s = (x - np) * v;
    double ej = 2.0 * x * v;
    for (int j = 1; j < 1000; ++j) {
      ej *= v * v;
      const double s1 = s + ej / (2 * j + 1);
      if (s1 == s) return s1;
      s = s1;
    }
    return s;
  }
  return x * std::log(x / np) + np - x;
}

double log_pmf(int64_t x, int64_t n, double p) {
  const double q = 1.0 - p;
  if (x == 0) return n * std::log1p(-p);
  if (x == n) return n * std::log(p);
  const double dx = static_cast<double>(x), dn = static_cast<double>(n);
  return stirlerr(dn) - stirlerr(dx) - stirlerr(dn - dx) - bd0(dx, dn * p) -
         bd0(dn - dx, dn * q) + 0.5 * std::log(dn / (2.0 * kPi * dx * (dn - dx)));
}

int64_t binom_mode(int64_t n, double p) {
  int64_t m = static_cast<int64_t>(std::floor((n + 1) * p));
  if (m > n) m = n;
  return m;
}

// Sum of pmf over i = from, from+dir, ... within [0, n], starting where the
// terms are largest and stopping once they no longer matter.
double tail_sum(int64_t from, int dir, int64_t n, double p) {
  const double q = 1.0 - p;
  double term = std::exp(log_pmf(from, n, p));
  double sum = 0.0;
  int64_t i = from;
  while (true) {
    sum += term;
    if (term <= 1e-18 * sum || term == 0.0) break;
    if (dir > 0) {
      if (i >= n) break;
      term *= (static_cast<double>(n - i) / static_cast<double>(i + 1)) * (p / q);
      ++i;
    } else {
      if (i <= 0) break;
      term *= (static_cast<double>(i) / static_cast<double>(n - i + 1)) * (q / p);
      --i;
    }
  }
  return sum;
}

double binom_sf_ge(int64_t t, int64_t n, double p);

// Pr(Bin(n, p) <= m).
double binom_cdf(int64_t m, int64_t n, double p) {
  if (m < 0) return 0.0;
  if (m >= n) return 1.0;
  if (p <= 0.0) return 1.0;
  if (p >= 1.0) return 0.0;
  if (m < binom_mode(n, p)) return std::fmin(1.0, tail_sum(m, -1, n, p));
  return 1.0 - binom_sf_ge(m + 1, n, p);
}

// Pr(Bin(n, p) >= t).
double binom_sf_ge(int64_t t, int64_t n, double p) {
  if (t <= 0) return 1.0;
  if (t > n) return 0.0;
  if (p <= 0.0) return 0.0;
  if (p >= 1.0) return 1.0;
  if (t > binom_mode(n, p)) return std::fmin(1.0, tail_sum(t, +1, n, p));
  return 1.0 - binom_cdf(t - 1, n, p);
}

template <class Ok>
bool min_int(int64_t lo, int64_t hi, Ok ok, int64_t* out) {
  if (!ok(hi)) return false;
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if (ok(mid)) hi = mid; else lo = mid + 1;
  }
  *out = lo;
  return true;
}

}  // namespace

double plan_p_underflow(int64_t S, int64_t t, int64_t N, int64_t k_req) {
  return binom_sf_ge(t, S, static_cast<double>(k_req - 1) / static_cast<double>(N));
}

double plan_p_overflow(int64_t S, int64_t t, int64_t N, int64_t M) {
  return binom_cdf(t - 1, S, static_cast<double>(M) / static_cast<double>(N));
}

double plan_z_upper(double p) { return z_upper(p); }

int make_plan(int64_t N, int64_t k, double eps, double recall,
              const profk_plan_opts_t& o, profk_plan_t* out) {
  if (!out) return PROFK_ENULL;
  if (N < 1 || k < 1 || k > N || N > static_cast<int64_t>(UINT32_MAX)) return PROFK_EINVAL;
  if (!(eps > 0.0 && eps < 1.0) || !(recall > 0.0 && recall <= 1.0)) return PROFK_EINVAL;
  if (o.S_min < 1 || o.S_max < o.S_min || !(o.cost_ratio > 0.0) ||
      !(o.eps_split > 0.0 && o.eps_split < 1.0) || o.force_mode < 0 || o.force_mode > 2)
    return PROFK_EINVAL;
  const double eps_a = o.eps_split * eps;
  const double eps_b = (1.0 - o.eps_split) * eps;
  int64_t k_req = static_cast<int64_t>(std::ceil(recall * static_cast<double>(k)));
  if (k_req < 1) k_req = 1;

  // Algorithm 1: z, S* (Theorem 2 with log2 k), round half up, clamp.
  const double z_a = z_upper(eps_a);
  const double z = z_a + z_upper(eps_b);
  const double s_star = std::pow(z * o.cost_ratio * std::log2(static_cast<double>(k)) / 2.0, 2.0 / 3.0) *
                        std::pow(static_cast<double>(k) * static_cast<double>(N - k), 1.0 / 3.0);
  double s_round = std::floor(s_star + 0.5);
  if (s_round > o.S_max) s_round = o.S_max;
  if (s_round < o.S_min) s_round = o.S_min;
  const int64_t S = static_cast<int64_t>(s_round);
  const double alpha = static_cast<double>(k) / static_cast<double>(N);

  int64_t t = 0, M = 0;
  bool t_ok = true;
  if (o.paper_literal) {
    // eq. (t_choice), Corollary 1 and the sparse-regime t = 1 rule, verbatim.
    const double f = 1.0 - static_cast<double>(S) / static_cast<double>(N);
    t = static_cast<int64_t>(std::ceil(S * alpha + z_a * std::sqrt(S * alpha * (1.0 - alpha) * f)));
    if (t < 1) t = 1;
    const long double num = static_cast<long double>(k) * static_cast<long double>(N - k);
    const double kn_over_s = static_cast<double>(num / static_cast<long double>(S));
    M = static_cast<int64_t>(std::ceil(k + z * std::sqrt(kn_over_s * f)));
    if (alpha * S < -std::log(eps_a)) t = 1;
    if (t > S) t = S;
    if (M < k) M = k;
    if (M > N) M = N;
  } else {
    if (!min_int(1, S, [&](int64_t tt) { return plan_p_underflow(S, tt, N, k_req) <= eps_a; }, &t)) {
      t_ok = false;
      t = S;
    }
    if (!min_int(k, N, [&](int64_t mm) { return plan_p_overflow(S, t, N, mm) <= eps_b; }, &M))
      M = N;
  }
  int32_t mode = PROFK_MODE_FILTER;
  if (o.force_mode == PROFK_FORCE_DIRECT) {
    mode = PROFK_MODE_DIRECT;
  } else if (o.force_mode == PROFK_FORCE_AUTO) {
    if (2 * S >= N || 8 * k > N || !t_ok) mode = PROFK_MODE_DIRECT;
  }
  out->N = N;
  out->k = k;
  out->eps = eps;
  out->recall = recall;
  out->k_req = k_req;
  out->S = S;
  out->t = t;
  out->M = M;
  out->mode = mode;
  out->lexicographic = o.lexicographic ? 1 : 0;
  out->p_underflow = plan_p_underflow(S, t, N, k_req);
  out->p_overflow = plan_p_overflow(S, t, N, M);
  return PROFK_OK;
}

}  // namespace profk
