// Adaptive ABFT detection frequencies (paper Sec. 4.5, Algorithm 1): host
// code that picks, per protection section, the fraction of training steps
// on which its checks run, and turns those fractions into a per-step
// section mask for attn_abft_forward / attn_abft_backward.
//
// Coverage model (Sec. 4.5). Errors of type e strike an operation of n
// flops as a Poisson process of rate lambda_e per flop. A section survives
// with no error, or with exactly one that is handled (checks on, f_S) or
// harmless (probability 1 - p, p from the paper's Table 4). Near 1 the
// coverage FC is computed through the failure probability U = 1 - FC:
//   U_S(f) = P(>= 2 errors in S) + (1 - f) * sum_i sum_e R_e(i) p_i^e
//   U_att  = 1 - prod_S (1 - U_S)
// with R_e(i) = lambda_e n_i exp(-mu_S), mu_S the section's mean count.
// U_S is linear in f_S, so each section gains coverage at the constant rate
// FCE_S = sum R_e(i) p_i^e / T_S per unit of check time; Algorithm 1 is the
// greedy allocation in descending FCE (the fractional knapsack of the first
// order expansion of the product): whole sections while the deficit
// allows, then the fraction that closes it. A target that even full
// checking misses checks every section always.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "attn_abft.h"

namespace {

constexpr int kTypes = 3;  // INF, NaN, near-INF
constexpr int kMaxSections = 16;

// P(k >= 2) of a Poisson law of mean mu, free of cancellation for small mu
double p_two_or_more(double mu) {
  if (mu > 0.5) return 1.0 - std::exp(-mu) * (1.0 + mu);
  double term = 0.5 * mu * mu, acc = 0.0;
  for (int k = 2; term > 0.0 && term > acc * 1e-18; ++k) {
    acc += term;
    term *= mu / double(k + 1);
  }
  return std::exp(-mu) * acc;
}

struct SectionTerms {
  double two_or_more;  // P(>= 2 errors)
  double harmful;      // sum R_e(i) p_i^e
};

SectionTerms terms(const abft_freq_op* ops, const abft_freq_section& s, const double* lambda) {
  double mu = 0.0;
  for (int i = 0; i < s.n_ops; ++i)
    for (int e = 0; e < kTypes; ++e) mu += lambda[e] * ops[s.first_op + i].flops;
  const double none = std::exp(-mu);
  double harm = 0.0;
  for (int i = 0; i < s.n_ops; ++i)
    for (int e = 0; e < kTypes; ++e)
      harm += lambda[e] * ops[s.first_op + i].flops * none * ops[s.first_op + i].p[e];
  return {p_two_or_more(mu), harm};
}

double unsafe_att(const std::vector<SectionTerms>& t, const double* f) {
  double lg = 0.0;
  for (size_t s = 0; s < t.size(); ++s)
    lg += std::log1p(-(t[s].two_or_more + (1.0 - f[s]) * t[s].harmful));
  return -std::expm1(lg);
}

bool valid(const abft_freq_op* ops, const abft_freq_section* secs, int32_t n_secs,
           const double* lambda) {
  if (!ops || !secs || !lambda || n_secs < 1 || n_secs > kMaxSections) return false;
  for (int e = 0; e < kTypes; ++e)
    if (!(lambda[e] >= 0.0) || !std::isfinite(lambda[e])) return false;
  for (int s = 0; s < n_secs; ++s) {
    if (secs[s].n_ops < 0 || secs[s].first_op < 0 || !(secs[s].cost >= 0.0) ||
        !std::isfinite(secs[s].cost))
      return false;
    for (int i = 0; i < secs[s].n_ops; ++i) {
      const abft_freq_op& o = ops[secs[s].first_op + i];
      if (!(o.flops >= 0.0) || !std::isfinite(o.flops)) return false;
      for (int e = 0; e < kTypes; ++e)
        if (!(o.p[e] >= 0.0 && o.p[e] <= 1.0)) return false;
    }
  }
  return true;
}

}  // namespace

extern "C" {

int attn_abft_unsafe_probability(const abft_freq_op* ops, const abft_freq_section* secs,
                                 int32_t n_secs, const double* lambda, const double* freqs,
                                 double* unsafe_out) {
  if (!valid(ops, secs, n_secs, lambda) || !freqs || !unsafe_out) return ABFT_ERR_INVALID;
  std::vector<SectionTerms> t;
  for (int s = 0; s < n_secs; ++s) {
    if (!(freqs[s] >= 0.0 && freqs[s] <= 1.0)) return ABFT_ERR_INVALID;
    t.push_back(terms(ops, secs[s], lambda));
  }
  *unsafe_out = unsafe_att(t, freqs);
  return ABFT_OK;
}

int attn_abft_optimize_frequencies(const abft_freq_op* ops, const abft_freq_section* secs,
                                   int32_t n_secs, const double* lambda, double fail_target,
                                   double* freqs_out) {
  if (!valid(ops, secs, n_secs, lambda) || !freqs_out || !(fail_target >= 0.0))
    return ABFT_ERR_INVALID;
  std::vector<SectionTerms> t;
  for (int s = 0; s < n_secs; ++s) t.push_back(terms(ops, secs[s], lambda));
  std::vector<double> ones(n_secs, 1.0), zeros(n_secs, 0.0);
  if (fail_target <= unsafe_att(t, ones.data())) {
    std::copy(ones.begin(), ones.end(), freqs_out);
    return ABFT_OK;
  }
  double deficit = unsafe_att(t, zeros.data()) - fail_target;
  // a check that costs nothing runs every step, and its coverage counts
  // before any paid section is considered
  std::vector<int> order;
  for (int s = 0; s < n_secs; ++s) {
    if (secs[s].cost > 0.0) {
      order.push_back(s);
      freqs_out[s] = 0.0;
    } else {
      freqs_out[s] = 1.0;
      deficit -= t[s].harmful;
    }
  }
  // paid sections by coverage gained per unit of check time, best first
  std::vector<double> eff(n_secs, 0.0);
  for (int s : order) eff[s] = t[s].harmful / secs[s].cost;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return eff[a] > eff[b]; });
  for (int s : order) {
    if (deficit <= 0.0) break;
    const double whole = t[s].harmful;  // gain of checking it every step
    if (whole <= deficit) {
      freqs_out[s] = 1.0;
      deficit -= whole;
    } else {
      freqs_out[s] = deficit / whole;
      deficit = 0.0;
    }
  }
  return ABFT_OK;
}

uint32_t attn_abft_sections_for_step(const double* freqs, int64_t step) {
  if (!freqs || step < 0) return 0u;
  static const uint32_t bit[4] = {ABFT_SEC_AS, ABFT_SEC_CL, ABFT_SEC_O, ABFT_SEC_BWD};
  uint32_t mask = 0;
  for (int s = 0; s < 4; ++s) {
    const double f = freqs[s];
    if (!(f > 0.0)) continue;
    if (f >= 1.0 || std::floor(double(step + 1) * f) > std::floor(double(step) * f)) mask |= bit[s];
  }
  return mask;
}

}  // extern "C"
