// I/O-aware dynamic verification width (paper Sec. 4.2): choose the number
// of candidates per round q* = argmin_q T_round(q) / U(q), the estimated round
// time per committed token, from measured costs and committed counts.
//
// Per candidate width the controller keeps exponentially weighted means of
// the round's parts (history transfer, verification compute, draft
// generation, rejection correction) and of the committed tokens.  The round
// time counts the transfer and the verification compute once, as the larger
// of the two (they overlap in the streamed pipeline).  A width with fewer than
// `min_samples` observations is sampled first, in ascending order; after
// that, widths without records are estimated from the measured ones:
// transfer time is independent of q, compute and draft time are linear in q
// (least squares over the measured widths).  Committed tokens follow the
// geometric acceptance model U(q) = (1 - a^q) / (1 - a) (U = q at a = 1;
// q candidate rows are q - 1 draft tokens plus one, and the target always
// commits at least one token).  Its per-token acceptance a is fitted to all
// measured widths, each weighted by its number of rounds, so the rounds run
// at the current width keep every other width's estimate current; a width's
// own record (the mean of its first rounds, exponentially weighted after
// that) is blended with the model's value in proportion to its rounds.
// The width changes only when the estimate improves on the current width's
// by more than the switching threshold.
#include <algorithm>
#include <cmath>
#include <new>
#include <vector>

#include "specstream.h"
#include "ss_error.h"

using ss::fail;

struct ss_width_ctl {
  std::vector<int32_t> widths;
  double threshold;
  int32_t min_samples;
  double decay;
  int32_t current;   // index into widths
  struct Stat {
    int32_t n = 0;
    double transfer = 0, compute = 0, draft = 0, correct = 0, committed = 0;
  };
  std::vector<Stat> st;
};

namespace {

constexpr int32_t kMaxWeight = 32;   // rounds beyond this add no weight to a width's record
// Weight, in rounds, of the acceptance model against a width's own record of
// committed tokens.  A round's count varies a lot (at a = 0.9 and q = 8 its
// standard deviation is 45% of its mean), so a width sampled a few times
// leans on the model fitted over every round until its own rounds add up.
constexpr double kPriorRounds = 16;

// Expected committed tokens of a round with q candidate rows (q - 1 draft
// tokens) under per-token acceptance a: 1 + a + ... + a^(q-1).
double committed_model(double a, int q) {
  if (a >= 1.0) return q;
  return (1.0 - std::pow(a, q)) / (1.0 - a);
}

// Variance of a round's committed tokens under the model: n = 1 + the
// accepted drafts before the first rejection, at most q, so P(n >= k) =
// a^(k-1) for k = 1..q and E[n^2] = sum_k (2k - 1) a^(k-1).
double committed_var(double a, int q) {
  double m = 0, m2 = 0, p = 1;
  for (int k = 1; k <= q; ++k) {
    m += p;
    m2 += (2.0 * k - 1.0) * p;
    p *= a;
  }
  return m2 - m * m;
}

// Per-token acceptance whose model matches the measured committed counts
// best: weighted least squares over the measured widths, each width's
// squared deviation weighted by its rounds over the model's variance of one
// round's count (a narrow width's steady record pins a as well as a few
// rounds of a wide one); a grid over [0, 1] refined once around its best
// point.
double fit_acceptance(const ss_width_ctl *c) {
  double best_a = 0.5, best_e = INFINITY;
  for (int pass = 0; pass < 2; ++pass) {
    const double lo = pass == 0 ? 0.0 : std::max(0.0, best_a - 0.01);
    const double hi = pass == 0 ? 1.0 : std::min(1.0, best_a + 0.01);
    for (int i = 0; i <= 100; ++i) {
      const double a = lo + (hi - lo) * i / 100.0;
      double e = 0;
      for (size_t k = 0; k < c->widths.size(); ++k)
        if (c->st[k].n > 0) {
          const int q = c->widths[k];
          const double d = committed_model(a, q) - c->st[k].committed;
          e += std::min(c->st[k].n, kMaxWeight) * d * d / (committed_var(a, q) + 0.05);
        }
      if (e < best_e) {
        best_e = e;
        best_a = a;
      }
    }
  }
  return best_a;
}

// Least-squares line y = p + s * q over the measured widths of one part.
void fit_line(const ss_width_ctl *c, double ss_width_ctl::Stat::*part, double *p, double *s) {
  double n = 0, sq = 0, sy = 0, sqq = 0, sqy = 0;
  for (size_t k = 0; k < c->widths.size(); ++k)
    if (c->st[k].n > 0) {
      const double q = c->widths[k], y = c->st[k].*part;
      n += 1;
      sq += q;
      sy += y;
      sqq += q * q;
      sqy += q * y;
    }
  const double den = n * sqq - sq * sq;
  if (n < 2 || den == 0) {
    *s = 0;
    *p = n > 0 ? sy / n : 0;
    return;
  }
  *s = (n * sqy - sq * sy) / den;
  *p = (sy - *s * sq) / n;
}

// Estimated seconds per committed token at width index k.
double cost_of(const ss_width_ctl *c, size_t k) {
  const ss_width_ctl::Stat &s = c->st[k];
  const int q = c->widths[k];
  double transfer, compute, draft, correct;
  if (s.n > 0) {
    transfer = s.transfer;
    compute = s.compute;
    draft = s.draft;
    correct = s.correct;
  } else {
    double p, sl;
    fit_line(c, &ss_width_ctl::Stat::transfer, &p, &sl);
    transfer = p;   // the history volume does not depend on q
    fit_line(c, &ss_width_ctl::Stat::compute, &p, &sl);
    compute = p + sl * q;
    fit_line(c, &ss_width_ctl::Stat::draft, &p, &sl);
    draft = p + sl * q;
    fit_line(c, &ss_width_ctl::Stat::correct, &p, &sl);
    correct = p;
  }
  const double model = committed_model(fit_acceptance(c), q);
  const double n = std::min(s.n, kMaxWeight);
  const double committed = (n * s.committed + kPriorRounds * model) / (n + kPriorRounds);
  const double round = std::max(transfer, compute) + draft + correct;
  return round / std::max(committed, 1e-9);
}

}  // namespace

extern "C" {

ss_status ss_width_create(ss_width_ctl **out, const int32_t *widths, int32_t num_widths, double switch_threshold,
                          int32_t min_samples, double decay) {
  if (out == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  if (widths == nullptr || num_widths < 1 || num_widths > 64)
    return fail(SS_ERR_INVALID_ARGUMENT, "need 1..64 candidate widths");
  for (int i = 0; i < num_widths; ++i) {
    if (widths[i] < 1 || widths[i] > SS_MAX_CANDIDATES)
      return fail(SS_ERR_INVALID_ARGUMENT, "width %d outside [1, %d]", widths[i], SS_MAX_CANDIDATES);
    if (i > 0 && widths[i] <= widths[i - 1]) return fail(SS_ERR_INVALID_ARGUMENT, "widths must ascend");
  }
  if (!(switch_threshold >= 0) || !(decay > 0 && decay <= 1) || min_samples < 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "need switch_threshold >= 0, 0 < decay <= 1, min_samples >= 1");
  ss_width_ctl *c = new (std::nothrow) ss_width_ctl();
  if (c == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "out of host memory");
  c->widths.assign(widths, widths + num_widths);
  c->threshold = switch_threshold;
  c->min_samples = min_samples;
  c->decay = decay;
  c->current = 0;
  c->st.resize(num_widths);
  *out = c;
  return SS_OK;
}

void ss_width_destroy(ss_width_ctl *c) { delete c; }

ss_status ss_width_observe(ss_width_ctl *c, int32_t width, double transfer_s, double compute_s, double draft_s,
                           double correct_s, double committed_tokens) {
  if (c == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "controller is null");
  size_t k = 0;
  while (k < c->widths.size() && c->widths[k] != width) ++k;
  if (k == c->widths.size()) return fail(SS_ERR_INVALID_ARGUMENT, "width %d is not a candidate", width);
  if (!(transfer_s >= 0) || !(compute_s >= 0) || !(draft_s >= 0) || !(correct_s >= 0) || !(committed_tokens >= 0))
    return fail(SS_ERR_INVALID_ARGUMENT, "observations must be finite and >= 0");
  ss_width_ctl::Stat &s = c->st[k];
  // the plain mean of the first rounds, then the exponential weighting (a
  // weight of `decay` from the start would leave the first round's value
  // with most of the weight for about 1 / decay rounds)
  const double w = std::max(c->decay, 1.0 / (s.n + 1));
  s.transfer += w * (transfer_s - s.transfer);
  s.compute += w * (compute_s - s.compute);
  s.draft += w * (draft_s - s.draft);
  s.correct += w * (correct_s - s.correct);
  s.committed += w * (committed_tokens - s.committed);
  ++s.n;
  return SS_OK;
}

int32_t ss_width_select(ss_width_ctl *c) {
  if (c == nullptr) return -1;
  for (size_t k = 0; k < c->widths.size(); ++k)   // initial sampling phase
    if (c->st[k].n < c->min_samples) {
      c->current = (int32_t)k;
      return c->widths[k];
    }
  size_t best = c->current;
  double best_cost = cost_of(c, c->current);
  const double cur_cost = best_cost;
  for (size_t k = 0; k < c->widths.size(); ++k) {
    const double x = cost_of(c, k);
    if (x < best_cost) {
      best_cost = x;
      best = k;
    }
  }
  if (best != (size_t)c->current && best_cost < cur_cost * (1.0 - c->threshold)) c->current = (int32_t)best;
  return c->widths[c->current];
}

double ss_width_estimate(const ss_width_ctl *c, int32_t width) {
  if (c == nullptr) return -1;
  for (size_t k = 0; k < c->widths.size(); ++k)
    if (c->widths[k] == width) return cost_of(c, k);
  return -1;
}

}  // extern "C"
