// vc_budget.cpp -- layer budgets of PruneKV on the host (Sec. 3.2, Eq.
// (parabolic) and the normalisation sum_{l<=h} b_l = h*m; Sec. 4, RR =
// p*q*(h/L)*m with p = 1; Algorithm 1, Step 1 for the top-q survivors).
// The fixed, arithmetic and geometric schedules of the budget ablation
// replace only the raw proportions (readings stated in viscache.h).
//
// Integer rule (a reading; the paper gives proportions only): the per-sequence
// total T = floor(RR*L*n + 0.5) is apportioned to layers 1..h in proportion to
// b_l by largest remainder, ties to the shallower layer.  Proportions above 1
// after scaling are held at 1 and the rest rescaled (water filling).  The
// double-precision expressions below are evaluated in a fixed order so that
// every implementation of this rule gets the same integers.
#include <algorithm>
#include <cmath>
#include <vector>

#include "vc_budget.h"

namespace vc {

bool budget_one(int32_t L, int32_t n, double rr, int32_t h_param, double m, int32_t schedule, int32_t drop_all,
                int32_t *k, int32_t *n_surv, int32_t *h_used) {
  if (L < 2 || n < 0) return false;
  if (!(rr > 0.0 && rr <= 1.0) || !(m > 0.0 && m <= 1.0)) return false;
  const int32_t h = h_param != 0 ? h_param : static_cast<int32_t>(std::floor(0.75 * L + 0.5));
  if (h < 2 || h > L) return false;

  std::vector<double> raw(h), prop(h);
  const double den = 2.0 * static_cast<double>(h - 1) * static_cast<double>(h - 1);
  for (int32_t i = 0; i < h; ++i) {
    const double li = static_cast<double>(i);  // l - 1
    switch (schedule) {
      case 0:  // parabolic
        raw[i] = 1.0 - (li * li) / den;
        break;
      case 1:  // fixed
        raw[i] = 1.0;
        break;
      case 2:  // arithmetic, 1 down to 1/2
        raw[i] = 1.0 - li / (2.0 * static_cast<double>(h - 1));
        break;
      case 3:  // geometric over four depth blocks
        raw[i] = std::ldexp(1.0, -static_cast<int>((4 * i) / h));
        break;
      default:
        return false;
    }
  }
  // Water filling towards sum = h*m.
  std::vector<bool> held(h, false);
  double scale = 0.0;
  for (;;) {
    int32_t nheld = 0;
    double rest = 0.0;
    for (int32_t i = 0; i < h; ++i) {
      if (held[i]) ++nheld;
      else rest += raw[i];
    }
    if (nheld == h) break;
    scale = (static_cast<double>(h) * m - static_cast<double>(nheld)) / rest;
    bool grew = false;
    for (int32_t i = 0; i < h; ++i) {
      if (!held[i] && scale * raw[i] > 1.0) {
        held[i] = true;
        grew = true;
      }
    }
    if (!grew) break;
  }
  for (int32_t i = 0; i < h; ++i) prop[i] = held[i] ? 1.0 : scale * raw[i];

  double q = rr / ((static_cast<double>(h) / static_cast<double>(L)) * m);
  if (q > 1.0 + 1e-9) return false;
  q = std::min(q, 1.0);

  const double total = std::floor(rr * static_cast<double>(L) * static_cast<double>(n) + 0.5);
  double psum = 0.0;
  for (int32_t i = 0; i < h; ++i) psum += prop[i];
  std::vector<double> rem(h);
  double given = 0.0;
  for (int32_t i = 0; i < h; ++i) {
    const double share = total * prop[i] / psum;
    const double whole = std::floor(share);
    k[i] = static_cast<int32_t>(whole);
    rem[i] = share - whole;
    given += whole;
  }
  const int32_t left = static_cast<int32_t>(total - given);
  if (left < 0 || left > h) return false;
  std::vector<int32_t> order(h);
  for (int32_t i = 0; i < h; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t a, int32_t b) { return rem[a] > rem[b]; });
  for (int32_t j = 0; j < left; ++j) k[order[j]] += 1;
  for (int32_t i = h; i < L; ++i) k[i] = 0;
  for (int32_t i = 0; i < h; ++i)
    if (k[i] > n) return false;

  int32_t ns = static_cast<int32_t>(std::floor(q * static_cast<double>(n) + 0.5));
  for (int32_t i = 0; i < h; ++i) ns = std::max(ns, k[i]);
  ns = std::min(ns, n);
  if (drop_all) ns = n;
  *n_surv = ns;
  if (h_used) *h_used = h;
  return true;
}

}  // namespace vc
