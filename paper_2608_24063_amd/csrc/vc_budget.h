// vc_budget.h -- host budget rule of libviscache (see vc_budget.cpp).
#pragma once
#include <stdint.h>

namespace vc {
// k[L] kept per layer, *n_surv survivors of the top-q cut (n with
// drop_all), *h_used the truncation layer; schedule is a vc_schedule value.
// Returns false for parameters without a valid budget.
bool budget_one(int32_t L, int32_t n, double rr, int32_t h_param, double m, int32_t schedule, int32_t drop_all,
                int32_t *k, int32_t *n_surv, int32_t *h_used);
}  // namespace vc
