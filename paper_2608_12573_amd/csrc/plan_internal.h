// Host-side internals shared by the planner and the C ABI layer.
#pragma once

#include <cstdint>

#include "profk.h"

namespace profk {

// Exact failure tails under i.i.d. uniform sampling (see plan.cpp).
double plan_p_underflow(int64_t S, int64_t t, int64_t N, int64_t k_req);
double plan_p_overflow(int64_t S, int64_t t, int64_t N, int64_t M);
double plan_z_upper(double p);

int make_plan(int64_t N, int64_t k, double eps, double recall,
              const profk_plan_opts_t& opts, profk_plan_t* out);

}  // namespace profk
