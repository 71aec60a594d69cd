// Fleet cost model (Sec. 3, "Cost Model: Why Splitting Always Helps").
//
// A homogeneous fleet at C_max = C_H needs G_homo = ceil(lambda / mu(C_H))
// GPUs; a dual-pool fleet whose short pool (C_max = C_S) serves a fraction
// alpha of the traffic needs G_dual = ceil(alpha lambda / mu(C_S)) +
// ceil((1 - alpha) lambda / mu(C_H)).  Ignoring the ceilings the fractional
// saving is the boxed equation alpha (1 - 1/rho), rho = mu(C_S) / mu(C_H).
// IEEE double, step by step in that order (built with -ffp-contract=off).
#include <cmath>

#include "common.h"

extern "C" int dp_cost_model(double lambda, double alpha, double mu_short, double mu_long, dp_cost_result* out) {
  using dpool::fail;
  if (!out) return fail(DP_EINVAL, "dp_cost_model: null result");
  if (!(lambda > 0.0) || !std::isfinite(lambda)) return fail(DP_EINVAL, "dp_cost_model: lambda must be positive");
  if (!(alpha >= 0.0 && alpha <= 1.0)) return fail(DP_EINVAL, "dp_cost_model: alpha must be in [0, 1]");
  if (!(mu_short > 0.0) || !(mu_long > 0.0) || !std::isfinite(mu_short) || !std::isfinite(mu_long))
    return fail(DP_EINVAL, "dp_cost_model: throughputs must be positive");
  const double g_homo = std::ceil(lambda / mu_long);
  const double g_short = std::ceil((alpha * lambda) / mu_short);
  const double g_long = std::ceil(((1.0 - alpha) * lambda) / mu_long);
  if (g_homo > 9.0e18 || g_short + g_long > 9.0e18) return fail(DP_EINVAL, "dp_cost_model: GPU counts overflow");
  const double rho = mu_short / mu_long;
  out->g_homo = (int64_t)g_homo;
  out->g_dual = (int64_t)g_short + (int64_t)g_long;
  out->rho = rho;
  out->savings_formula = alpha * (1.0 - 1.0 / rho);
  out->savings_fleet = (g_homo - (g_short + g_long)) / g_homo;
  return DP_OK;
}
