// Token-budget pool routing: Sec. 2.1 Eq. 3-5; the dispatch rule of Sec. 2.2
// (Algorithm 1).
// Host only.  Compiled with -ffp-contract=off: every double operation is
// rounded on its own, in the order written, so that any IEEE-754 double
// implementation of the same steps agrees bit for bit.
#include <cmath>
#include <cstdint>

#include "common.h"

namespace {

constexpr int kShort = 0;
constexpr int kLong = 1;

bool overloaded(const dp_route_params* p, const dp_pool_state& pool) {
  return (double)pool.in_flight >= p->spill_theta * (double)pool.capacity;
}

// Eq. 5: conservative bytes-per-token ratio, floored at c_min.
double conservative_ratio(const dp_route_params* p, const dp_cat_state& c) {
  double r = c.c_hat - p->gamma * c.sigma;
  if (r < p->c_min) r = p->c_min;
  return r;
}

// The pool that serves a request of l_total tokens (Sec. 2.2).  A pool is
// eligible when its C_max holds l_total; the long pool is the fallback when
// the short one is not.  The token budget prefers the short pool for
// l_total <= B_short and the long pool above it.  A preferred pool that is
// overloaded gives the request to the other pool if that one is eligible and
// not overloaded.  A preferred pool that cannot hold it (a long pool with
// the smaller C_max) falls back to the long pool.
int pick_pool(const dp_route_params* p, const dp_pool_state* pools, int64_t l_total) {
  const bool eligible[2] = {l_total <= pools[kShort].c_max, l_total <= pools[kLong].c_max};
  if (!eligible[kShort]) return kLong;
  const int pref = (double)l_total <= p->b_short ? kShort : kLong;
  const int other = 1 - pref;
  const bool hand_over = overloaded(p, pools[pref]) && eligible[other] && !overloaded(p, pools[other]);
  const int pick = hand_over ? other : pref;
  return eligible[pick] ? pick : kLong;
}

}  // namespace

extern "C" int route_default_params(dp_route_params* params) {
  if (!params) return dpool::fail(DP_EINVAL, "route_default_params: null");
  params->b_short = 8192.0;  // Sec. 2.2 "Choosing B_short"
  params->beta = 0.95;       // Eq. 4
  params->gamma = 1.0;       // Eq. 5
  params->c0 = 4.0;          // Sec. 2.1 cold start
  params->c_min = 1.0;
  params->spill_theta = 1.0;
  return DP_OK;
}

extern "C" int route_init(const dp_route_params* params, dp_cat_state* cats, int32_t n_cats) {
  if (!params || (!cats && n_cats > 0) || n_cats < 0) return dpool::fail(DP_EINVAL, "route_init: bad arguments");
  for (int32_t k = 0; k < n_cats; ++k) {
    cats[k].c_hat = params->c0;
    cats[k].sigma = 0.0;
  }
  return DP_OK;
}

extern "C" int route_requests(const dp_route_params* params, const dp_cat_state* cats, int32_t n_cats,
                              dp_pool_state pools[2], const int64_t* req_bytes, const int32_t* req_cat,
                              const int64_t* req_max_out, int64_t n, int8_t* out_pool, int64_t* out_l_total) {
  using dpool::fail;
  if (!params || !cats || !pools || n_cats <= 0 || n < 0) return fail(DP_EINVAL, "route_requests: bad arguments");
  if (n == 0) return DP_OK;
  if (!req_bytes || !req_cat || !req_max_out) return fail(DP_EINVAL, "route_requests: null request arrays");
  if (!(params->c_min > 0.0)) return fail(DP_EINVAL, "route_requests: c_min must be > 0");
  for (int64_t i = 0; i < n; ++i) {
    if (req_bytes[i] < 0 || req_max_out[i] < 0 || req_cat[i] < 0 || req_cat[i] >= n_cats)
      return fail(DP_EINVAL, "route_requests: request %lld has bytes/max_out < 0 or category out of range",
                  (long long)i);
  }
  for (int64_t i = 0; i < n; ++i) {
    const double c_star = conservative_ratio(params, cats[req_cat[i]]);          // Eq. 5
    const int64_t l_total = (int64_t)std::ceil((double)req_bytes[i] / c_star) + req_max_out[i];  // Eq. 3
    const int choice = pick_pool(params, pools, l_total);
    pools[choice].in_flight += 1;
    if (out_pool) out_pool[i] = (int8_t)choice;
    if (out_l_total) out_l_total[i] = l_total;
  }
  return DP_OK;
}

extern "C" int route_on_response(const dp_route_params* params, dp_cat_state* cats, int32_t n_cats, int32_t cat,
                                 int64_t req_bytes, int64_t prompt_tokens) {
  using dpool::fail;
  if (!params || !cats || cat < 0 || cat >= n_cats || req_bytes < 0 || prompt_tokens <= 0)
    return fail(DP_EINVAL, "route_on_response: bad arguments (cat %d, bytes %lld, prompt_tokens %lld)", cat,
                (long long)req_bytes, (long long)prompt_tokens);
  dp_cat_state& st = cats[cat];
  const double c_obs = (double)req_bytes / (double)prompt_tokens;       // Eq. 4
  const double one_minus_beta = 1.0 - params->beta;
  st.c_hat = params->beta * st.c_hat + one_minus_beta * c_obs;         // Eq. 4 EMA
  st.sigma = params->beta * st.sigma + one_minus_beta * std::fabs(c_obs - st.c_hat);  // uncertainty EMA
  return DP_OK;
}

// Adaptive B_short: the control rule include/dpool.h documents (Sec. 7's
// future-work direction, Sec. 6's 1% preemption alert level as the default
// target, Sec. 4.6's 4K-16K plateau as the default bounds).
extern "C" int route_adapt_default_params(dp_adapt_params* ap) {
  if (!ap) return dpool::fail(DP_EINVAL, "route_adapt_default_params: null");
  ap->w_preempt = 1.0;
  ap->w_oom = 1.0;
  ap->w_reject = 1.0;
  ap->target = 0.01;
  ap->step = 0.05;
  ap->b_min = 4096.0;
  ap->b_max = 16384.0;
  return DP_OK;
}

extern "C" int route_adapt_threshold(const dp_adapt_params* ap, const dp_pool_signals signals[2], double* b_short,
                                     int32_t* action) {
  using dpool::fail;
  if (!ap || !signals || !b_short) return fail(DP_EINVAL, "route_adapt_threshold: null argument");
  for (int i = 0; i < 2; ++i) {
    const dp_pool_signals& g = signals[i];
    if (g.admitted < 0 || g.preempted < 0 || g.oom < 0 || g.rejected < 0)
      return fail(DP_EINVAL, "route_adapt_threshold: negative count in pool %d", i);
  }
  if (!(ap->w_preempt >= 0.0 && ap->w_oom >= 0.0 && ap->w_reject >= 0.0 && ap->target >= 0.0))
    return fail(DP_EINVAL, "route_adapt_threshold: weights and target must be >= 0");
  if (!(ap->step > 0.0 && ap->step < 1.0)) return fail(DP_EINVAL, "route_adapt_threshold: step must be in (0, 1)");
  if (!(ap->b_min > 0.0 && ap->b_min <= ap->b_max && std::isfinite(ap->b_max)))
    return fail(DP_EINVAL, "route_adapt_threshold: need 0 < b_min <= b_max < inf");
  const double b = *b_short;
  if (!(std::isfinite(b) && b > 0.0)) return fail(DP_EINVAL, "route_adapt_threshold: b_short must be finite and > 0");
  double x[2];
  for (int i = 0; i < 2; ++i) {
    const dp_pool_signals& g = signals[i];
    double e = ap->w_preempt * (double)g.preempted;
    e = e + ap->w_oom * (double)g.oom;
    e = e + ap->w_reject * (double)g.rejected;
    const double n = g.admitted > 0 ? (double)g.admitted : 1.0;
    x[i] = e / n - ap->target;
  }
  double nb = b;
  int32_t act = 0;
  if (x[kShort] > 0.0 && x[kShort] > x[kLong]) {
    nb = b - ap->step * b;
    act = -1;
  } else if (x[kLong] > 0.0 && x[kLong] > x[kShort]) {
    nb = b + ap->step * b;
    act = 1;
  }
  if (nb < ap->b_min) nb = ap->b_min;
  if (nb > ap->b_max) nb = ap->b_max;
  *b_short = nb;
  if (action) *action = act;
  return DP_OK;
}
