"""Token-budget routing: Eq. 3-5 and Algorithm 1 (Sec. 2.1-2.2), in IEEE float64.

Test infrastructure only (see the package header).

Steps, in the paper's order:

Route(r, k)                                               (Algorithm 1, Route)
  c*      = c_hat_k - gamma * sigma_k                      (Eq. 5, conservative ratio)
  L_total = ceil(|r| / c*) + max_output_tokens             (Eq. 3, total token budget)
  then the pool: a budget beyond the short pool's C_max (strict >) goes long
  at once; otherwise L_total <= B_short (inclusive) prefers the short pool and
  anything larger the long one; a preferred pool that is overloaded hands the
  request to the other when that one can serve it; a pool whose C_max is below
  L_total is never the answer (the long pool is)
OnResponse(r, k, prompt_tokens)                           (Algorithm 1, OnResponse)
  c_obs   = |r| / prompt_tokens                            (Eq. 4)
  c_hat_k = beta * c_hat_k + (1 - beta) * c_obs            (Eq. 4 EMA, beta = 0.95)
  sigma_k = EMA(sigma_k, |c_obs - c_hat_k|), same beta, using the c_hat_k just updated

Defaults: c0 = 4.0 (cold start), beta = 0.95, gamma = 1.0, B_short = 8192.

Readings where the paper is silent:
  * sigma starts at 0 (its initial value is not given).
  * c* is clamped below at c_min = 1.0 byte/token, so that gamma * sigma >= c_hat
    cannot give a zero or negative ratio.
  * "overloaded" is in_flight >= spill_theta * capacity (the paper names queue
    depth or utilization, without a formula); "the alternate pool can serve r"
    is L_total <= C_max(alternate) and the alternate not overloaded.
  * Each routed request increments the chosen pool's in_flight, so a batch is
    routed sequentially.
  * The feasibility branch returns straight away (no spillover), as the
    algorithm's early return says.
  * (1 - beta) is evaluated at run time (0.050000000000000044 for 0.95).
  * OnResponse with prompt_tokens <= 0 is rejected and changes nothing.

Parity: pinned by hand-computed boundary vectors at cold start (8192 -> short,
8193 -> long), by the closed form of n identical observations
(c_hat_n = c + beta^n (c0 - c), sigma_n = n (1 - beta) beta^n |c0 - c|), and by
the safety invariant (the chosen pool always has C_max >= L_total).

Adaptive B_short (``adapt_threshold``).  Sec. 7 leaves as future work a
threshold that follows runtime signals (preemption rate, OOM events,
rejections) without manual tuning; it gives no rule.  The rule here is this
library's reading, one step per control interval:
  pressure_i = (w_p * preempted_i + w_o * oom_i + w_r * rejected_i) / max(admitted_i, 1)
  excess_i   = pressure_i - target            (i = short, long)
  short excess positive and larger  -> B_short lowered by the fraction step
  long excess positive and larger   -> B_short raised by the fraction step
  otherwise                         -> unchanged;  then clamped to [b_min, b_max]
Defaults: target 0.01 (Sec. 6 alerts on a preemption rate above 1%), step
0.05, bounds 4096..16384 (Sec. 4.6: any B_short in 4K-16K keeps over 80% of
the peak savings), unit weights (the paper does not rank the three signals).
Parity: the paper prints no value for it ("parity unpinned" against the paper);
the pins are hand-computed single steps, the bounds, the dead band, and a
closed-loop property (on a toy pool whose preemptions are its overflow, the
controller settles within one step of the threshold that fills the pool).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

SHORT = 0
LONG = 1


@dataclass
class RouteParams:
    b_short: float = 8192.0
    beta: float = 0.95
    gamma: float = 1.0
    c0: float = 4.0
    c_min: float = 1.0
    spill_theta: float = 1.0


@dataclass
class CatState:
    c_hat: float
    sigma: float


@dataclass
class PoolState:
    c_max: int
    capacity: int
    in_flight: int = 0


def init_categories(params: RouteParams, n_cats: int):
    return [CatState(params.c0, 0.0) for _ in range(n_cats)]


def conservative_ratio(params: RouteParams, cat: CatState) -> float:
    c = cat.c_hat - params.gamma * cat.sigma
    if c < params.c_min:
        c = params.c_min
    return c


def token_budget(req_bytes: int, max_out: int, c_star: float) -> int:
    return int(math.ceil(float(req_bytes) / c_star)) + int(max_out)


def overloaded(params: RouteParams, pool: PoolState) -> bool:
    return float(pool.in_flight) >= params.spill_theta * float(pool.capacity)


def route_one(params: RouteParams, cats, pools, req_bytes: int, cat: int, max_out: int):
    """Algorithm 1 Route for one request; updates pools[chosen].in_flight. Returns (pool, L_total)."""
    c_star = conservative_ratio(params, cats[cat])
    l_total = token_budget(req_bytes, max_out, c_star)
    if l_total > pools[SHORT].c_max:
        # too long for the short pool: only the long pool can take it
        choice = LONG
    else:
        # the token budget decides; an overloaded pool hands the request to
        # the other pool when that pool can hold it and has room
        choice = SHORT if l_total <= params.b_short else LONG
        alt = 1 - choice
        if (overloaded(params, pools[choice]) and l_total <= pools[alt].c_max
                and not overloaded(params, pools[alt])):
            choice = alt
        # never a pool whose C_max is below the request's budget
        if l_total > pools[choice].c_max:
            choice = LONG
    pools[choice].in_flight += 1
    return choice, l_total


def route_requests(params: RouteParams, cats, pools, req_bytes, req_cat, req_max_out):
    out_pool, out_l = [], []
    for b, k, mo in zip(req_bytes, req_cat, req_max_out):
        p, l_total = route_one(params, cats, pools, int(b), int(k), int(mo))
        out_pool.append(p)
        out_l.append(l_total)
    return out_pool, out_l


def on_response(params: RouteParams, cats, cat: int, req_bytes: int, prompt_tokens: int) -> bool:
    """Algorithm 1 OnResponse.  Returns False (state unchanged) when prompt_tokens <= 0."""
    if prompt_tokens <= 0:
        return False
    st = cats[cat]
    c_obs = float(req_bytes) / float(prompt_tokens)
    one_minus_beta = 1.0 - params.beta
    st.c_hat = params.beta * st.c_hat + one_minus_beta * c_obs
    st.sigma = params.beta * st.sigma + one_minus_beta * abs(c_obs - st.c_hat)
    return True


@dataclass
class AdaptParams:
    w_preempt: float = 1.0
    w_oom: float = 1.0
    w_reject: float = 1.0
    target: float = 0.01
    step: float = 0.05
    b_min: float = 4096.0
    b_max: float = 16384.0


def adapt_threshold(ap: AdaptParams, signals, b_short: float):
    """One control step.  signals = [(admitted, preempted, oom, rejected)] * 2 (short, long).

    Returns (new B_short, action) with action -1 lowered, 0 kept, +1 raised.
    """
    excess = []
    for admitted, preempted, oom, rejected in signals:
        events = ap.w_preempt * float(preempted)
        events = events + ap.w_oom * float(oom)
        events = events + ap.w_reject * float(rejected)
        denom = float(admitted) if admitted > 0 else 1.0
        excess.append(events / denom - ap.target)
    xs, xl = excess
    b = float(b_short)
    action = 0
    if xs > 0.0 and xs > xl:
        b = b - ap.step * b
        action = -1
    elif xl > 0.0 and xl > xs:
        b = b + ap.step * b
        action = 1
    b = min(max(b, ap.b_min), ap.b_max)
    return b, action
