"""Pins of the adaptive B_short controller (the Sec. 7 future-work direction, this
library's reading of it) and C/Python bit-exact agreement.

The paper prints no value for the controller, so the pins are hand-computed
single steps, its bounds and dead band, and a closed-loop property on a toy
pool whose preemptions are the requests it cannot hold.
"""
import numpy as np
import pytest

from oracle import route

QUIET = (1000, 0, 0, 0)


def test_defaults_follow_the_paper_numbers():
    ap = route.AdaptParams()
    assert ap.target == 0.01                       # Sec. 6: alert above a 1% preemption rate
    assert (ap.b_min, ap.b_max) == (4096.0, 16384.0)  # Sec. 4.6: the 4K-16K plateau


def test_quiet_interval_keeps_the_threshold():
    assert route.adapt_threshold(route.AdaptParams(), [QUIET, QUIET], 8192.0) == (8192.0, 0)


def test_events_inside_the_dead_band_keep_the_threshold():
    ap = route.AdaptParams()
    # 10 preemptions in 1000 admitted = exactly the 1% target: not above it
    assert route.adapt_threshold(ap, [(1000, 10, 0, 0), QUIET], 8192.0) == (8192.0, 0)
    assert route.adapt_threshold(ap, [QUIET, (1000, 5, 2, 3)], 8192.0) == (8192.0, 0)


def test_short_pressure_lowers_by_one_step():
    ap = route.AdaptParams()
    # 8192 - 0.05 * 8192 = 8192 - 409.6 = 7782.4
    assert route.adapt_threshold(ap, [(1000, 30, 0, 0), QUIET], 8192.0) == (7782.4, -1)
    assert route.adapt_threshold(ap, [(1000, 0, 11, 0), QUIET], 8192.0) == (7782.4, -1)   # OOM counts
    assert route.adapt_threshold(ap, [(1000, 0, 0, 11), QUIET], 8192.0) == (7782.4, -1)   # rejections count


def test_long_pressure_raises_by_one_step():
    # 8192 + 409.6 = 8601.6
    assert route.adapt_threshold(route.AdaptParams(), [QUIET, (200, 9, 0, 0)], 8192.0) == (8601.6, 1)


def test_the_more_pressed_pool_wins_and_ties_hold():
    ap = route.AdaptParams()
    assert route.adapt_threshold(ap, [(100, 5, 0, 0), (100, 3, 0, 0)], 8192.0)[1] == -1
    assert route.adapt_threshold(ap, [(100, 3, 0, 0), (100, 5, 0, 0)], 8192.0)[1] == 1
    assert route.adapt_threshold(ap, [(100, 4, 0, 0), (100, 4, 0, 0)], 8192.0) == (8192.0, 0)


def test_zero_admitted_counts_events_per_one_request():
    assert route.adapt_threshold(route.AdaptParams(), [(0, 1, 0, 0), QUIET], 8192.0) == (7782.4, -1)


def test_bounds_are_reached_and_held():
    ap = route.AdaptParams()
    b, steps = 16384.0, 0
    while b > ap.b_min:
        b, _ = route.adapt_threshold(ap, [(10, 5, 0, 0), QUIET], b)
        steps += 1
    # 16384 * 0.95^k > 4096 for k <= 27 (0.95^27 = 0.2503); the 28th step clamps
    assert steps == 28 and b == 4096.0
    assert route.adapt_threshold(ap, [(10, 5, 0, 0), QUIET], b) == (4096.0, -1)
    b = 4096.0
    for _ in range(40):
        b, _ = route.adapt_threshold(ap, [QUIET, (10, 5, 0, 0)], b)
    assert b == 16384.0
    # a threshold set outside the bounds is brought inside even when nothing happens
    assert route.adapt_threshold(ap, [QUIET, QUIET], 65536.0) == (16384.0, 0)


def _closed_loop(b0, short_cap, long_cap, n=10000, steps=200):
    """Toy fleet: each interval routes the same n budgets by the threshold; a pool
    preempts whatever it cannot hold.  Returns the trajectory of B_short."""
    rng = np.random.default_rng(7)
    budgets = np.sort(np.clip(rng.lognormal(np.log(600.0), 1.2, n), 16, 65536) + 256)
    ap = route.AdaptParams()
    b, traj = b0, [b0]

    def signals(b):
        ns = int(np.searchsorted(budgets, b, side="right"))   # budgets <= b go short
        nl = n - ns
        return [(ns, max(0, ns - short_cap), 0, 0), (nl, max(0, nl - long_cap), 0, 0)]

    for _ in range(steps):
        b, _ = route.adapt_threshold(ap, signals(b), b)
        traj.append(b)
    return traj, signals, ap


def _pressure(sig, ap):
    (a, p, o, r) = sig
    return (p + o + r) / max(a, 1) - ap.target


def test_closed_loop_short_overflow_settles_one_step_below_the_crossing():
    traj, signals, ap = _closed_loop(16384.0, short_cap=9600, long_cap=10**9)
    b = traj[-1]
    assert traj[-1] == traj[-2]                           # settled
    assert _pressure(signals(b)[0], ap) <= 0.0            # the short pool now copes
    assert _pressure(signals(b / (1 - ap.step))[0], ap) > 0.0   # one step up it did not
    assert all(x >= y for x, y in zip(traj, traj[1:]))    # monotone descent, no oscillation


def test_closed_loop_long_overflow_raises_until_the_long_pool_copes():
    traj, signals, ap = _closed_loop(4096.0, short_cap=10**9, long_cap=300)
    b = traj[-1]
    assert traj[-1] == traj[-2]
    assert _pressure(signals(b)[1], ap) <= 0.0
    assert _pressure(signals(b / (1 + ap.step))[1], ap) > 0.0
    assert all(x <= y for x, y in zip(traj, traj[1:]))


def test_c_library_matches_oracle_bit_for_bit(host_lib):
    rng = np.random.default_rng(43)
    cp = host_lib.default_adapt_params()
    op = route.AdaptParams()
    assert (cp.w_preempt, cp.w_oom, cp.w_reject, cp.target, cp.step, cp.b_min, cp.b_max) == (
        op.w_preempt, op.w_oom, op.w_reject, op.target, op.step, op.b_min, op.b_max)
    for i in range(3000):
        ap = route.AdaptParams(*(float(x) for x in rng.uniform(0, 3, 3)), float(rng.uniform(0, 0.05)),
                               float(rng.uniform(0.01, 0.5)), 1024.0 * float(rng.integers(1, 5)),
                               1024.0 * float(rng.integers(5, 65)))
        cpar = host_lib.AdaptParams(ap.w_preempt, ap.w_oom, ap.w_reject, ap.target, ap.step, ap.b_min, ap.b_max)
        sig = [tuple(int(x) for x in rng.integers(0, [5000, 200, 20, 50])) for _ in range(2)]
        if i % 7 == 0:
            sig[0] = (0,) + sig[0][1:]
        b = float(rng.uniform(512, 70000))
        assert host_lib.adapt_threshold(cpar, sig[0], sig[1], b) == route.adapt_threshold(ap, sig, b)


@pytest.mark.parametrize("bad", [
    dict(step=0.0), dict(step=1.0), dict(b_min=0.0), dict(b_min=9000.0, b_max=8000.0), dict(target=-0.1),
    dict(w_oom=-1.0), dict(b_max=float("inf")),
])
def test_c_library_rejects_bad_params(host_lib, bad):
    p = host_lib.default_adapt_params()
    for k, v in bad.items():
        setattr(p, k, v)
    with pytest.raises(host_lib.DpoolError) as e:
        host_lib.adapt_threshold(p, QUIET, QUIET, 8192.0)
    assert e.value.code == host_lib.DP_EINVAL


@pytest.mark.parametrize("sig,b", [((QUIET, (-1, 0, 0, 0)), 8192.0), (((10, 0, -2, 0), QUIET), 8192.0),
                                   ((QUIET, QUIET), 0.0), ((QUIET, QUIET), float("nan"))])
def test_c_library_rejects_bad_signals_and_threshold(host_lib, sig, b):
    with pytest.raises(host_lib.DpoolError):
        host_lib.adapt_threshold(host_lib.default_adapt_params(), sig[0], sig[1], b)
