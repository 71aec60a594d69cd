"""Pins of the oracle's pool sizing (Eq. 1, Eq. 2) and routing (Eq. 3-5, Algorithm 1).

Pool sizing is pinned by the paper's worked MI300X case study (Sec. 4.7) and
its fragmentation estimate (Sec. 3 effect 3), both checked from tests/golden/,
and here by the 8x concurrency ratio of Sec. 1.1; routing by hand-computed
boundary vectors, the closed form of repeated identical observations, and
the algorithm's safety guarantee.
"""
import math

import numpy as np
import pytest

from oracle import pool, route


# ---------------- pool sizing -------------------------------------------------

def test_llama_per_token_and_8x_ratio():
    assert pool.kv_bytes_per_token(80, 8, 128, 2) == 320 * 1024
    ms8 = pool.m_seq(80, 8, 128, 2, 8192)
    ms64 = pool.m_seq(80, 8, 128, 2, 65536)
    n8, n64 = pool.n_seq(288e9, 0.9, 0.0, ms8), pool.n_seq(288e9, 0.9, 0.0, ms64)
    assert (n8, n64) == (96, 12) and n8 == 8 * n64


def test_benchmark_pool_sizes():
    # per-layer share of a KV-only 288 GB GPU, used by the workload configs
    assert pool.size_pool(80, 8, 128, 2, 16, 8192, 288e9, 0.9, 0.0)[3] == 49152
    assert pool.size_pool(80, 8, 128, 2, 16, 65536, 288e9, 0.9, 0.0)[3] == 49152
    assert pool.size_pool(94, 4, 128, 1, 16, 8192, 288e9, 0.9, 0.0)[3] == 167936


def test_nseq_clamps_at_zero_and_blocks():
    assert pool.n_seq(10e9, 0.9, 20e9, 1000) == 0
    assert pool.blocks_per_seq(8192) == 512 and pool.blocks_per_seq(8193) == 513
    assert pool.blocks_for_tokens(0) == 0 and pool.blocks_for_tokens(1) == 1 and pool.blocks_for_tokens(17) == 2


# ---------------- routing -----------------------------------------------------

def fresh(n_cats=1, **kw):
    p = route.RouteParams(**kw)
    cats = route.init_categories(p, n_cats)
    pools = [route.PoolState(8192, 128), route.PoolState(65536, 16)]
    return p, cats, pools


@pytest.mark.parametrize("nbytes,max_out,want_l,want_pool", [
    (32000, 0, 8000, route.SHORT),
    (32772, 0, 8193, route.LONG),        # feasibility: 8193 > C_max(short) = 8192
    (4001, 7191, 8192, route.SHORT),     # inclusive <= B_short
    (4001, 7192, 8193, route.LONG),
    (0, 0, 0, route.SHORT),
    (1, 0, 1, route.SHORT),
    (200 * 4, 8192, 8392, route.LONG),   # short prompt, long generation goes long (Sec. 2.1)
])
def test_cold_start_vectors(nbytes, max_out, want_l, want_pool):
    p, cats, pools = fresh()
    got_pool, got_l = route.route_one(p, cats, pools, nbytes, 0, max_out)
    assert (got_pool, got_l) == (want_pool, want_l)
    assert pools[want_pool].in_flight == 1


def test_ema_closed_form_repeated_observations():
    p, cats, _ = fresh()
    c, c0, beta = 2.5, 4.0, 0.95
    for n in range(1, 201):
        route.on_response(p, cats, 0, 2500, 1000)
        assert abs(cats[0].c_hat - (c + beta ** n * (c0 - c))) < 1e-13
        assert abs(cats[0].sigma - n * (1 - beta) * beta ** n * abs(c0 - c)) < 1e-13


def test_one_observation_values_and_conservative_ratio():
    p, cats, _ = fresh()
    route.on_response(p, cats, 0, 2000, 1000)        # c_obs = 2.0
    # c_hat = 0.95*4 + 0.05*2 = 3.9 ; sigma = 0.05*|2 - 3.9| = 0.095
    assert abs(cats[0].c_hat - 3.9) < 1e-15
    assert abs(cats[0].sigma - 0.095) < 1e-15
    assert abs(route.conservative_ratio(p, cats[0]) - 3.805) < 1e-15


def test_conservative_estimate_biases_borderline_long():
    p, cats, pools = fresh()
    # bytes such that L = 8192 with c_hat but > 8192 with c_hat - sigma
    cats[0].c_hat, cats[0].sigma = 4.0, 0.01
    l_plain = math.ceil(32760 / 4.0)
    assert l_plain <= 8192
    pool_id, l_total = route.route_one(p, cats, pools, 32760, 0, 0)
    assert l_total > 8192 and pool_id == route.LONG


def test_c_star_clamped_at_c_min():
    p, cats, pools = fresh()
    cats[0].c_hat, cats[0].sigma = 2.0, 5.0
    assert route.conservative_ratio(p, cats[0]) == 1.0
    _, l_total = route.route_one(p, cats, pools, 1000, 0, 0)
    assert l_total == 1000


def test_spillover_short_to_long_when_short_overloaded():
    p, cats, pools = fresh()
    pools[0].in_flight = 128                      # at capacity -> overloaded
    got, _ = route.route_one(p, cats, pools, 400, 0, 10)
    assert got == route.LONG


def test_no_spill_when_alternate_also_overloaded():
    p, cats, pools = fresh()
    pools[0].in_flight, pools[1].in_flight = 128, 16
    got, _ = route.route_one(p, cats, pools, 400, 0, 10)
    assert got == route.SHORT


def test_long_to_short_spill_impossible_when_b_short_equals_cmax_short():
    p, cats, pools = fresh()
    pools[1].in_flight = 16
    rng = np.random.default_rng(0)
    for _ in range(2000):
        b = int(rng.integers(0, 300000))
        mo = int(rng.integers(0, 20000))
        got, l_total = route.route_one(p, cats, pools, b, 0, mo)
        if l_total > 8192:
            assert got == route.LONG


def test_long_to_short_spill_when_threshold_below_cmax_short():
    p, cats, pools = fresh(b_short=4096)
    pools[1].in_flight = 16
    got, l_total = route.route_one(p, cats, pools, 4 * 5000, 0, 0)   # 5000 > B_short but fits short
    assert l_total == 5000 and got == route.SHORT


def test_safety_invariant_random():
    rng = np.random.default_rng(1)
    p, cats, pools = fresh(n_cats=3, spill_theta=0.5)
    for i in range(20000):
        k = int(rng.integers(0, 3))
        b = int(rng.integers(0, 400000))
        mo = int(rng.integers(0, 9000))
        got, l_total = route.route_one(p, cats, pools, b, k, mo)
        if l_total <= pools[1].c_max:
            assert l_total <= pools[got].c_max
        if i % 3 == 0:
            route.on_response(p, cats, k, b, max(1, int(b / rng.uniform(1.5, 5.0))))
        if i % 50 == 0:
            pools[0].in_flight = int(rng.integers(0, 200))
            pools[1].in_flight = int(rng.integers(0, 30))


def test_on_response_rejects_nonpositive_tokens():
    p, cats, _ = fresh()
    assert route.on_response(p, cats, 0, 100, 0) is False
    assert route.on_response(p, cats, 0, 100, -5) is False
    assert (cats[0].c_hat, cats[0].sigma) == (4.0, 0.0)


def test_per_category_state_is_separate():
    p, cats, _ = fresh(n_cats=3)
    for _ in range(50):
        route.on_response(p, cats, 1, 2000, 1000)   # CJK-like 2.0 bytes/token
    assert cats[0].c_hat == 4.0 and cats[2].c_hat == 4.0
    assert abs(cats[1].c_hat - (2.0 + 0.95 ** 50 * 2.0)) < 1e-13
