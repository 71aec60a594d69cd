"""Pins of the fleet cost model (Sec. 3) and C/Python bit-exact agreement.

The paper's printed worked examples are checked from tests/golden/.
"""
import numpy as np
import pytest

from oracle import cost


def test_fleet_counts_approach_the_boxed_equation():
    for alpha, ms, ml in ((0.8, 11.2, 2.8), (0.68, 11.2, 2.8), (0.95, 8.0, 1.0), (0.0, 5.0, 2.0), (1.0, 3.0, 3.0)):
        got = cost.savings_fleet(1e12, alpha, ms, ml)
        assert abs(got - cost.savings_formula(alpha, cost.rho(ms, ml))) < 1e-9


def test_short_pool_only_gains_and_alpha_zero_saves_nothing():
    assert cost.savings_formula(0.0, 4.0) == 0.0
    assert cost.savings_formula(0.9, 1.0) == 0.0
    assert cost.g_dual(1000.0, 0.0, 11.2, 2.8) == cost.g_homo(1000.0, 2.8)


def test_c_library_matches_oracle_bit_for_bit(host_lib):
    rng = np.random.default_rng(41)
    cases = [(1000.0, 0.8, 11.2, 2.8), (1000.0, 0.68, 11.2, 2.8), (100.0, 0.7, 2.0, 1.0)]
    cases += [(float(rng.uniform(1, 1e4)), float(rng.random()), float(rng.uniform(0.1, 50)),
               float(rng.uniform(0.1, 50))) for _ in range(2000)]
    for lam, a, ms, ml in cases:
        r = host_lib.cost_model(lam, a, ms, ml)
        assert r.g_homo == cost.g_homo(lam, ml)
        assert r.g_dual == cost.g_dual(lam, a, ms, ml)
        assert r.rho == cost.rho(ms, ml)
        assert r.savings_formula == cost.savings_formula(a, cost.rho(ms, ml))
        assert r.savings_fleet == cost.savings_fleet(lam, a, ms, ml)


@pytest.mark.parametrize("args", [(0.0, 0.5, 1.0, 1.0), (1.0, -0.1, 1.0, 1.0), (1.0, 1.1, 1.0, 1.0),
                                  (1.0, 0.5, 0.0, 1.0), (1.0, 0.5, 1.0, -1.0), (float("nan"), 0.5, 1.0, 1.0)])
def test_c_library_rejects_bad_arguments(host_lib, args):
    with pytest.raises(host_lib.DpoolError):
        host_lib.cost_model(*args)
