"""Fleet cost model (Sec. 3, "Cost Model: Why Splitting Always Helps"), in IEEE float64.

Test infrastructure only (see the package header).

mu(C_max) is a pool's per-GPU throughput.  A homogeneous fleet at C_max = C_H
serving rate lambda needs G_homo = ceil(lambda / mu(C_H)) GPUs; a dual-pool
fleet whose short pool (C_max = C_S) serves a fraction alpha of the traffic
needs G_dual = ceil(alpha lambda / mu(C_S)) + ceil((1 - alpha) lambda / mu(C_H)).
Without the ceilings the fractional saving is the boxed equation
alpha (1 - 1/rho), rho = mu(C_S) / mu(C_H).

Parity: pinned by the paper's printed numbers: 0.80 x 0.75 = 60% and the
"conservative" 35% (Sec. 3), the model-validation predictions 60.0% and
51.0% with rho = 11.2 / 2.8 = 4.0 from Table 1 (Sec. 4.2), and the 358-GPU
homogeneous fleet at 1,000 req/s of Table 2 (= ceil(1000 / 2.8)); the
ceiling-free limit of the fleet counts is checked against the boxed equation.
"""
from __future__ import annotations

import math


def g_homo(lam: float, mu_long: float) -> int:
    """GPUs of the homogeneous fleet: ceil(lambda / mu(C_H))."""
    return int(math.ceil(lam / mu_long))


def g_dual(lam: float, alpha: float, mu_short: float, mu_long: float) -> int:
    """GPUs of the dual-pool fleet: ceil(alpha lambda / mu(C_S)) + ceil((1 - alpha) lambda / mu(C_H))."""
    return int(math.ceil((alpha * lam) / mu_short)) + int(math.ceil(((1.0 - alpha) * lam) / mu_long))


def rho(mu_short: float, mu_long: float) -> float:
    """Throughput gain ratio mu(C_S) / mu(C_H)."""
    return mu_short / mu_long


def savings_formula(alpha: float, rho_: float) -> float:
    """The boxed equation: Delta G / G_homo = alpha (1 - 1/rho)."""
    return alpha * (1.0 - 1.0 / rho_)


def savings_fleet(lam: float, alpha: float, mu_short: float, mu_long: float) -> float:
    """(G_homo - G_dual) / G_homo with the integer GPU counts."""
    gh = g_homo(lam, mu_long)
    return (gh - g_dual(lam, alpha, mu_short, mu_long)) / gh
