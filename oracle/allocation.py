"""Oracle of the paper's branch allocation (Section IV, Eq. 11-14) -- test infrastructure.

Written from the optimisation it solves: maximise sum_k alpha^k log(alpha + (1 - alpha)
R(F_k)) subject to sum_k F_k = B_alloc, with R(F) ~ 1 - c F^-beta.  The stationarity
condition c beta (1 - alpha) alpha^k F_k^-(beta+1) = lambda gives F_k proportional to
eta^k, eta = alpha^(1/(beta+1)); the budget fixes the scale.  Integer reading (the paper is
silent): largest-remainder rounding of the real optimum, ties to the shallower depth.
"""
from __future__ import annotations

from typing import List

import numpy as np


def real_allocation(b_alloc: float, gamma: int, alpha: float, beta: float) -> np.ndarray:
    """Real optimum: geometric weights alpha^(k/(beta+1)) scaled to sum to b_alloc."""
    weights = np.array([alpha ** (k / (beta + 1.0)) for k in range(gamma)])
    return b_alloc * weights / weights.sum()


def stationarity_multipliers(F: np.ndarray, alpha: float, beta: float, c: float = 1.0):
    """lambda_k = c beta (1 - alpha) alpha^k F_k^-(beta+1): equal for all k at the optimum."""
    k = np.arange(len(F))
    return c * beta * (1.0 - alpha) * alpha ** k * F ** (-(beta + 1.0))


def integer_allocation(real: np.ndarray, b_alloc: int) -> List[int]:
    """Largest remainders: floors, then one more branch at the depths with the largest
    fractional parts (shallower depth first on ties) until the sum is b_alloc."""
    floors = [int(np.floor(x)) for x in real]
    frac = [(float(x) - f, -k) for k, (x, f) in enumerate(zip(real, floors))]
    missing = b_alloc - sum(floors)
    for _, negk in sorted(frac, reverse=True)[:missing]:
        floors[-negk] += 1
    return floors
