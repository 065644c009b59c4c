"""Edge-side tree shape of the paper (Section IV): the network-aware budget (Eq. 5) and
the geometric-decay branch allocation (Eq. 14), in integers.

The optimum of the weighted log hit-rate under the budget puts F*_k = B_alloc (1 - eta) /
(1 - eta^gamma) eta^k alternative branches at depth k, with eta = alpha^(1 / (beta + 1))
(alpha: main-chain acceptance rate, beta: power-law exponent of the residual tail).  The
paper leaves the rounding open; here the real allocation is rounded by largest remainders
so that the integers sum to B_alloc exactly (ties to the shallower depth, where a branch
is worth more).  These shapes drive the synthetic trees of the verify benchmark; the edge
side itself (drafting, WAN probing) is not part of this library.
"""
from __future__ import annotations

import math
from typing import Callable, List


def decay_factor(alpha: float, beta: float) -> float:
    """eta = alpha^(1 / (beta + 1)), in (0, 1) for alpha in (0, 1) and beta > 0."""
    if not (0.0 < alpha < 1.0) or not beta > 0.0:
        raise ValueError("alpha must be in (0, 1) and beta > 0")
    return alpha ** (1.0 / (beta + 1.0))


def budget(b_max: int, tree_draft_inverse: Callable[[float], float], rtt: float,
           t_verify: float) -> int:
    """B* = min(B_max, floor(T_tree_draft^-1(RTT + T_verify)))."""
    return int(min(b_max, math.floor(tree_draft_inverse(rtt + t_verify))))


def branch_allocation(b_alloc: int, gamma: int, eta: float) -> List[int]:
    """Integer F_0 .. F_{gamma-1} >= 0 summing to b_alloc, closest to the geometric optimum."""
    if gamma < 1 or b_alloc < 0 or not (0.0 < eta <= 1.0):
        raise ValueError("gamma >= 1, b_alloc >= 0 and eta in (0, 1] required")
    if eta == 1.0:
        real = [b_alloc / gamma] * gamma
    else:
        base = b_alloc * (1.0 - eta) / (1.0 - eta ** gamma)
        real = [base * eta ** k for k in range(gamma)]
    f = [int(math.floor(x)) for x in real]
    short = b_alloc - sum(f)
    order = sorted(range(gamma), key=lambda k: (-(real[k] - f[k]), k))
    for k in order[:short]:
        f[k] += 1
    return f
