"""Oracle of the migration cost model (test infrastructure only; see the package docstring).

Eq. 9: a swap s between ranks a and b costs C(s) = alpha_{a,b} + (S(e_a) + S(e_b)) / beta_{a,b}.
Eq. 10: the planner admits migrations within B_l = max(0, T^attn_{r(l)} - delta).

With a uniform expert size S_e and one link type, every swap costs the same, so the time budget is a
swap count: the largest integer n with n * C <= B_l.  Times are in microseconds, sizes in bytes,
bandwidth in bytes per microsecond.

For the time-budgeted planner the cost is an exact integer number of nanoseconds: alpha and beta
depend on whether the two ranks share a node (the paper's intra-node and inter-node links), the
transfer term is rounded up so a cost never under-states the time, and an empty slot transfers
nothing (S = 0).
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import NamedTuple, Optional, Sequence


def swap_cost_us(alpha_us: float, beta_bytes_per_us: float, bytes_a: int, bytes_b: int) -> float:
    """Eq. 9."""
    if beta_bytes_per_us <= 0 or alpha_us < 0 or bytes_a < 0 or bytes_b < 0:
        raise ValueError("invalid cost-model parameters")
    return alpha_us + (bytes_a + bytes_b) / beta_bytes_per_us


def window_us(t_attn_us: float, delta_us: float) -> float:
    """Eq. 10."""
    return max(0.0, t_attn_us - delta_us)


def swap_budget(t_attn_us: float, delta_us: float, alpha_us: float, beta_bytes_per_us: float,
                expert_bytes: int) -> int:
    """Number of equal-cost swaps that fit in the attention window."""
    c = swap_cost_us(alpha_us, beta_bytes_per_us, expert_bytes, expert_bytes)
    if c <= 0:
        raise ValueError("swap cost must be positive")
    for v in (t_attn_us, delta_us, alpha_us, beta_bytes_per_us):
        if not math.isfinite(v):
            raise ValueError("non-finite cost-model input")
    # largest n with n * C <= B_l, decided exactly on the two (double) quantities
    return int(math.floor(Fraction(window_us(t_attn_us, delta_us)) / Fraction(c)))


class CostModel(NamedTuple):
    """Migration cost model and time budget of the planner (Eq. 9-10, budgets per rank and link).

    rank_node          node id of every rank; two ranks on the same node use link type 0, else 1
    expert_bytes       S(e) of every expert (bytes transferred when it moves)
    alpha_ns           per-swap overhead (launch, protocol) for link types 0 and 1, in ns (>= 1)
    beta_bytes_per_us  point-to-point bandwidth for link types 0 and 1 (>= 1)
    rank_budget_ns     B_l: transfer time each rank may take part in
    link_budget_ns     transfer time each rank pair may carry; None means rank_budget_ns
    """
    rank_node: Sequence[int]
    expert_bytes: Sequence[int]
    alpha_ns: Sequence[int]
    beta_bytes_per_us: Sequence[int]
    rank_budget_ns: int
    link_budget_ns: Optional[int] = None


def link_type(cm: CostModel, a: int, b: int) -> int:
    return 0 if int(cm.rank_node[a]) == int(cm.rank_node[b]) else 1


def swap_cost_ns(cm: CostModel, a: int, b: int, bytes_a: int, bytes_b: int) -> int:
    """Eq. 9 in whole nanoseconds: alpha + ceil((S(e_a) + S(e_b)) / beta)."""
    t = link_type(cm, a, b)
    alpha, beta = int(cm.alpha_ns[t]), int(cm.beta_bytes_per_us[t])
    if alpha < 1 or beta < 1 or bytes_a < 0 or bytes_b < 0:
        raise ValueError("invalid cost-model parameters")
    return alpha + math.ceil(Fraction((bytes_a + bytes_b) * 1000, beta))
