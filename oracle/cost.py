"""Oracle of the migration cost model (test infrastructure only; see the package docstring).

Eq. 9: a swap s between ranks a and b costs C(s) = alpha_{a,b} + (S(e_a) + S(e_b)) / beta_{a,b}.
Eq. 10: the planner admits migrations within B_l = max(0, T^attn_{r(l)} - delta).

With a uniform expert size S_e and one link type, every swap costs the same, so the time budget is a
swap count: the largest integer n with n * C <= B_l.  Times are in microseconds, sizes in bytes,
bandwidth in bytes per microsecond.
"""
from __future__ import annotations

import math
from fractions import Fraction


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
