"""Oracle of the budgeted expert-swap planner (test infrastructure only; see the package docstring).

Follows Sec. "Budgeted Expert-Swap Planning" and Alg. 1:

* a swap exchanges expert e_a on rank a with expert e_b on rank b and changes only those two rank
  loads: L'_a = L_a - n_{e_a} + n_{e_b},  L'_b = L_b - n_{e_b} + n_{e_a}  (Eq. 6-7);
* a candidate is scored by its reduction of Phi(L) = max_r L_r + gamma * sum_r (L_r - mean L)^2
  (Eq. 8), Delta = Phi(L) - Phi(L'); candidates with Delta <= 0 are discarded;
* candidates are ordered by decreasing benefit-to-cost ratio (a uniform cost under a swap-count
  budget, so by decreasing Delta), ties broken lexicographically by layer id, source rank,
  destination rank and the two logical expert ids;
* a candidate is accepted only if neither expert has been selected already and the budgets allow it;
  loads and residual budgets are updated after every accepted swap;
* in the default frontier mode only experts on the most loaded and the least loaded rank are
  considered; Alg. 1 keeps choosing a positive-benefit swap between a heavier and a lighter rank
  while its loop condition (imbalance above tau) holds and budget remains, and stops when no such
  swap exists.

Readings of points the paper leaves open:

* Iterative reading of Alg. 1: every round re-enumerates and re-scores the candidates at the current
  loads and accepts the best one.  Sorting once up front would let stale scores accept swaps whose
  benefit has become negative.
* The loop condition of Alg. 1 (an imbalance above tau) is read as L_max - L_min > tau (integer
  tokens, default tau = 0).
* gamma is a rational gamma_num / gamma_den (passed as the pair); the default is gamma = 1 / N with
  N = sum of counts.
* The source rank is the more loaded one (its load drops), the destination the less loaded one.
* Frontier ranks: the most loaded rank (lowest rank id on ties) and the least loaded rank (lowest
  rank id on ties).  Full mode considers every ordered pair (a, b) with L_a > L_b.
* Empty slots (-1 in the slot table) are bounded staging space: they take part as virtual items with
  zero load and logical id E + r * S + s, so a "swap" with an empty slot moves one expert.  Two
  empty slots never form a candidate.  Every item (expert or empty slot) moves at most once.
* The per-rank budget (the paper enforces budgets per participant, not only globally) is a cap on the
  number of accepted swaps a rank takes part in; 0 means no per-rank cap.
* The benefit reported for a swap is gamma_den * Delta, an exact integer.

Time-budgeted planning (the cost form of the same section, Eq. 9-10, with the budget enforced per
rank and per link), used when a cost model is given:

* every candidate costs C = alpha + ceil((S(e_a) + S(e_b)) / beta) whole nanoseconds on its link
  (oracle.cost.swap_cost_ns; an empty slot transfers nothing);
* a candidate is admissible only if C fits the remaining budget of both ranks and of their link;
* candidates are ordered by decreasing Delta / C, then by the same lexicographic tie-break;
* after an accepted swap both ranks' and the link's remaining budgets drop by C.
The swap cap and the per-rank cap still apply on top of the time budget.

Replicated placements (oracle.replicas: slot value e + E * j is replica j of expert e): the items are
the replicas with their shares as loads, real items keep their slot value as id and empty slots take
the ids E * J + r * S + s (J = the largest replica count; J = 1 without replicas, which gives the ids
above).  A candidate may not put a replica on a rank that already holds a replica of the same expert
(this also rules out exchanging two replicas of one expert); every replica moves at most once.  Swaps
report slot values, and expert_to_rank gives the rank of replica 0.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, NamedTuple, Optional, Tuple

import numpy as np

from .cost import CostModel, swap_cost_ns
from .replicas import decode, replica_counts, replica_share

FRONTIER, FULL = "frontier", "full"


class Swap(NamedTuple):
    src_rank: int
    dst_rank: int
    src_slot: int
    dst_slot: int
    expert_src: int   # expert leaving the source rank, -1 for an empty slot
    expert_dst: int   # expert leaving the destination rank, -1 for an empty slot
    gain: int         # gamma_den * Delta


class Plan(NamedTuple):
    swaps: List[Swap]
    slots: np.ndarray          # new slot table R x S
    expert_to_rank: np.ndarray
    rank_loads: np.ndarray     # loads after the plan
    loads_before: np.ndarray
    costs: List[int]           # cost of every swap in ns (time-budgeted planning), else empty


def phi(L, gamma: Fraction) -> Fraction:
    """Eq. 8, evaluated literally with exact rationals."""
    L = [Fraction(int(v)) for v in L]
    mean = sum(L, Fraction(0)) / len(L)
    return max(L) + gamma * sum(((v - mean) ** 2 for v in L), Fraction(0))


def plan_swaps(counts, slots, max_swaps: int, *, gamma: Optional[Tuple[int, int]] = None,
               tau: int = 0, mode: str = FRONTIER, per_rank_cap: int = 0,
               layer_id: int = 0, cost: Optional[CostModel] = None) -> Plan:
    counts = [int(c) for c in np.asarray(counts).reshape(-1)]
    E = len(counts)
    table = np.asarray(slots, dtype=np.int64)
    R, S = table.shape
    reps = replica_counts(table, E)
    if max_swaps < 0 or tau < 0 or per_rank_cap < 0:
        raise ValueError("negative budget or threshold")

    # items: slot contents; empty slots become virtual zero-load items with ids E*J + r*S + s
    V = E * max(reps)               # slot values are below V; virtual ids start there
    item = [[int(table[r, s]) if table[r, s] >= 0 else V + r * S + s for s in range(S)]
            for r in range(R)]

    def expert_of(i: int) -> int:
        return decode(i, E)[0] if i < V else -1

    def load_of(i: int) -> int:
        if i >= V:
            return 0
        e, j = decode(i, E)
        return replica_share(counts[e], reps[e], j)

    held = [set(expert_of(i) for i in item[r] if i < V) for r in range(R)]

    L = [sum(load_of(i) for i in item[r]) for r in range(R)]
    before = np.array(L, dtype=np.int64)
    N = sum(L)
    if gamma is None:
        gamma = (1, N) if N > 0 else (0, 1)
    g_num, g_den = int(gamma[0]), int(gamma[1])
    if g_num < 0 or g_den <= 0:
        raise ValueError("gamma must be a non-negative ratio with a positive denominator")
    gamma = Fraction(g_num, g_den)
    moved = set()
    part = [0] * R
    swaps: List[Swap] = []
    costs: List[int] = []
    if cost is not None:
        if len(cost.rank_node) != R or len(cost.expert_bytes) != E:
            raise ValueError("cost model does not match the placement")
        if any(int(v) < 0 for v in cost.expert_bytes) or cost.rank_budget_ns < 0 or \
                (cost.link_budget_ns is not None and cost.link_budget_ns < 0):
            raise ValueError("negative size or budget")
        rank_left = [int(cost.rank_budget_ns)] * R
        link_cap = int(cost.rank_budget_ns if cost.link_budget_ns is None else cost.link_budget_ns)
        link_used = {}

    def bytes_of(i: int) -> int:
        return int(cost.expert_bytes[expert_of(i)]) if i < V else 0

    def lowest_argmax(vals):
        return max(range(len(vals)), key=lambda r: (vals[r], -r))

    def lowest_argmin(vals):
        return min(range(len(vals)), key=lambda r: (vals[r], r))

    active = N > 0 and max_swaps > 0 and R > 1
    while active and len(swaps) < max_swaps:
        a_max, b_min = lowest_argmax(L), lowest_argmin(L)
        if L[a_max] - L[b_min] <= tau:
            break
        if mode == FRONTIER:
            pairs = [(a_max, b_min)]
        elif mode == FULL:
            pairs = [(a, b) for a in range(R) for b in range(R) if L[a] > L[b]]
        else:
            raise ValueError(f"unknown mode {mode!r}")
        phi_now = phi(L, gamma)
        best = None
        for a, b in pairs:
            if per_rank_cap and (part[a] >= per_rank_cap or part[b] >= per_rank_cap):
                continue
            for p in range(S):
                for q in range(S):
                    i, j = item[a][p], item[b][q]
                    if i in moved or j in moved or (i >= V and j >= V):
                        continue
                    if (i < V and expert_of(i) in held[b]) or (j < V and expert_of(j) in held[a]):
                        continue
                    L2 = list(L)
                    L2[a] = L[a] - load_of(i) + load_of(j)     # Eq. 6
                    L2[b] = L[b] - load_of(j) + load_of(i)     # Eq. 7
                    delta = phi_now - phi(L2, gamma)
                    if delta <= 0:
                        continue
                    if cost is None:
                        c, order = 0, -delta
                    else:
                        c = swap_cost_ns(cost, a, b, bytes_of(i), bytes_of(j))
                        link = (min(a, b), max(a, b))
                        if c > rank_left[a] or c > rank_left[b] or \
                                c > link_cap - link_used.get(link, 0):
                            continue
                        order = -(delta / c)
                    rank_key = (order, layer_id, a, b, i, j)
                    if best is None or rank_key < best[0]:
                        best = (rank_key, a, b, p, q, L2, delta, c)
        if best is None:
            break
        _, a, b, p, q, L2, delta, c = best
        i, j = item[a][p], item[b][q]
        item[a][p], item[b][q] = j, i
        for r, gone, came in ((a, i, j), (b, j, i)):
            if gone < V:
                held[r].discard(expert_of(gone))
            if came < V:
                held[r].add(expert_of(came))
        L = L2
        moved.update((i, j))
        part[a] += 1
        part[b] += 1
        g = delta * g_den
        assert g.denominator == 1
        swaps.append(Swap(a, b, p, q, i if i < V else -1, j if j < V else -1, int(g)))
        if cost is not None:
            rank_left[a] -= c
            rank_left[b] -= c
            link = (min(a, b), max(a, b))
            link_used[link] = link_used.get(link, 0) + c
            costs.append(c)

    new_slots = np.array([[i if i < V else -1 for i in row] for row in item], dtype=np.int32)
    e2r = np.empty(E, dtype=np.int32)
    for r in range(R):
        for i in item[r]:
            if i < E:               # replica 0 of expert i
                e2r[i] = r
    return Plan(swaps, new_slots, e2r, np.array(L, dtype=np.int64), before, costs)
