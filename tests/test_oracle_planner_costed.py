"""Pins of the time-budgeted planner oracle (no GPU).

The cost form of Sec. "Budgeted Expert-Swap Planning": every swap costs C = alpha + (S(e_a) +
S(e_b)) / beta on its link (Eq. 9, here in whole nanoseconds, rounded up), the budget B_l of Eq. 10
is enforced per rank and per link, and candidates are ordered by benefit-to-cost ratio.

Pinned by: hand-worked plans (tests/golden/planner_costed_hand.json), the reduction to the pinned
swap-count planner when every swap costs the same (a time budget of m equal costs per rank is a
per-rank cap of m), budgets that are never overrun, costs recomputed from Eq. 9 by hand, and a brute
force over every admissible candidate of the first round.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import planner as PL
from oracle.cost import CostModel


def _cases(golden_dir):
    with open(os.path.join(golden_dir, "planner_costed_hand.json")) as f:
        return json.load(f)["cases"]


def test_hand_worked_costed_plans(golden_dir):
    for c in _cases(golden_dir):
        p = PL.plan_swaps(c["counts"], c["slots"], c["max_swaps"], mode=c["mode"],
                          cost=CostModel(**c["cost"]))
        assert [list(s) for s in p.swaps] == c["swaps"], c["name"]
        assert p.costs == c["costs"], c["name"]
        assert p.slots.tolist() == c["new_slots"], c["name"]
        assert p.rank_loads.tolist() == c["rank_loads"], c["name"]


def _placement(g, R, S, E):
    cells = g.permutation(R * S)[:E]
    slots = np.full(R * S, -1, np.int64)
    slots[cells] = np.arange(E)
    return slots.reshape(R, S)


@settings(max_examples=120, deadline=None)
@given(st.integers(2, 5), st.integers(1, 4), st.integers(0, 10 ** 6), st.integers(0, 6),
       st.sampled_from(["frontier", "full"]), st.integers(1, 3), st.integers(1, 5000))
def test_uniform_cost_is_a_per_rank_cap(R, S, seed, B, mode, m, unit):
    # No empty slots, one node, equal expert sizes: every swap costs the same C, so a time budget
    # of m * C per rank (and per link) admits exactly the plans of the swap-count planner with a
    # per-rank cap of m.
    g = np.random.default_rng(seed)
    E = R * S
    slots = _placement(g, R, S, E)
    counts = g.integers(0, 40, size=E)
    cm = CostModel([0] * R, [unit] * E, (7, 7), (250, 250), 0)
    C = 7 + math.ceil(Fraction(2 * unit * 1000, 250))
    cm = cm._replace(rank_budget_ns=m * C)
    timed = PL.plan_swaps(counts, slots, B, mode=mode, cost=cm)
    capped = PL.plan_swaps(counts, slots, B, mode=mode, per_rank_cap=m)
    assert timed.swaps == capped.swaps
    assert np.array_equal(timed.slots, capped.slots)
    assert timed.costs == [C] * len(timed.swaps)


def _cost_by_hand(cm, a, b, ea, eb):
    t = 0 if cm.rank_node[a] == cm.rank_node[b] else 1
    nbytes = (cm.expert_bytes[ea] if ea >= 0 else 0) + (cm.expert_bytes[eb] if eb >= 0 else 0)
    # alpha + S / beta in ns, with beta in bytes per microsecond, rounded up to a whole ns
    return cm.alpha_ns[t] + -(-nbytes * 1000 // cm.beta_bytes_per_us[t])


def _random_cost_model(g, R, E):
    nodes = g.integers(0, 2, size=R).tolist()
    return CostModel(nodes, g.integers(1, 400, size=E).tolist(),
                     (int(g.integers(1, 50)), int(g.integers(1, 200))),
                     (int(g.integers(100, 2000)), int(g.integers(20, 400))),
                     int(g.integers(0, 12000)),
                     None if g.random() < 0.5 else int(g.integers(0, 12000)))


@settings(max_examples=150, deadline=None)
@given(st.integers(2, 5), st.integers(1, 4), st.integers(0, 10 ** 6), st.integers(0, 6),
       st.sampled_from(["frontier", "full"]))
def test_budgets_hold_and_costs_follow_eq9(R, S, seed, B, mode):
    g = np.random.default_rng(seed)
    E = int(g.integers(R, R * S + 1))
    slots = _placement(g, R, S, E)
    counts = g.integers(0, 50, size=E)
    cm = _random_cost_model(g, R, E)
    p = PL.plan_swaps(counts, slots, B, mode=mode, cost=cm)
    assert len(p.swaps) == len(p.costs) <= B
    spent = [0] * R
    link = {}
    for s, c in zip(p.swaps, p.costs):
        assert c == _cost_by_hand(cm, s.src_rank, s.dst_rank, s.expert_src, s.expert_dst)
        spent[s.src_rank] += c
        spent[s.dst_rank] += c
        key = (min(s.src_rank, s.dst_rank), max(s.src_rank, s.dst_rank))
        link[key] = link.get(key, 0) + c
    cap = cm.rank_budget_ns if cm.link_budget_ns is None else cm.link_budget_ns
    assert max(spent) <= cm.rank_budget_ns
    assert all(v <= cap for v in link.values())
    # every expert is still placed once and moved at most once
    assert sorted(e for e in p.slots.reshape(-1) if e >= 0) == list(range(E))
    moved = [e for s in p.swaps for e in (s.expert_src, s.expert_dst) if e >= 0]
    assert len(moved) == len(set(moved))


def _loads(counts, slots):
    return [sum(int(counts[e]) for e in row if e >= 0) for row in slots]


@settings(max_examples=80, deadline=None)
@given(st.integers(2, 4), st.integers(0, 10 ** 6))
def test_first_swap_has_the_best_ratio(R, seed):
    # Brute force over every ordered rank pair and slot pair: the accepted swap of a one-swap plan
    # in full mode has the largest Delta / C among admissible candidates (Delta from Phi of the
    # resulting slot tables, C by hand).
    g = np.random.default_rng(seed)
    S = 2
    E = R * S - 1
    slots = np.append(np.arange(E), -1)[g.permutation(R * S)].reshape(R, S)
    counts = g.integers(0, 30, size=E)
    cm = _random_cost_model(g, R, E)
    plan = PL.plan_swaps(counts, slots, 1, mode="full", cost=cm)
    N = int(counts.sum())
    gam = Fraction(1, N) if N else Fraction(0)
    L = _loads(counts, slots)
    base = PL.phi(L, gam)
    cap = cm.rank_budget_ns if cm.link_budget_ns is None else cm.link_budget_ns
    best = None
    for a in range(R):
        for b in range(R):
            if not L[a] > L[b]:
                continue
            for p in range(S):
                for q in range(S):
                    if slots[a][p] < 0 and slots[b][q] < 0:
                        continue
                    c = _cost_by_hand(cm, a, b, slots[a][p], slots[b][q])
                    if c > cm.rank_budget_ns or c > cap:
                        continue
                    t = slots.copy()
                    t[a][p], t[b][q] = slots[b][q], slots[a][p]
                    d = base - PL.phi(_loads(counts, t), gam)
                    if d > 0 and (best is None or d / c > best):
                        best = d / c
    if N == 0 or best is None:
        assert plan.swaps == []
        return
    assert len(plan.swaps) == 1
    s = plan.swaps[0]
    t = [list(r) for r in slots]
    t[s.src_rank][s.src_slot], t[s.dst_rank][s.dst_slot] = s.expert_dst, s.expert_src
    d = base - PL.phi(_loads(counts, t), gam)
    assert d / plan.costs[0] == best
