"""Pins of the swap-planner oracle (no GPU).

Hand-worked plans (tests/golden/planner_hand.json), and properties the paper states or the definitions
imply: the plan never exceeds the budget, never raises the maximum rank load, strictly lowers Phi with
every accepted swap, preserves the slot count of every rank and the total load, moves each expert at
most once, and is a deterministic function of (layer, placement, counts).  The load update of Eq. 6-7
is cross-checked by recomputing rank loads from the resulting slot table.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import planner as PL
from oracle import predictor as P
from workloads import CONFIGS, contiguous_placement, make_layer


def _cases(golden_dir):
    with open(os.path.join(golden_dir, "planner_hand.json")) as f:
        return json.load(f)["cases"]


def _run(c):
    return PL.plan_swaps(c["counts"], c["slots"], c["max_swaps"], mode=c["mode"],
                         per_rank_cap=c.get("per_rank_cap", 0), tau=c.get("tau", 0),
                         gamma=tuple(c["gamma"]) if "gamma" in c else None)


def test_hand_worked_plans(golden_dir):
    for c in _cases(golden_dir):
        p = _run(c)
        assert [list(s) for s in p.swaps] == c["swaps"], c["name"]
        assert p.slots.tolist() == c["new_slots"], c["name"]
        assert p.expert_to_rank.tolist() == c["new_expert_to_rank"], c["name"]
        assert p.rank_loads.tolist() == c["rank_loads"], c["name"]


def _loads_from_slots(counts, slots):
    return [sum(counts[e] for e in row if e >= 0) for row in slots]


def _check_plan(counts, slots, B, plan, gamma=None, per_rank_cap=0):
    counts = list(map(int, counts))
    slots = np.asarray(slots)
    R, S = slots.shape
    N = sum(counts)
    g = Fraction(1, N) if (gamma is None and N) else Fraction(*(gamma or (0, 1)))
    assert len(plan.swaps) <= B
    # Eq. 6-7 load updates agree with the loads of the resulting placement
    assert plan.rank_loads.tolist() == _loads_from_slots(counts, plan.slots)
    assert plan.loads_before.tolist() == _loads_from_slots(counts, slots)
    # slot count per rank preserved (pairwise exchange), every expert still placed exactly once
    assert plan.slots.shape == (R, S)
    assert sorted(e for e in plan.slots.reshape(-1) if e >= 0) == list(range(len(counts)))
    assert all(plan.expert_to_rank[e] == r for r in range(R) for e in plan.slots[r] if e >= 0)
    assert plan.rank_loads.sum() == plan.loads_before.sum() == N
    # replay: every swap strictly lowers Phi and never raises the maximum
    cur = [list(row) for row in slots]
    L = _loads_from_slots(counts, cur)
    moved = []
    part = [0] * R
    for s in plan.swaps:
        assert L[s.src_rank] > L[s.dst_rank]
        assert cur[s.src_rank][s.src_slot] == s.expert_src and cur[s.dst_rank][s.dst_slot] == s.expert_dst
        cur[s.src_rank][s.src_slot], cur[s.dst_rank][s.dst_slot] = s.expert_dst, s.expert_src
        L2 = _loads_from_slots(counts, cur)
        d = PL.phi(L, g) - PL.phi(L2, g)
        assert d > 0 and max(L2) <= max(L)
        assert s.gain == d * (g.denominator if gamma is None else gamma[1])
        moved += [e for e in (s.expert_src, s.expert_dst) if e >= 0]
        part[s.src_rank] += 1
        part[s.dst_rank] += 1
        L = L2
    assert len(moved) == len(set(moved))
    if per_rank_cap:
        assert max(part) <= per_rank_cap
    assert cur == plan.slots.tolist()


placements = st.integers(2, 5).flatmap(lambda R: st.integers(1, 4).flatmap(
    lambda S: st.tuples(st.just(R), st.just(S), st.integers(R, R * S))))


@settings(max_examples=150, deadline=None)
@given(placements, st.integers(0, 10 ** 6), st.integers(0, 5), st.sampled_from(["frontier", "full"]),
       st.integers(0, 2), st.sampled_from([None, (0, 1), (1, 3), (5, 1)]))
def test_plan_properties(shape, seed, B, mode, cap, gamma):
    R, S, E = shape
    g = np.random.default_rng(seed)
    cells = g.permutation(R * S)[:E]
    slots = np.full(R * S, -1, np.int64)
    slots[cells] = np.arange(E)
    slots = slots.reshape(R, S)
    counts = g.integers(0, 50, size=E) * (g.random(E) < 0.8)
    plan = PL.plan_swaps(counts, slots, B, mode=mode, per_rank_cap=cap, gamma=gamma)
    _check_plan(counts, slots, B, plan, gamma=gamma, per_rank_cap=cap)
    again = PL.plan_swaps(counts, slots, B, mode=mode, per_rank_cap=cap, gamma=gamma)
    assert again.swaps == plan.swaps and np.array_equal(again.slots, plan.slots)


@settings(max_examples=60, deadline=None)
@given(st.integers(2, 4), st.integers(0, 10 ** 6))
def test_first_swap_is_the_best_single_swap(R, seed):
    # With B = 1 in full mode the plan is the single swap of largest Delta over every ordered rank
    # pair; brute force over all item pairs, Phi recomputed from the resulting slot table.
    g = np.random.default_rng(seed)
    S = 2
    E = R * S - 1
    slots = np.append(np.arange(E), -1)[g.permutation(R * S)].reshape(R, S)
    counts = g.integers(0, 30, size=E)
    plan = PL.plan_swaps(counts, slots, 1, mode="full")
    N = int(counts.sum())
    gam = Fraction(1, N) if N else Fraction(0)
    base = PL.phi(_loads_from_slots(counts, slots), gam)
    best = Fraction(0)
    for a in range(R):
        for b in range(R):
            for p in range(S):
                for q in range(S):
                    if a == b or (slots[a][p] < 0 and slots[b][q] < 0):
                        continue
                    t = slots.copy()
                    t[a][p], t[b][q] = slots[b][q], slots[a][p]
                    best = max(best, base - PL.phi(_loads_from_slots(counts, t), gam))
    if best > 0:
        assert len(plan.swaps) == 1
        t = [list(r) for r in slots]
        s = plan.swaps[0]
        t[s.src_rank][s.src_slot], t[s.dst_rank][s.dst_slot] = s.expert_dst, s.expert_src
        assert base - PL.phi(_loads_from_slots(counts, t), gam) == best
    else:
        assert plan.swaps == []


def test_layer_id_only_orders_ties():
    c = _cases_by_name()["two-ranks-tie-break"]
    a = PL.plan_swaps(c["counts"], c["slots"], 2, layer_id=0)
    b = PL.plan_swaps(c["counts"], c["slots"], 2, layer_id=57)
    assert a.swaps == b.swaps


def _cases_by_name():
    here = os.path.join(os.path.dirname(__file__), "golden", "planner_hand.json")
    with open(here) as f:
        return {c["name"]: c for c in json.load(f)["cases"]}


def test_mixtral_workload_plan_is_empty():
    # one expert plus one spare slot per rank: no move or swap can lower Phi
    wl = CONFIGS["mixtral"].with_T(2048)
    li = make_layer(wl, 0)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    out = P.predict_load(li.x, li.w, wl.dtype, wl.k, wl.kind, e2r, wl.R)
    for mode in ("frontier", "full"):
        plan = PL.plan_swaps(out["counts"], slots, wl.budget, mode=mode)
        assert plan.swaps == [] and np.array_equal(plan.slots, slots)


def test_dsv3_like_workload_plan_improves_balance():
    wl = CONFIGS["dsv3"].with_T(1024)
    li = make_layer(wl, 0)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    out = P.predict_load(li.x, li.w, wl.dtype, wl.k, wl.kind, e2r, wl.R,
                         select_bias=li.select_bias, n_group=wl.n_group,
                         topk_group=wl.topk_group, group_topn=wl.group_topn)
    plan = PL.plan_swaps(out["counts"], slots, wl.budget)
    _check_plan(out["counts"], slots, wl.budget, plan)
    assert 1 <= len(plan.swaps) <= wl.budget
    assert P.max_to_mean(plan.rank_loads) < P.max_to_mean(plan.loads_before)


def test_degenerate_inputs():
    slots = [[0, 1], [2, 3]]
    assert PL.plan_swaps([0, 0, 0, 0], slots, 4).swaps == []          # empty batch
    assert PL.plan_swaps([5, 1, 1, 1], [[0, 1, 2, 3]], 4).swaps == []  # one rank
    with pytest.raises(ValueError):
        PL.plan_swaps([1, 1, 1, 1], [[0, 1], [1, 3]], 1)            # expert placed twice
    with pytest.raises(ValueError):
        PL.plan_swaps([1, 1, 1, 1], [[0, 1], [2, -1]], 1)           # expert missing
    with pytest.raises(ValueError):
        PL.plan_swaps([1, 1, 1, 1], [[0, 1], [2, 7]], 1)            # bad id
