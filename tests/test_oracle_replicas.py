"""Pins of the replicated-placement oracle (no GPU).

Readings (oracle/replicas.py): slot value e + E * j is replica j of expert e; replica j takes
floor(n_e / c_e) tokens plus one if j < n_e mod c_e; no rank holds two replicas of one expert; the
planner of Sec. "Budgeted Expert-Swap Planning" (Eq. 6-8, Alg. 1) moves replicas with their shares.

Pinned by: hand-worked plans (tests/golden/planner_replicas_hand.json), the shares against a
token-by-token round-robin dispatch, the rank loads against a per-token count, a brute-force greedy
that re-folds the whole slot table for every candidate (no incremental Eq. 6-7 update), the
placement rules after every plan, and the reduction to the pinned planner without replicas.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import planner as PL
from oracle import replicas as RP
from workloads import random_replicated_placement


def _cases(golden_dir):
    with open(os.path.join(golden_dir, "planner_replicas_hand.json")) as f:
        return json.load(f)["cases"]


def test_hand_worked_replicated_plans(golden_dir):
    for c in _cases(golden_dir):
        assert RP.slot_rank_loads(c["counts"], c["slots"]).tolist() == c["loads_before"], c["name"]
        p = PL.plan_swaps(c["counts"], c["slots"], c["max_swaps"], mode=c["mode"])
        assert [list(s) for s in p.swaps] == c["swaps"], c["name"]
        assert p.slots.tolist() == c["new_slots"], c["name"]
        assert p.rank_loads.tolist() == c["rank_loads"], c["name"]
        assert p.loads_before.tolist() == c["loads_before"], c["name"]


@settings(max_examples=200, deadline=None)
@given(st.integers(0, 500), st.integers(1, 9))
def test_shares_follow_round_robin_dispatch(n, c):
    # token t of the expert goes to replica t mod c
    got = [0] * c
    for t in range(n):
        got[t % c] += 1
    assert [RP.replica_share(n, c, j) for j in range(c)] == got


def _random_replicated(g, R, S):
    got = random_replicated_placement(g, R, S)
    if got is None:
        pytest.skip("no valid placement drawn")
    return got


@settings(max_examples=120, deadline=None)
@given(st.integers(1, 4), st.integers(1, 4), st.integers(0, 10 ** 6))
def test_rank_loads_count_every_token_once(R, S, seed):
    g = np.random.default_rng(seed)
    table, E = _random_replicated(g, R, S)
    counts = g.integers(0, 30, size=E)
    # dispatch token by token: the t-th token of expert e goes to its replica t mod c_e
    where = {}
    for r in range(R):
        for v in table[r]:
            if v >= 0:
                where[int(v)] = r
    c = RP.replica_counts(table, E)
    L = [0] * R
    for e in range(E):
        for t in range(int(counts[e])):
            L[where[e + E * (t % c[e])]] += 1
    assert RP.slot_rank_loads(counts, table).tolist() == L


@pytest.mark.parametrize("table,msg", [
    ([[0, 1], [0, -1]], "placed twice"),
    ([[0, 1], [4, -1]], "not 0 .. c - 1"),
    ([[0, 2], [1, -1]], "one rank"),
    ([[0, -1], [-1, -1]], "missing"),
    ([[0, -2], [1, -1]], "invalid"),
])
def test_invalid_replicated_placements_are_refused(table, msg):
    with pytest.raises(ValueError, match=msg):
        RP.replica_counts(table, 2)
    with pytest.raises(ValueError):
        PL.plan_swaps([1, 1], table, 1)


def _brute_force_plan(counts, table, B, mode):
    """The greedy of Alg. 1 from the definitions: every candidate is applied to a copy of the slot
    table, which is checked against the placement rules and folded into loads from scratch."""
    counts = [int(v) for v in counts]
    E = len(counts)
    cur = np.array(table, dtype=np.int64)
    R, S = cur.shape
    V = E * max(RP.replica_counts(cur, E))
    ids = [[int(cur[r, s]) if cur[r, s] >= 0 else V + r * S + s for s in range(S)] for r in range(R)]
    N = sum(counts)
    gam = Fraction(1, N) if N else Fraction(0)
    moved, swaps = set(), []
    while N > 0 and R > 1 and len(swaps) < B:
        L = RP.slot_rank_loads(counts, cur).tolist()
        if max(L) - min(L) <= 0:
            break
        if mode == "frontier":
            pairs = [(L.index(max(L)), L.index(min(L)))]
        else:
            pairs = [(a, b) for a in range(R) for b in range(R) if L[a] > L[b]]
        base = PL.phi(L, gam)
        best = None
        for a, b in pairs:
            for p in range(S):
                for q in range(S):
                    i, j = ids[a][p], ids[b][q]
                    if i in moved or j in moved or (i >= V and j >= V):
                        continue
                    if i < V and j < V and i % E == j % E:
                        continue        # two replicas of one expert are never exchanged
                    t = cur.copy()
                    t[a, p], t[b, q] = cur[b, q], cur[a, p]
                    try:
                        L2 = RP.slot_rank_loads(counts, t)
                    except ValueError:
                        continue        # two replicas of one expert would share a rank
                    d = base - PL.phi(L2.tolist(), gam)
                    if d > 0 and (best is None or (-d, a, b, i, j) < best[0]):
                        best = ((-d, a, b, i, j), a, b, p, q, t, d)
        if best is None:
            break
        _, a, b, p, q, t, d = best
        i, j = ids[a][p], ids[b][q]
        ids[a][p], ids[b][q] = j, i
        moved.update((i, j))
        cur = t
        swaps.append((a, b, p, q, i if i < V else -1, j if j < V else -1, int(d * N)))
    return swaps, cur


@settings(max_examples=150, deadline=None)
@given(st.integers(2, 4), st.integers(1, 3), st.integers(0, 10 ** 6), st.integers(0, 5),
       st.sampled_from(["frontier", "full"]))
def test_planner_matches_brute_force_on_replicated_placements(R, S, seed, B, mode):
    g = np.random.default_rng(seed)
    table, E = _random_replicated(g, R, S)
    counts = g.integers(0, 25, size=E)
    p = PL.plan_swaps(counts, table, B, mode=mode)
    swaps, slots = _brute_force_plan(counts, table, B, mode)
    assert [tuple(s) for s in p.swaps] == swaps
    assert np.array_equal(p.slots, slots)
    # the planner's loads after the plan are the fold of its slot table
    assert p.rank_loads.tolist() == RP.slot_rank_loads(counts, p.slots).tolist()
    # the plan keeps the replica multiset and the placement rules
    assert sorted(v for v in p.slots.reshape(-1) if v >= 0) == \
        sorted(int(v) for v in table.reshape(-1) if v >= 0)
    RP.replica_counts(p.slots, E)
    moved = [v for s in p.swaps for v in (s.expert_src, s.expert_dst) if v >= 0]
    assert len(moved) == len(set(moved))


@settings(max_examples=60, deadline=None)
@given(st.integers(2, 5), st.integers(1, 3), st.integers(0, 10 ** 6), st.integers(0, 5))
def test_placements_without_replicas_read_as_before(R, S, seed, B):
    # every slot value below E: the replica reading is the plain placement (shares are the counts)
    g = np.random.default_rng(seed)
    E = int(g.integers(1, R * S + 1))
    cells = g.permutation(R * S)[:E]
    table = np.full(R * S, -1, np.int64)
    table[cells] = np.arange(E)
    table = table.reshape(R, S)
    counts = g.integers(0, 40, size=E)
    assert RP.replica_counts(table, E) == [1] * E
    e2r = np.empty(E, np.int64)
    for r in range(R):
        for v in table[r]:
            if v >= 0:
                e2r[v] = r
    assert RP.slot_rank_loads(counts, table).tolist() == \
        np.bincount(e2r, weights=counts, minlength=R).astype(np.int64).tolist()


def test_replicating_the_hot_expert_of_a_mixtral_like_placement():
    # One expert per rank plus a spare slot: without replicas no swap can lower the max (the rank
    # holding the hottest expert keeps it).  With the hottest expert replicated into the spare slot
    # of the least loaded rank, the max drops to the larger half of its tokens.
    counts = [40, 12, 10, 9, 8, 7, 6, 4]
    plain = np.array([[e, -1] for e in range(8)])
    assert PL.plan_swaps(counts, plain, 4).swaps == []
    repl = plain.copy()
    repl[7, 1] = 0 + 8 * 1          # replica 1 of expert 0
    L = RP.slot_rank_loads(counts, repl)
    assert L.tolist() == [20, 12, 10, 9, 8, 7, 6, 24]
    p = PL.plan_swaps(counts, repl, 4)
    assert p.rank_loads.max() < L.max()
    assert p.rank_loads.tolist() == RP.slot_rank_loads(counts, p.slots).tolist()
