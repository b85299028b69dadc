"""A plain CPU model of the full-mode round with stored frontiers, against the oracle (no GPU).

The device planner's full mode on small tables (gamma > 0) scores, per rank pair, only the
candidates on the pair's staircase: with D = L_a - L_b and u = |D + 2d| the benefit (Eq. 8
difference) falls strictly as u grows whatever the other ranks' loads are, so a candidate (u, C, tk)
cannot be a round's best while its pair has an admissible candidate with u' <= u, C' <= C and
(u', C', tk') lexicographically smaller.  The staircase is the lexicographic minimum of (u, C, tk),
then the minimum among the candidates that cost less, and so on; it changes only when a swap touches
one of the pair's ranks.  This model keeps the staircases exactly that way (rebuilt only for the
pairs of the previous swap, at most `cap` points per pair, else every candidate of the pair is
scored) and must give the oracle's plan (Alg. 1 in full mode, Eq. 9 costs, budgets per rank and per
link) on every instance.  It tests the reasoning, not the kernel: the GPU tests compare the kernel
with the host planner and the oracle.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import planner as OP
from oracle.cost import CostModel, swap_cost_ns


def _model_plan(counts, slots, max_swaps, gamma, tau, per_rank_cap, cost, cap):
    counts = [int(c) for c in counts]
    E = len(counts)
    R, S = slots.shape
    V = E
    item = [[int(slots[r, s]) if slots[r, s] >= 0 else V + r * S + s for s in range(S)]
            for r in range(R)]

    def load(i):
        return counts[i] if i < V else 0

    L = [sum(load(i) for i in item[r]) for r in range(R)]
    N = sum(L)
    g_num, g_den = gamma if gamma is not None else (1, N) if N > 0 else (0, 1)
    assert g_num > 0
    moved = [[False] * S for _ in range(R)]
    part = [0] * R
    if cost is not None:
        rank_left = [cost.rank_budget_ns] * R
        link_cap = cost.rank_budget_ns if cost.link_budget_ns is None else cost.link_budget_ns
        link_used = {}

    def setup(x, y):
        if L[x] == L[y]:
            return None
        ra, rb = (x, y) if L[x] > L[y] else (y, x)
        if per_rank_cap and (part[ra] >= per_rank_cap or part[rb] >= per_rank_cap):
            return None
        return ra, rb

    def cand(ra, rb, p, q):
        i, j = item[ra][p], item[rb][q]
        if moved[ra][p] or moved[rb][q] or (i >= V and j >= V):
            return None
        d = load(j) - load(i)
        u = abs(L[ra] - L[rb] + 2 * d)
        c = 1
        if cost is not None:
            c = swap_cost_ns(cost, ra, rb, int(cost.expert_bytes[i]) if i < V else 0,
                             int(cost.expert_bytes[j]) if j < V else 0)
            link = (min(ra, rb), max(ra, rb))
            if c > rank_left[ra] or c > rank_left[rb] or c > link_cap - link_used.get(link, 0):
                return None
        return u, c, (ra, rb, i, j), d

    stairs = {}

    def rebuild(x, y):
        st = setup(x, y)
        stairs[(x, y)] = []
        if st is None:
            return
        keys = {}
        for p in range(S):
            for q in range(S):
                k = cand(st[0], st[1], p, q)
                if k is not None:
                    keys[(p, q)] = k
        out, limit = [], None
        while True:
            pool = [pq for pq in keys if limit is None or keys[pq][1] < limit]
            if not pool:
                break
            if len(out) == cap:
                stairs[(x, y)] = "all"
                return
            w = min(pool, key=lambda pq: keys[pq][:3])
            out.append(w)
            limit = keys[w][1]
        stairs[(x, y)] = out

    pairs = [(x, y) for y in range(R) for x in range(y)]
    swaps, last = [], None
    while len(swaps) < max_swaps and N > 0 and R > 1:
        amax = max(range(R), key=lambda r: (L[r], -r))
        amin = min(range(R), key=lambda r: (L[r], r))
        if L[amax] - L[amin] <= tau:
            break
        for pr in pairs if last is None else [pr for pr in pairs if pr[0] in last or pr[1] in last]:
            rebuild(*pr)
        M, best = L[amax], None
        for (x, y) in pairs:
            pts = stairs[(x, y)]
            if not pts:
                continue
            ra, rb = setup(x, y)
            others = [L[r] for r in range(R) if r != ra and r != rb]
            if pts == "all":
                pts = [(p, q) for p in range(S) for q in range(S)]
            for p, q in pts:
                k = cand(ra, rb, p, q)
                if k is None:
                    continue
                u, c, tk, d = k
                m2 = max([L[ra] + d, L[rb] - d] + others)
                gain = g_den * (M - m2) + g_num * 2 * d * (L[rb] - L[ra] - d)
                if gain <= 0:
                    continue
                key = (-Fraction(gain, c), tk)
                if best is None or key < best[0]:
                    best = (key, ra, rb, p, q, d, gain, c)
        if best is None:
            break
        _, ra, rb, p, q, d, gain, c = best
        i, j = item[ra][p], item[rb][q]
        item[ra][p], item[rb][q] = j, i
        moved[ra][p] = moved[rb][q] = True
        L[ra] += d
        L[rb] -= d
        part[ra] += 1
        part[rb] += 1
        if cost is not None:
            rank_left[ra] -= c
            rank_left[rb] -= c
            link = (min(ra, rb), max(ra, rb))
            link_used[link] = link_used.get(link, 0) + c
        swaps.append((ra, rb, p, q, i if i < V else -1, j if j < V else -1, gain))
        last = (ra, rb)
    return swaps


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_stored_frontier_model_gives_the_oracle_plan(seed):
    g = np.random.default_rng(seed)
    for it in range(70):
        R = int(g.integers(2, 8))
        S = int(g.integers(1, 5))
        E = int(g.integers(max(1, R * S // 2), R * S + 1))
        t = np.full(R * S, -1, np.int64)
        t[g.permutation(R * S)[:E]] = np.arange(E)
        slots = t.reshape(R, S)
        counts = g.integers(0, [5, 50, 1000][it % 3], E)
        if it % 7 == 0:
            counts = np.full(E, 3)                  # many equal benefits: the tie keys decide
        gamma = [None, (1, 3), (2, 5)][it % 3]
        cap_, tau, B = int(g.integers(0, 3)), int(g.integers(0, 2)), int(g.integers(1, 10))
        cost = None
        if it % 2:
            sizes = g.integers(0, 5, E) * 1000 if it % 4 == 1 else np.full(E, 2000)
            link = None if g.random() < 0.5 else int(g.integers(1000, 12000))
            cost = CostModel(list(g.integers(0, 2, R)), list(sizes), [3, 7], [1000, 500],
                             int(g.integers(2000, 20000)), link)
        ref = OP.plan_swaps(counts, slots, B, gamma=gamma, tau=tau, mode="full",
                            per_rank_cap=cap_, cost=cost)
        # cap 1 forces the pairs with longer staircases to be scored in full
        got = _model_plan(counts, slots, B, gamma, tau, cap_, cost, cap=1 if it % 5 == 0 else 8)
        want = [(s.src_rank, s.dst_rank, s.src_slot, s.dst_slot, s.expert_src, s.expert_dst, s.gain)
                for s in ref.swaps]
        assert got == want, (seed, it)
