"""Oracle of replicated placements (test infrastructure only; see the package docstring).

The paper's swaps never create replicas (pairwise exchange keeps one copy of every expert), but its
evaluation also runs FreeBalance on top of a history-driven placement that does replicate hot
experts (the "EPLB + Ours" columns of Table 1).  Replication makes the router divide an expert's
tokens among its copies, a dispatch policy the paper does not spell out.  Readings:

* A slot holds a replica: value v >= 0 is replica j = v // E of expert e = v % E, -1 is an empty
  slot.  A placement without replicas has every v < E, so it reads exactly as before.
* Expert e has c_e >= 1 replicas with ordinals 0 .. c_e - 1, each exactly once, and no rank holds
  two replicas of one expert.
* Dispatch splits the n_e tokens of expert e as evenly as possible: replica j takes
  floor(n_e / c_e) tokens, plus one if j < n_e mod c_e.  The ordinal belongs to the replica and
  moves with it, so a swap changes only the loads of the two ranks it touches (Eq. 6-7 with the
  replica shares in place of n_e).
* The rank load L_r is the sum of the shares on rank r; the max-to-mean ratio is as without
  replicas.
"""
from __future__ import annotations

from typing import List

import numpy as np


def decode(v: int, E: int):
    """Slot value -> (expert, replica ordinal)."""
    return v % E, v // E


def replica_counts(slots, E: int) -> List[int]:
    """c_e of every expert, after checking the placement rules above (ValueError otherwise)."""
    table = np.asarray(slots, dtype=np.int64)
    if table.ndim != 2:
        raise ValueError("slot table must be R x S")
    ordinals = [set() for _ in range(E)]
    for r in range(table.shape[0]):
        on_rank = set()
        for v in table[r]:
            v = int(v)
            if v == -1:
                continue
            if v < 0:
                raise ValueError("slot table holds an invalid value")
            e, j = decode(v, E)
            if j in ordinals[e]:
                raise ValueError("replica placed twice")
            if e in on_rank:
                raise ValueError("two replicas of one expert on one rank")
            ordinals[e].add(j)
            on_rank.add(e)
    c = []
    for e in range(E):
        if not ordinals[e]:
            raise ValueError("expert missing from the slot table")
        if ordinals[e] != set(range(len(ordinals[e]))):
            raise ValueError("replica ordinals of an expert are not 0 .. c - 1")
        c.append(len(ordinals[e]))
    return c


def replica_share(n: int, c: int, j: int) -> int:
    """Tokens replica j of an expert with n tokens and c replicas receives."""
    return n // c + (1 if j < n % c else 0)


def slot_rank_loads(counts, slots) -> np.ndarray:
    """L_r = sum of the replica shares on rank r."""
    counts = [int(v) for v in np.asarray(counts).reshape(-1)]
    E = len(counts)
    c = replica_counts(slots, E)
    table = np.asarray(slots, dtype=np.int64)
    L = np.zeros(table.shape[0], dtype=np.int64)
    for r in range(table.shape[0]):
        for v in table[r]:
            if v >= 0:
                e, j = decode(int(v), E)
                L[r] += replica_share(counts[e], c[e], j)
    return L
