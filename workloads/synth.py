"""Seeded synthetic prefill workloads.

Every array is drawn from ``numpy.random.Generator(PCG64(SeedSequence([SEED_ROOT, cfg_id, layer,
stream, extra])))`` so that any (workload, layer, stream) can be regenerated on its own.  Streams:

* ``STREAM_ROUTER``  router weight of the layer, N(0, 0.02^2), shape E x H;
* ``STREAM_BIAS``    per-expert selection bias, N(0, 0.01^2) (sigmoid-scored workloads only);
* ``STREAM_CLUSTER`` token -> cluster draw, shared by every layer of a workload (layer slot 0);
* ``STREAM_NOISE``   per-layer hidden-state noise N(0, 1), one generator per 2048-row chunk
  (``extra`` = chunk index + 1);
* ``STREAM_RESID``   per-layer residual update N(0, sigma^2) that turns h_{l-1} into the target
  router input H_l, one generator per chunk like the noise.

The hidden state entering layer l is ``h = 3 * w_l[z_t] + N(0, 1)`` for token cluster ``z_t``, so a
token's own cluster expert gets a large logit and the cluster frequencies (truncated Zipf) become the
routing skew the planner has to fight.  Floating-point draws are made in float32 and, for bfloat16
workloads, stored as bfloat16 bit patterns by round-to-nearest-even.

The module contains no part of the predictor (no logits, scores, selections or counts) and no part of
the planner.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence, Tuple

import numpy as np

SEED_ROOT = 260814205
STREAM_ROUTER, STREAM_BIAS, STREAM_CLUSTER, STREAM_NOISE, STREAM_RESID = range(5)

# Token rows are generated in fixed chunks so that a workload's bytes do not depend on how the caller
# slices it, and so that the 65536 x 7168 sweep layers never need a full float32 copy in memory.
_CHUNK = 2048


def rng(cfg_id: int, layer: int, stream: int, extra: int = 0) -> np.random.Generator:
    """Independent generator for one (workload, layer, stream[, extra]) slot."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [SEED_ROOT, int(cfg_id), int(layer), int(stream), int(extra)])))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bfloat16 (round-to-nearest, ties to even); return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("bf16_bits_from_f32: inputs must be finite")
    u = x.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def truncated_zipf_probs(s: float, K: int) -> np.ndarray:
    """p_i proportional to i^-s for i = 1..K (cluster i-1); defined for any s >= 0."""
    i = np.arange(1, K + 1, dtype=np.float64)
    p = i ** (-float(s))
    return p / p.sum()


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape, routing rule, placement and input recipe of one synthetic prefill workload."""

    name: str
    cfg_id: int
    T: int
    H: int
    E: int
    k: int
    dtype: str                 # "bf16" | "f32": storage and MFMA input type of hidden and router
    kind: str                  # "softmax" | "sigmoid"
    n_group: int = 1           # expert groups for group-limited selection (1 = plain top-k)
    topk_group: int = 1        # groups kept per token
    group_topn: int = 1        # group score = sum of the group's top-n scores
    select_bias: bool = False  # per-expert bias added to the sigmoid score (selection only)
    R: int = 8                 # placement ranks
    S: int = 2                 # expert slots per rank
    budget: int = 1            # swap cap per layer
    sigma: float = 0.3         # residual-update std between h_{l-1} and H_l
    zipf_s: Tuple[float, ...] = (1.2,)   # one exponent, or one per task for a task mixture
    n_clusters: int = 16
    layers: int = 1
    budgets: Tuple[int, ...] = ()        # swap caps reported by the multi-task sweep

    @property
    def experts_per_rank(self) -> int:
        return self.E // self.R

    @property
    def tasks(self) -> int:
        return len(self.zipf_s)

    def with_T(self, T: int) -> "Workload":
        return dataclasses.replace(self, T=int(T))

    def input_bytes(self) -> int:
        b = 2 if self.dtype == "bf16" else 4
        return (self.T * self.H + self.E * self.H) * b


CONFIGS = {
    "tiny": Workload("tiny", 0, T=512, H=1024, E=16, k=2, dtype="f32", kind="softmax",
                     R=8, S=2, budget=2, sigma=0.3, zipf_s=(1.2,), n_clusters=16),
    "mixtral": Workload("mixtral", 1, T=8192, H=4096, E=8, k=2, dtype="bf16", kind="softmax",
                        R=8, S=2, budget=1, sigma=0.3, zipf_s=(1.2,), n_clusters=8),
    "qwen3": Workload("qwen3", 2, T=16384, H=2048, E=128, k=8, dtype="bf16", kind="softmax",
                      R=32, S=4, budget=6, sigma=0.2, zipf_s=(1.0,), n_clusters=128, layers=48),
    "dsv3": Workload("dsv3", 3, T=32768, H=7168, E=256, k=8, dtype="bf16", kind="sigmoid",
                     n_group=8, topk_group=4, group_topn=2, select_bias=True,
                     R=32, S=8, budget=8, sigma=0.25, zipf_s=(1.1,), n_clusters=256),
}


def sweep_workload(T: int) -> Workload:
    """Multi-task skew sweep: DeepSeek-V3 shapes, 4 tasks with Zipf exponents 0.8..1.6 over
    independently permuted clusters, Dirichlet(1) mixing, 58 layers, caps {0, 4, 8, 16}."""
    base = CONFIGS["dsv3"]
    return dataclasses.replace(base, name=f"sweep-T{T}", cfg_id=4, T=int(T), layers=58,
                               zipf_s=tuple(float(s) for s in np.linspace(0.8, 1.6, 4)),
                               budgets=(0, 4, 8, 16), budget=8)


SWEEP_T = (4096, 16384, 65536)


def contiguous_placement(E: int, R: int, S: int) -> Tuple[np.ndarray, np.ndarray]:
    """Rank r holds experts r*epr .. r*epr+epr-1 (epr = E // R) in its first slots; the remaining
    S - epr slots of each rank are empty (-1).  Returns (slot table R x S, expert -> rank)."""
    if E % R != 0:
        raise ValueError("contiguous_placement: E must be a multiple of R")
    epr = E // R
    if epr > S:
        raise ValueError("contiguous_placement: more experts per rank than slots")
    slots = np.full((R, S), -1, dtype=np.int32)
    for r in range(R):
        slots[r, :epr] = np.arange(r * epr, (r + 1) * epr, dtype=np.int32)
    e2r = (np.arange(E, dtype=np.int32) // epr).astype(np.int32)
    return slots, e2r


def random_replicated_placement(g: np.random.Generator, R: int, S: int,
                                max_tries: int = 50) -> Optional[Tuple[np.ndarray, int]]:
    """A random replicated slot table (value e + E * j = replica j of expert e, -1 = empty): a
    random E <= R * S, random extra replicas (at most R per expert), replicas placed on random ranks
    with a free slot and no replica of the same expert.  Returns (table int32 R x S, E), or None if
    no draw succeeds."""
    for _ in range(max_tries):
        E = int(g.integers(1, R * S + 1))
        c = [1] * E
        for _ in range(int(g.integers(0, R * S - E + 1))):
            e = int(g.integers(0, E))
            if c[e] < R:
                c[e] += 1
        items = [(e, j) for e in range(E) for j in range(c[e])]
        g.shuffle(items)
        table = np.full((R, S), -1, dtype=np.int32)
        fill = [0] * R
        holds = [set() for _ in range(R)]
        ok = True
        for e, j in items:
            ranks = [r for r in range(R) if fill[r] < S and e not in holds[r]]
            if not ranks:
                ok = False
                break
            r = ranks[int(g.integers(0, len(ranks)))]
            table[r, fill[r]] = e + E * j
            fill[r] += 1
            holds[r].add(e)
        if ok:
            for r in range(R):
                table[r] = table[r][g.permutation(S)]
            return table, E
    return None


def replicated_placement(popularity: Sequence[float], R: int, S: int) -> np.ndarray:
    """Stand-in for a history-driven placement that replicates hot experts (the starting point of
    the paper's "EPLB + Ours" runs; not that system's algorithm).  ``popularity`` is the expected
    share of tokens of every expert (here the cluster frequencies of the input recipe).  The
    R * S - E spare slots take one extra replica each of the most popular experts (again from the
    top while slots remain, at most R replicas per expert); then the replicas, heaviest first
    (popularity / replicas, ties to the lower expert and ordinal), go to the rank with the least
    popularity placed so far (lowest rank on ties) that has a free slot and no replica of that expert.
    Returns the slot table (value e + E * j = replica j of expert e)."""
    pop = np.asarray(popularity, dtype=np.float64)
    E = pop.size
    if E > R * S:
        raise ValueError("more experts than slots")
    order = sorted(range(E), key=lambda e: (-pop[e], e))
    c = [1] * E
    spare = R * S - E
    while spare > 0 and any(v < R for v in c):
        for e in order:
            if spare == 0:
                break
            if c[e] < R:
                c[e] += 1
                spare -= 1
    items = sorted(((pop[e] / c[e], e, j) for e in range(E) for j in range(c[e])),
                   key=lambda t: (-t[0], t[1], t[2]))
    table = np.full((R, S), -1, dtype=np.int32)
    fill = [0] * R
    placed = [0.0] * R
    holds = [set() for _ in range(R)]
    for w, e, j in items:
        ranks = [r for r in range(R) if fill[r] < S and e not in holds[r]]
        if not ranks:
            raise ValueError("no rank can take the replica")
        r = min(ranks, key=lambda q: (placed[q], q))
        table[r, fill[r]] = e + E * j
        fill[r] += 1
        placed[r] += w
        holds[r].add(e)
    return table


@dataclasses.dataclass
class LayerInputs:
    """One layer's inputs.  ``x`` / ``h_target`` / ``w`` hold bf16 bit patterns (uint16) for bf16
    workloads and float32 values for f32 workloads."""

    x: np.ndarray                    # T x H: residual hidden state h_{l-1}
    w: np.ndarray                    # E x H: router weight of layer l (row e = expert e)
    select_bias: Optional[np.ndarray]  # E float32 or None
    logit_bias: Optional[np.ndarray]   # E float32 or None (the b of the linear router)
    h_target: Optional[np.ndarray]   # T x H: the target router input H_l, or None
    clusters: np.ndarray             # T int32: token cluster ids


def _token_clusters(wl: Workload, T: int) -> np.ndarray:
    g = rng(wl.cfg_id, 0, STREAM_CLUSTER, extra=T)
    K = wl.n_clusters
    if wl.tasks == 1:
        return g.choice(K, size=T, p=truncated_zipf_probs(wl.zipf_s[0], K)).astype(np.int32)
    perms = [g.permutation(K) for _ in range(wl.tasks)]
    mix = g.dirichlet(np.ones(wl.tasks))
    task = g.choice(wl.tasks, size=T, p=mix)
    out = np.empty(T, dtype=np.int32)
    for j in range(wl.tasks):
        sel = np.nonzero(task == j)[0]
        ranks = g.choice(K, size=sel.size, p=truncated_zipf_probs(wl.zipf_s[j], K))
        out[sel] = perms[j][ranks]
    return out


def _store(wl: Workload, a: np.ndarray) -> np.ndarray:
    return bf16_bits_from_f32(a) if wl.dtype == "bf16" else np.ascontiguousarray(a, np.float32)


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover - non-Linux
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def make_layer(wl: Workload, layer: int = 0, with_target: bool = False,
               rows: Optional[Sequence[int]] = None) -> LayerInputs:
    """Generate layer ``layer`` of workload ``wl``.

    Token rows come in chunks of ``_CHUNK`` rows; chunk c draws its hidden-state noise and its
    residual update from generators of their own (``extra`` = c + 1), so chunks are generated
    independently (in parallel threads) and any subset of rows is bit-identical to the full draw.
    ``rows`` restricts the returned hidden states to those token rows (only the chunks holding them
    are generated).
    """
    T, H, E = wl.T, wl.H, wl.E
    w32 = rng(wl.cfg_id, layer, STREAM_ROUTER).normal(0.0, 0.02, size=(E, H)).astype(np.float32)
    sb = None
    if wl.select_bias:
        sb = rng(wl.cfg_id, layer, STREAM_BIAS).normal(0.0, 0.01, size=E).astype(np.float32)
    clusters = _token_clusters(wl, T)
    centers = np.float32(3.0) * w32

    want = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    store_dtype = np.uint16 if wl.dtype == "bf16" else np.float32
    x_out = np.empty((want.size, H), dtype=store_dtype)
    h_out = np.empty((want.size, H), dtype=store_dtype) if with_target else None
    if rows is None:
        chunks = list(range(0, T, _CHUNK))
    else:
        chunks = sorted({int(t) // _CHUNK * _CHUNK for t in want})

    def one(c0: int) -> None:
        c1 = min(T, c0 + _CHUNK)
        cid = c0 // _CHUNK + 1
        h = centers[clusters[c0:c1]] + rng(wl.cfg_id, layer, STREAM_NOISE, cid).standard_normal(
            (c1 - c0, H), dtype=np.float32)
        if with_target:
            upd = rng(wl.cfg_id, layer, STREAM_RESID, cid).standard_normal((c1 - c0, H), dtype=np.float32)
            # sigma = 0 must give H_l identical to h_{l-1} bit for bit (no -0.0 -> +0.0 flips)
            ht = h.copy() if wl.sigma == 0 else h + np.float32(wl.sigma) * upd
        if rows is None:
            x_out[c0:c1] = _store(wl, h)
            if with_target:
                h_out[c0:c1] = _store(wl, ht)
        else:
            sel = np.nonzero((want >= c0) & (want < c1))[0]
            loc = want[sel] - c0
            x_out[sel] = _store(wl, h[loc])
            if with_target:
                h_out[sel] = _store(wl, ht[loc])

    if len(chunks) > 1 and _workers() > 1:
        with ThreadPoolExecutor(max_workers=_workers()) as ex:
            list(ex.map(one, chunks))
    else:
        for c0 in chunks:
            one(c0)
    return LayerInputs(x=x_out, w=_store(wl, w32), select_bias=sb, logit_bias=None,
                       h_target=h_out, clusters=clusters[want] if rows is not None else clusters)
