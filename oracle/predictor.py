"""Oracle of the residual workload predictor (test infrastructure only; see the package docstring).

Follows Sec. "Residual Workload Prediction":

* Eq. 2  early pre-routing logits  G^_l = g_l(h_{l-1});
* Eq. 4  linear router  g_l(X) = X W_l + 1 b_l^T  with W_l in R^{d x E}.  The router weight is
  passed here as ``w`` of shape E x H (row e is column e of W_l), i.e. ``w = W_l^T``;
* the model's own top-k rule applied to G^_l gives the estimated assignments T^_l(i) (Sec.
  "Mixture-of-Expert Architecture": W_l, I_l = topk(G(h_l)));
* Eq. 5  predicted workload  n^_{l,e} = sum_i 1[e in T^_l(i)];
* Alg. 1, the aggregation step under the placement pi_l:  L_r = sum_{e: pi(e) = r} n^_e;
* Sec. "Metrics": max-to-mean rank-load ratio, 1 = perfect balance.

Precision: hidden states and router weights are widened exactly to float64, the contraction is a
float64 GEMM (each bf16 x bf16 product is exact in float64; the sum over H <= 7168 terms is far below a
float32 half-ulp) and the logits are rounded once to float32.  Selection decisions are then taken on
float32 scores, the precision the GPU kernel takes them in.

Routing rules ("the original top-k rule" of the routed model):

* ``softmax``: the routing probabilities are softmax(z) per token; softmax is strictly increasing
  within a row, so the selected set equals the top-k of z (pinned against an explicit float64 softmax
  in the tests).  Renormalising the selected weights changes weights only, never membership, so it
  has no effect on counts.
* ``sigmoid``: score s = sigmoid(z) rounded to float32, plus an optional per-expert selection bias
  added in float32 (DeepSeek-V3 style; the bias steers selection only).
* group-limited selection (``n_group`` > 1): experts are split into ``n_group`` contiguous groups, a
  group's score is the float32 sum of its ``group_topn`` largest scores (largest first), the
  ``topk_group`` best groups are kept (score descending, lower group index first on ties) and the k
  experts are chosen among the kept groups only.  With softmax scoring only the group maximum
  (``group_topn`` = 1) is taken, the one group score that ranks logits and probabilities alike.

Ties between equal float32 scores go to the lower expert index, everywhere.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

SOFTMAX, SIGMOID = "softmax", "sigmoid"


def widen(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored inputs: bf16 bit patterns (uint16) or float32."""
    if dtype == "bf16":
        if a.dtype != np.uint16:
            raise TypeError("bf16 inputs are passed as uint16 bit patterns")
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def router_logits(x: np.ndarray, w: np.ndarray, dtype: str,
                  logit_bias: Optional[np.ndarray] = None, chunk: int = 1024) -> np.ndarray:
    """Eq. 2 / Eq. 4: z = X W + 1 b^T for one token batch, as float32 (T x E).

    ``x`` is T x H, ``w`` is E x H (= W^T).  The float64 product is done in token chunks only to bound
    memory; chunking does not change any value (each row is an independent dot product set).
    """
    T = x.shape[0]
    E = w.shape[0]
    w64 = widen(w, dtype)
    b64 = None if logit_bias is None else np.asarray(logit_bias, np.float32).astype(np.float64)
    out = np.empty((T, E), dtype=np.float32)
    for c0 in range(0, T, chunk):
        z = widen(x[c0:c0 + chunk], dtype) @ w64.T
        if b64 is not None:
            z = z + b64[None, :]
        out[c0:c0 + chunk] = z.astype(np.float32)
    return out


def router_scores(z: np.ndarray, kind: str, select_bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Per-expert selection scores (float32) from float32 logits."""
    z = np.asarray(z, dtype=np.float32)
    if kind == SOFTMAX:
        if select_bias is not None:
            raise ValueError("softmax routing takes no selection bias")
        return z.copy()
    if kind == SIGMOID:
        s = (1.0 / (1.0 + np.exp(-z.astype(np.float64)))).astype(np.float32)
        if select_bias is not None:
            s = (s + np.asarray(select_bias, np.float32)[None, :]).astype(np.float32)
        return s
    raise ValueError(f"unknown scoring kind {kind!r}")


def group_scores(s: np.ndarray, n_group: int, group_topn: int) -> np.ndarray:
    """Score of each contiguous expert group: float32 sum of its ``group_topn`` largest scores,
    accumulated largest first.  Returns T x n_group float32."""
    T, E = s.shape
    if E % n_group != 0:
        raise ValueError("n_group must divide E")
    g = np.sort(s.reshape(T, n_group, E // n_group), axis=-1)[..., ::-1]
    acc = g[..., 0].astype(np.float32)
    for j in range(1, group_topn):
        acc = (acc + g[..., j]).astype(np.float32)
    return acc


def group_keep_mask(s: np.ndarray, n_group: int, topk_group: int, group_topn: int) -> np.ndarray:
    """Boolean T x E mask of the experts that belong to a kept group."""
    T, E = s.shape
    if n_group == 1:
        return np.ones((T, E), dtype=bool)
    gs = group_scores(s, n_group, group_topn)
    gid = np.broadcast_to(np.arange(n_group), gs.shape)
    order = np.lexsort((gid, -gs), axis=-1)          # score descending, then lower group index
    keep_g = np.zeros((T, n_group), dtype=bool)
    np.put_along_axis(keep_g, order[:, :topk_group], True, axis=-1)
    return np.repeat(keep_g, E // n_group, axis=1)


def topk_experts(s: np.ndarray, k: int, allowed: Optional[np.ndarray] = None) -> np.ndarray:
    """T^(i): the k experts with the largest scores, in descending score order, lower index first
    on equal scores; experts outside ``allowed`` are never chosen.  Returns T x k int32."""
    T, E = s.shape
    if not 1 <= k <= E:
        raise ValueError("k must be in [1, E]")
    key = -s.astype(np.float64)
    if allowed is not None:
        if np.any(allowed.sum(axis=1) < k):
            raise ValueError("fewer than k selectable experts")
        key = np.where(allowed, key, np.inf)
    eid = np.broadcast_to(np.arange(E), s.shape)
    order = np.lexsort((eid, key), axis=-1)
    return order[:, :k].astype(np.int32)


def select(z: np.ndarray, k: int, kind: str, select_bias=None, n_group: int = 1,
           topk_group: int = 1, group_topn: int = 1):
    """The routed model's top-k rule on float32 logits.  Returns (topk T x k, scores, allowed).

    Softmax routing with groups scored by the sum of their two best scores is rejected: the
    probabilities' sums do not rank groups like the logits' sums, and a selection computed on logits
    would not be the routed model's.  The group maximum ranks them alike (softmax is monotone)."""
    if kind == SOFTMAX and n_group > 1 and group_topn > 1:
        raise ValueError("softmax routing takes group_topn 1 only")
    s = router_scores(z, kind, select_bias)
    allowed = group_keep_mask(s, n_group, topk_group, group_topn)
    return topk_experts(s, k, allowed if n_group > 1 else None), s, allowed


def expert_histogram(topk: np.ndarray, E: int) -> np.ndarray:
    """Eq. 5: number of tokens whose estimated assignment contains expert e."""
    return np.bincount(np.asarray(topk).reshape(-1), minlength=E).astype(np.int64)[:E]


def rank_loads(counts: np.ndarray, expert_to_rank: np.ndarray, R: int) -> np.ndarray:
    """Alg. 1, second step: L_r = sum of the counts of the experts placed on rank r."""
    e2r = np.asarray(expert_to_rank)
    if np.any((e2r < 0) | (e2r >= R)):
        raise ValueError("rank id out of range")
    L = np.zeros(R, dtype=np.int64)
    for e, c in enumerate(np.asarray(counts)):
        L[e2r[e]] += int(c)
    return L


def max_to_mean(loads: np.ndarray) -> float:
    """max_r L_r / mean_r L_r, mean over all R ranks; 1.0 for an empty batch."""
    L = np.asarray(loads, dtype=np.int64)
    N = int(L.sum())
    if N == 0:
        return 1.0
    return float(L.max()) * L.size / float(N)


def predict_load(x, w, dtype: str, k: int, kind: str, expert_to_rank, R: int,
                 select_bias=None, logit_bias=None, n_group: int = 1, topk_group: int = 1,
                 group_topn: int = 1) -> dict:
    """The whole early pass for one layer: logits, selection, counts, rank loads, max/mean."""
    z = router_logits(x, w, dtype, logit_bias)
    topk, s, allowed = select(z, k, kind, select_bias, n_group, topk_group, group_topn)
    counts = expert_histogram(topk, w.shape[0])
    L = rank_loads(counts, expert_to_rank, R)
    return {"logits": z, "scores": s, "allowed": allowed, "topk": topk, "counts": counts,
            "rank_loads": L, "max_mean": max_to_mean(L)}


def hit_rate(topk_pred: np.ndarray, topk_actual: np.ndarray) -> float:
    """Sec. "Metrics": fraction of the final top-k assignments recovered by the early pass."""
    T, k = topk_actual.shape
    if T == 0:
        return 1.0
    hits = sum(len(set(map(int, a)) & set(map(int, b))) for a, b in zip(topk_pred, topk_actual))
    return hits / float(T * k)


def mean_cosine(a: np.ndarray, b: np.ndarray) -> float:
    """Mean over rows of the cosine similarity between matching rows of a and b (float64)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    num = (a * b).sum(axis=1)
    den = np.linalg.norm(a, axis=1) * np.linalg.norm(b, axis=1)
    return float(np.mean(num / den))
