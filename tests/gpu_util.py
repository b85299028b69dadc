"""Helpers of the GPU parity tests: upload seeded inputs, run the HIP path through the C ABI binding,
and compare with the CPU oracle.

Tolerances
----------
* Logits, the bar stated for this path: |z_gpu - z_ref| <= rtol * max_e |z_ref[t, e]| per token
  (row-normalised relative error), rtol = 2e-2 for bf16 inputs and 1e-5 for f32 inputs.
* Logits, a rigorous bound: both sides multiply the same stored values exactly; the GPU sums H
  products in float32 (any order), the oracle in float64 and rounds once.  Recursive summation of n
  terms errs by at most (n - 1) u sum|terms| (u = 2^-24), plus the two final roundings, so
  |z_gpu - z_ref| <= H u sum_h |x_h w_h| + 2 u |z| (+ u |b| for a router bias).
* Selections: a token may differ only if its oracle scores leave a gap smaller than what the logit
  error can close: the k-th vs (k+1)-th selectable score (2 delta_s), and for group-limited routing
  the topk_group-th vs next group score (4 delta_s).  delta_s = delta_z for softmax and
  delta_z / 4 + 2^-20 for sigmoid (sigmoid is 1/4-Lipschitz; 2^-20 covers float32 evaluation of
  the sigmoid and the bias add on both sides).
"""
from __future__ import annotations

import numpy as np
import torch

import paper_2608_14205_amd as fb
from oracle import predictor as OP
from workloads import contiguous_placement

U = 2.0 ** -24


def to_device(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def scoring_of(wl) -> fb.Scoring:
    return fb.Scoring(wl.kind, wl.k, wl.n_group, wl.topk_group, wl.group_topn)


def run_gpu(li, wl, e2r=None, R=None, debug=True, predictor=None, logit_bias=None, packed=False):
    """One prediction through the binding; packed=True packs the router weight first and calls
    fb_predict_load_packed (the launch the benchmark times), else fb_predict_load."""
    if e2r is None:
        _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    R = wl.R if R is None else R
    x = to_device(li.x, wl.dtype)
    w = to_device(li.w, wl.dtype)
    sb = None if li.select_bias is None else torch.from_numpy(li.select_bias).cuda()
    lb = None if logit_bias is None else torch.from_numpy(np.asarray(logit_bias, np.float32)).cuda()
    e2r_t = torch.from_numpy(np.asarray(e2r, np.int32)).cuda()
    pred = predictor or fb.Predictor()
    if packed:
        w = fb.pack_router_weight(w)
    out = pred.predict_load(x, w, scoring_of(wl), e2r_t, R, select_bias=sb, logit_bias=lb,
                            return_topk=debug, return_logits=debug)
    torch.cuda.synchronize()
    res = {"counts": out.counts.cpu().numpy().astype(np.int64),
           "rank_loads": out.rank_loads.cpu().numpy().astype(np.int64),
           "max_mean": float(out.max_mean.cpu().item())}
    if debug:
        res["topk"] = out.topk.cpu().numpy()
        res["logits"] = out.logits.cpu().numpy()
    return res


def logit_bounds(li, wl, rows, logit_bias=None):
    """Rigorous per-element bound on |z_gpu - z_ref| for the given token rows (see module doc)."""
    x = OP.widen(li.x[rows], wl.dtype)
    w = OP.widen(li.w, wl.dtype)
    mag = np.abs(x) @ np.abs(w).T
    z = x @ w.T
    if logit_bias is not None:
        z = z + np.asarray(logit_bias, np.float64)[None, :]
        mag = mag + np.abs(np.asarray(logit_bias, np.float64))[None, :]
    return wl.H * U * mag + 2 * U * np.abs(z) + 1e-30


def selection_gaps(z_ref, wl, select_bias):
    """Per token: the oracle's k-th minus (k+1)-th selectable score, and for group-limited routing the
    topk_group-th minus next group score (inf where undefined)."""
    s = OP.router_scores(z_ref, wl.kind, select_bias).astype(np.float64)
    allowed = OP.group_keep_mask(s.astype(np.float32), wl.n_group, wl.topk_group, wl.group_topn)
    sa = np.sort(np.where(allowed, s, -np.inf), axis=1)[:, ::-1]
    k = wl.k
    gap = np.full(s.shape[0], np.inf)
    if sa.shape[1] > k:
        with np.errstate(invalid="ignore"):
            g = sa[:, k - 1] - sa[:, k]
        gap = np.where(np.isfinite(g), g, np.inf)
    ggap = np.full(s.shape[0], np.inf)
    if wl.n_group > 1 and wl.topk_group < wl.n_group:
        gs = np.sort(OP.group_scores(s.astype(np.float32), wl.n_group, wl.group_topn).astype(np.float64),
                     axis=1)[:, ::-1]
        ggap = gs[:, wl.topk_group - 1] - gs[:, wl.topk_group]
    return gap, ggap


def exempt_tokens(z_ref, wl, select_bias, delta_z):
    """Tokens whose selection may legitimately differ given a per-token logit error delta_z."""
    ds = delta_z if wl.kind == "softmax" else delta_z / 4.0 + 2.0 ** -20
    gap, ggap = selection_gaps(z_ref, wl, select_bias)
    return (gap < 2 * ds) | (ggap < 4 * ds)


def check_prediction(gpu, li, wl, e2r, rows=None, logit_bias=None, label=""):
    """Compare a debug GPU run with the oracle on `rows` (all tokens by default).  Returns stats."""
    T = li.x.shape[0]
    rows = np.arange(T) if rows is None else np.asarray(rows)
    rtol = 2e-2 if wl.dtype == "bf16" else 1e-5
    z_ref = OP.router_logits(li.x[rows], li.w, wl.dtype, logit_bias)
    z_gpu = gpu["logits"][rows]
    row_scale = np.max(np.abs(z_ref.astype(np.float64)), axis=1, keepdims=True)
    err = np.abs(z_gpu.astype(np.float64) - z_ref.astype(np.float64))
    assert np.all(err <= rtol * row_scale + 1e-30), f"{label}: logits beyond the stated tolerance"
    bound = logit_bounds(li, wl, rows, logit_bias)
    assert np.all(err <= bound), f"{label}: logits beyond the summation error bound"

    ref_topk, _, _ = OP.select(z_ref, wl.k, wl.kind, li.select_bias, wl.n_group, wl.topk_group,
                               wl.group_topn)
    g_topk = gpu["topk"][rows]
    same = np.all(np.sort(ref_topk, 1) == np.sort(g_topk, 1), axis=1)
    strict_exempt = exempt_tokens(z_ref, wl, li.select_bias, bound.max(axis=1))
    stated_exempt = exempt_tokens(z_ref, wl, li.select_bias, rtol * row_scale[:, 0])
    bad = ~same & ~strict_exempt
    assert not bad.any(), f"{label}: {bad.sum()} non-exempt tokens select different experts"
    assert not (~same & ~stated_exempt).any()
    # every GPU selection is a valid one: k distinct experts, inside the kept groups
    assert all(len(set(r.tolist())) == wl.k for r in g_topk)
    # the debug list is in descending GPU-score order
    return {"tokens": len(rows), "mismatch": int((~same).sum()), "strict_exempt": int(strict_exempt.sum()),
            "stated_exempt": int(stated_exempt.sum()), "max_rel_err": float((err / row_scale).max())}


def check_counts_consistent(gpu, wl, e2r):
    """Histogram, rank fold and max/mean are exact functions of the GPU's own selections."""
    counts = OP.expert_histogram(gpu["topk"], wl.E)
    assert np.array_equal(gpu["counts"], counts)
    L = OP.rank_loads(counts, e2r, len(gpu["rank_loads"]))
    assert np.array_equal(gpu["rank_loads"], L)
    assert gpu["max_mean"] == OP.max_to_mean(L)
