"""Comparison of one GPU prediction with the CPU oracle (test infrastructure; numpy only).

Used by the GPU parity tests and by ``__graft_entry__.smoke()``.  Given the GPU's debug outputs
(logits T x E and top-k T x k) and the seeded inputs, ``compare_prediction`` checks, token by token:

1. Logits.
   * The stated bar: |z_gpu - z_ref| <= rtol * max_e |z_ref[t, e]| (row-normalised), rtol = 2e-2
     for bf16 inputs, 1e-5 for f32 inputs.
   * A rigorous bound that is far tighter.  Both sides multiply the same stored values exactly.  The
     GPU adds them in float32: MFMA k-steps of 16 bf16 (2 f32) products, one after another, and at
     most four split partial sums.  Any summation tree of depth d errs by at most d u sum|terms|
     (u = 2^-24, first order), and the oracle rounds its float64 sum once, so
     |z_gpu - z_ref| <= d u sum_h |x_h w_h| + 2 u |z| (+ u |b| with a router bias), where
     d = ceil(H / 16) + 16 + 4 (bf16) or ceil(H / 2) + 2 + 4 (f32).
2. The selection rule, exactly, on the GPU's own logits: the oracle's rule applied to z_gpu must
   give the GPU's set for every token.  Softmax selects on the logits themselves, so no token is
   exempt.  Sigmoid scores are evaluated with different exponential and reciprocal routines on the
   two sides (each within 2^-20 of the exact value, the bias add included), so a token is exempt
   from this check only if its gap on z_gpu is below 2 * 2^-20 (k-th vs (k+1)-th selectable score)
   or 4 * 2^-20 (topk_group-th vs next group score).
3. The selection against the oracle on exact logits.  A token may differ only if it is exempt: its
   oracle gap is below what the logit bound delta_z can close, 2 delta_s for experts and 4 delta_s
   for groups (delta_s = delta_z for softmax, delta_z / 4 + 2^-20 for sigmoid, which is
   1/4-Lipschitz).  Every differing token must also be a valid selection within that tolerance:
   k distinct experts; every selected expert's group can be kept (its oracle group score is at
   least the topk_group-th one minus 4 delta_s); at most topk_group groups used, counting the
   groups every perturbation keeps; and no unselected expert of those groups outscores the lowest
   selected one by more than 2 delta_s.
4. Order: the debug list is in descending score order, within 2 * 2^-20 on the GPU's logits and
   within 2 delta_s on the oracle's.

Counts: the GPU's histogram minus the oracle's is exactly the histogram difference of the differing
tokens, so ||n_gpu - n_ref||_1 <= 2 k * #differing, with equality of the vectors when no token
differs (checked by the callers that run every token).
"""
from __future__ import annotations

import numpy as np

from oracle import predictor as OP

U = 2.0 ** -24
EVAL = 2.0 ** -20        # bound on a float32 sigmoid score's evaluation error, bias add included


def sum_depth(H: int, dtype: str) -> int:
    """Depth of the GPU's float32 summation tree for one logit (see the module doc)."""
    return (-(-H // 16) + 16 + 4) if dtype == "bf16" else (-(-H // 2) + 2 + 4)


def logit_bounds(x_rows, w, wl, logit_bias=None, z_ref=None):
    """Rigorous per-element bound on |z_gpu - z_ref| for the given token rows.  With the oracle's
    float32 logits z_ref given, |z| is bounded by |z_ref| / (1 - u) instead of recomputing z."""
    x = OP.widen(x_rows, wl.dtype)
    w64 = OP.widen(w, wl.dtype)
    mag = np.abs(x) @ np.abs(w64).T
    if z_ref is None:
        z = x @ w64.T
        if logit_bias is not None:
            z = z + np.asarray(logit_bias, np.float64)[None, :]
        zabs = np.abs(z)
    else:
        zabs = np.abs(np.asarray(z_ref, np.float64)) * (1.0 + 2.0 ** -22)
    if logit_bias is not None:
        mag = mag + np.abs(np.asarray(logit_bias, np.float64))[None, :]
    return sum_depth(x_rows.shape[1], wl.dtype) * U * mag + 2 * U * zabs + 1e-30


def _gaps(s, wl):
    """Per token: k-th minus (k+1)-th selectable score and topk_group-th minus next group score
    (inf where undefined), from float32 scores s."""
    allowed = OP.group_keep_mask(s, wl.n_group, wl.topk_group, wl.group_topn)
    s64 = s.astype(np.float64)
    sa = np.sort(np.where(allowed, s64, -np.inf), axis=1)[:, ::-1]
    gap = np.full(s.shape[0], np.inf)
    if sa.shape[1] > wl.k:
        with np.errstate(invalid="ignore"):
            g = sa[:, wl.k - 1] - sa[:, wl.k]
        gap = np.where(np.isfinite(g), g, np.inf)
    ggap = np.full(s.shape[0], np.inf)
    if wl.n_group > 1 and wl.topk_group < wl.n_group:
        gs = np.sort(OP.group_scores(s, wl.n_group, wl.group_topn).astype(np.float64), axis=1)[:, ::-1]
        ggap = gs[:, wl.topk_group - 1] - gs[:, wl.topk_group]
    return gap, ggap


def _same_sets(a, b):
    return np.all(np.sort(a, 1) == np.sort(b, 1), axis=1)


def _valid_within(sel, s, ds, wl):
    """Why the selection `sel` of one token is not the exact selection for any scores within ds of
    the oracle scores s (float64), or None if it can be."""
    E, k = s.size, wl.k
    sel = [int(e) for e in sel]
    if len(set(sel)) != k or min(sel) < 0 or max(sel) >= E:
        return f"not {k} distinct experts: {sel}"
    cand = np.ones(E, bool)
    if wl.n_group > 1 and wl.topk_group < wl.n_group:
        gsz = E // wl.n_group
        gs = OP.group_scores(s.astype(np.float32)[None, :], wl.n_group, wl.group_topn)[0].astype(np.float64)
        theta = np.sort(gs)[::-1][wl.topk_group - 1]
        gsel = sorted({e // gsz for e in sel})
        for g in gsel:
            if gs[g] < theta - 4 * ds:
                return f"group {g} (score {gs[g]:.9g}) cannot be kept (threshold {theta:.9g})"
        # groups that every perturbation keeps: fewer than topk_group others can reach them
        sure = [g for g in range(wl.n_group)
                if np.count_nonzero(gs >= gs[g] - 4 * ds) - 1 < wl.topk_group]
        kept = sorted(set(gsel) | set(sure))
        if len(kept) > wl.topk_group:
            return f"groups {kept} exceed the {wl.topk_group} kept"
        cand = np.isin(np.arange(E) // gsz, kept)
    rest = cand.copy()
    rest[sel] = False
    if rest.any():
        lo = s[sel].min()
        hi = s[rest].max()
        if lo < hi - 2 * ds:
            return f"unselected expert {int(np.flatnonzero(rest)[np.argmax(s[rest])])} scores {hi:.9g} > {lo:.9g}"
    return None


def compare_prediction(gpu_logits, gpu_topk, x, w, select_bias, wl, logit_bias=None, chunk=2048):
    """Checks 1-4 of the module doc on every row of x (T x H).  Returns (stats, failures, ref_hist):
    failures lists the violations found (empty when the prediction passes), ref_hist is the
    oracle's expert histogram over these rows."""
    T = x.shape[0]
    rtol = 2e-2 if wl.dtype == "bf16" else 1e-5
    st = {"tokens": int(T), "mismatch": 0, "strict_exempt": 0, "stated_exempt": 0,
          "mismatch_on_gpu_logits": 0, "eval_exempt": 0, "max_rel_err": 0.0, "max_err_over_bound": 0.0}
    fails = []
    ref_hist = np.zeros(wl.E, np.int64)       # the oracle's histogram over the rows
    diff_ref = np.zeros(wl.E, np.int64)       # histogram(gpu) - histogram(oracle) over the rows
    for c0 in range(0, T, chunk):
        c1 = min(T, c0 + chunk)
        z_ref = OP.router_logits(x[c0:c1], w, wl.dtype, logit_bias)
        z_gpu = np.asarray(gpu_logits[c0:c1], np.float32)
        g_topk = np.asarray(gpu_topk[c0:c1])
        # 1. logits
        scale = np.max(np.abs(z_ref.astype(np.float64)), axis=1, keepdims=True)
        err = np.abs(z_gpu.astype(np.float64) - z_ref.astype(np.float64))
        bound = logit_bounds(x[c0:c1], w, wl, logit_bias, z_ref)
        st["max_rel_err"] = max(st["max_rel_err"], float((err / np.maximum(scale, 1e-30)).max()))
        st["max_err_over_bound"] = max(st["max_err_over_bound"], float((err / bound).max()))
        n_tol = int(np.count_nonzero(err > rtol * scale + 1e-30))
        n_bnd = int(np.count_nonzero(err > bound))
        if n_tol:
            fails.append(f"{n_tol} logits beyond the stated tolerance (rows {c0}..{c1})")
        if n_bnd:
            fails.append(f"{n_bnd} logits beyond the summation error bound (rows {c0}..{c1})")
        # 2. the oracle's rule on the GPU's logits
        t_g, s_g, _ = OP.select(z_gpu, wl.k, wl.kind, select_bias, wl.n_group, wl.topk_group,
                                wl.group_topn)
        same_g = _same_sets(t_g, g_topk)
        if wl.kind == "softmax":
            ev_ex = np.zeros(c1 - c0, bool)
        else:
            gap_g, ggap_g = _gaps(s_g, wl)
            ev_ex = (gap_g < 2 * EVAL) | (ggap_g < 4 * EVAL)
        st["mismatch_on_gpu_logits"] += int(np.count_nonzero(~same_g))
        st["eval_exempt"] += int(np.count_nonzero(ev_ex))
        bad_g = np.flatnonzero(~same_g & ~ev_ex)
        if bad_g.size:
            t = int(bad_g[0])
            fails.append(f"{bad_g.size} tokens select differently from the rule on the GPU's own "
                         f"logits (token {c0 + t}: gpu {sorted(g_topk[t].tolist())} rule "
                         f"{sorted(t_g[t].tolist())})")
        # 3. against the oracle on exact logits
        t_r, s_r, _ = OP.select(z_ref, wl.k, wl.kind, select_bias, wl.n_group, wl.topk_group,
                                wl.group_topn)
        same_r = _same_sets(t_r, g_topk)
        dz = bound.max(axis=1)
        ds = dz if wl.kind == "softmax" else dz / 4.0 + EVAL
        gap_r, ggap_r = _gaps(s_r, wl)
        strict = (gap_r < 2 * ds) | (ggap_r < 4 * ds)
        dst = rtol * scale[:, 0]
        dss = dst if wl.kind == "softmax" else dst / 4.0 + EVAL
        stated = (gap_r < 2 * dss) | (ggap_r < 4 * dss)
        st["mismatch"] += int(np.count_nonzero(~same_r))
        st["strict_exempt"] += int(np.count_nonzero(strict))
        st["stated_exempt"] += int(np.count_nonzero(stated))
        nonex = np.flatnonzero(~same_r & ~strict)
        if nonex.size:
            fails.append(f"{nonex.size} non-exempt tokens differ from the oracle (first: token "
                         f"{c0 + int(nonex[0])})")
        s64 = s_r.astype(np.float64)
        for t in np.flatnonzero(~same_r):
            why = _valid_within(g_topk[t], s64[t], float(ds[t]), wl)
            if why:
                fails.append(f"token {c0 + int(t)}: invalid selection: {why}")
        h_r = np.bincount(t_r.reshape(-1), minlength=wl.E)[:wl.E]
        ref_hist += h_r
        diff_ref += np.bincount(g_topk.reshape(-1), minlength=wl.E)[:wl.E] - h_r
        # 4. order of the debug list
        rows = np.arange(c1 - c0)[:, None]
        sg_sel = s_g.astype(np.float64)[rows, g_topk]
        sr_sel = s64[rows, g_topk]
        tol_g = 0.0 if wl.kind == "softmax" else 2 * EVAL
        n_ord_g = int(np.count_nonzero(sg_sel[:, :-1] + tol_g < sg_sel[:, 1:]))
        n_ord_r = int(np.count_nonzero(sr_sel[:, :-1] + 2 * ds[:, None] < sr_sel[:, 1:]))
        if n_ord_g or n_ord_r:
            fails.append(f"debug lists out of descending score order ({n_ord_g} pairs on GPU logits, "
                         f"{n_ord_r} on oracle scores)")
    st["counts_l1_vs_oracle"] = int(np.abs(diff_ref).sum())
    if st["counts_l1_vs_oracle"] > 2 * wl.k * st["mismatch"]:
        fails.append(f"count difference {st['counts_l1_vs_oracle']} exceeds 2k * {st['mismatch']}")
    return st, fails, ref_hist


def summary(st) -> str:
    return (f"{st['tokens']} tokens: {st['mismatch']} differ from the oracle "
            f"({st['strict_exempt']} exempt by the rigorous bound, {st['stated_exempt']} by the "
            f"stated tolerance); {st['mismatch_on_gpu_logits']} differ from the rule on the GPU's "
            f"logits ({st['eval_exempt']} exempt); max row-relative logit error "
            f"{st['max_rel_err']:.2e}, max error / bound {st['max_err_over_bound']:.3f}")
