"""Helpers of the GPU parity tests: upload seeded inputs, run the HIP path through the C ABI binding,
and compare with the CPU oracle (the comparison rules are in tests/parity.py).

Every comparison's statistics are printed and, when the environment variable FB_PARITY_LOG names a
file, appended to it as one JSON line, so the counts of differing and exempt tokens are kept.
"""
from __future__ import annotations

import json
import os

import numpy as np
import torch

import paper_2608_14205_amd as fb
import parity as P
from oracle import predictor as OP
from workloads import contiguous_placement

# stated ceilings: tokens that may differ from the oracle (each one exempt and valid), and tokens
# exempt from the exact rule on the GPU's own logits (sigmoid evaluation near-ties)
MAX_MISMATCH_FRAC = 2e-3
MAX_EVAL_EXEMPT_FRAC = 1e-3


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


def record(label: str, stats: dict) -> None:
    """Print the statistics of one comparison and append them to $FB_PARITY_LOG, if set."""
    print(f"[parity] {label}: {stats}", flush=True)
    path = os.environ.get("FB_PARITY_LOG")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps({"label": label, **stats}) + "\n")


def check_prediction(gpu, li, wl, e2r, rows=None, logit_bias=None, label=""):
    """Compare a debug GPU run with the oracle on `rows` (all tokens by default): the checks of
    tests/parity.py, with the counts of differing and exempt tokens in every message, and the
    stated ceilings on both.  With every row compared, the GPU's counts are also compared with the
    oracle's histogram: equal when no token differs, else within 2k per differing token.  Returns
    the statistics."""
    T = li.x.shape[0]
    rows = np.arange(T) if rows is None else np.asarray(rows)
    st, fails, ref_hist = P.compare_prediction(gpu["logits"][rows], gpu["topk"][rows], li.x[rows],
                                               li.w, li.select_bias, wl, logit_bias)
    msg = f"{label}: {P.summary(st)}"
    assert not fails, msg + "\n  " + "\n  ".join(fails[:10])
    n = st["tokens"]
    assert st["mismatch"] <= max(2, MAX_MISMATCH_FRAC * n), msg + " (above the differing-token ceiling)"
    assert st["eval_exempt"] <= max(2, MAX_EVAL_EXEMPT_FRAC * n), msg + " (above the exemption ceiling)"
    if rows.size == T:
        l1 = int(np.abs(gpu["counts"] - ref_hist).sum())
        st["counts_l1_vs_oracle"] = l1
        assert l1 <= 2 * wl.k * st["mismatch"], msg + f" (counts differ from the oracle's by {l1})"
        if st["mismatch"] == 0:
            assert np.array_equal(gpu["counts"], ref_hist), msg
    record(label, st)
    return st


def check_counts_consistent(gpu, wl, e2r):
    """Histogram, rank fold and max/mean are exact functions of the GPU's own selections."""
    counts = OP.expert_histogram(gpu["topk"], wl.E)
    assert np.array_equal(gpu["counts"], counts)
    L = OP.rank_loads(counts, e2r, len(gpu["rank_loads"]))
    assert np.array_equal(gpu["rank_loads"], L)
    assert gpu["max_mean"] == OP.max_to_mean(L)
