"""Per-layer report of the multi-layer workloads on the GPU, checked against the oracle.

    python tests/layer_report.py qwen3|sweep-4096|sweep-16384|sweep-65536 [--layers A:B] [--out FILE]

For every layer l of the workload (48 Qwen3-MoE-shaped layers, or 58 DeepSeek-V3-shaped sweep
layers at one T), with the seeded inputs h_{l-1} (the residual stream entering layer l) and the
layer's actual router input H_l = h_{l-1} + residual update:

* the predicted pass on h_{l-1} and the actual pass on H_l through fb_predict_load_packed, with
  their top-k lists and logits;
* the predicted pass against the oracle on every token (tests/parity.py): differing and exempt
  tokens, the count difference from the oracle's histogram (at most 2k per differing token, zero
  when none differs);
* prediction quality on the GPU (Sec. "Metrics" and the prediction-quality study): top-k hit rate
  (fb_topk_hits), hidden-state and logit cosines (fb_row_cosine_mean);
* for every budget of the workload: the device plan of the predicted counts (fb_plan_swaps_device)
  against the oracle's plan, the predicted max/mean before and after, and the realised max/mean of
  the actual counts under pi and under pi' (fb_fold_rank_loads), i.e. whether the plan made from the
  prediction lowered the imbalance the layer really had (the 95% claim of the prediction-quality
  study, and Table 3's max/mean per length).

Writes one JSON document (per-layer records and a summary) and prints one line per layer.  Any
mismatch with the oracle (selection beyond the exemptions, counts, plans) raises.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
for p in (ROOT, HERE):
    if p not in sys.path:
        sys.path.insert(0, p)


def _workload(name):
    from workloads import CONFIGS, sweep_workload
    if name == "qwen3":
        wl = CONFIGS["qwen3"]
        return wl, (wl.budget,)
    if name.startswith("sweep-"):
        wl = sweep_workload(int(name.split("-")[1]))
        return wl, wl.budgets
    raise SystemExit(f"unknown workload {name!r}")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("workload")
    ap.add_argument("--layers", default=None, help="A:B (default: every layer)")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()

    import torch

    import paper_2608_14205_amd as fb
    import parity as P
    from oracle import planner as OPL
    from workloads import contiguous_placement, make_layer

    wl, budgets = _workload(args.workload)
    lo, hi = 0, wl.layers
    if args.layers:
        a, b = args.layers.split(":")
        lo, hi = int(a or 0), int(b or wl.layers)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    slots_d = torch.from_numpy(slots).to(dev)
    e2r_d = torch.from_numpy(e2r).to(dev)
    scoring = fb.Scoring(wl.kind, wl.k, wl.n_group, wl.topk_group, wl.group_topn)
    pred = fb.Predictor(dev)

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    layers = []
    t_start = time.time()
    for layer in range(lo, hi):
        t0 = time.time()
        li = make_layer(wl, layer, with_target=True)
        x, h = up(li.x), up(li.h_target)
        wp = fb.pack_router_weight(up(li.w))
        sb = None if li.select_bias is None else torch.from_numpy(li.select_bias).to(dev)
        p_out = pred.predict_load(x, wp, scoring, e2r_d, wl.R, select_bias=sb, return_topk=True,
                                  return_logits=True)
        a_out = fb.Prediction(torch.empty_like(p_out.counts), torch.empty_like(p_out.rank_loads),
                              torch.empty_like(p_out.max_mean))
        pred.predict_load(h, wp, scoring, e2r_d, wl.R, select_bias=sb, out=a_out, return_topk=True,
                          return_logits=True)
        hits, hit_rate = fb.topk_hits(p_out.topk, a_out.topk, with_rate=True)
        hcos = fb.row_cosine_mean(x, h)
        lcos = fb.row_cosine_mean(p_out.logits, a_out.logits)
        torch.cuda.synchronize()
        counts = p_out.counts.cpu().numpy().astype(np.int64)
        act_counts = a_out.counts.cpu().numpy().astype(np.int64)
        topk = p_out.topk.cpu().numpy()
        assert np.array_equal(counts, np.bincount(topk.reshape(-1), minlength=wl.E)[:wl.E])
        assert np.array_equal(act_counts,
                              np.bincount(a_out.topk.cpu().numpy().reshape(-1), minlength=wl.E)[:wl.E])
        # the predicted pass against the oracle, every token
        st, fails, ref_hist = P.compare_prediction(p_out.logits.cpu().numpy(), topk, li.x, li.w,
                                                   li.select_bias, wl)
        if fails:
            raise AssertionError(f"layer {layer}: {P.summary(st)}\n  " + "\n  ".join(fails[:10]))
        l1 = int(np.abs(counts - ref_hist).sum())
        if l1 > 2 * wl.k * st["mismatch"] or (st["mismatch"] == 0 and l1):
            raise AssertionError(f"layer {layer}: counts differ from the oracle's by {l1}")
        rec = {"layer": layer, "T": wl.T,
               "predicted": {"max_mean": float(p_out.max_mean.item()),
                             "rank_loads": p_out.rank_loads.cpu().numpy().tolist(),
                             "counts": counts.tolist()},
               "actual": {"max_mean": float(a_out.max_mean.item()),
                          "rank_loads": a_out.rank_loads.cpu().numpy().tolist(),
                          "counts": act_counts.tolist()},
               "oracle": {"tokens": st["tokens"], "differing_tokens": st["mismatch"],
                          "exempt_tokens": st["strict_exempt"],
                          "differing_on_gpu_logits": st["mismatch_on_gpu_logits"],
                          "eval_exempt": st["eval_exempt"], "counts_l1": l1,
                          "max_rel_logit_err": st["max_rel_err"]},
               "quality": {"hit_rate": float(hit_rate.item()), "hits": int(hits.item()),
                           "hidden_cosine": float(hcos.item()), "logit_cosine": float(lcos.item())},
               "plans": []}
        counts_d = torch.from_numpy(counts.astype(np.int32)).to(dev)
        act_d = a_out.counts
        for B in budgets:
            dplan = fb.plan_swaps_device(counts_d, slots_d, fb.Budget(B, layer_id=layer))
            r_loads, r_mm = fb.fold_rank_loads(act_d, dplan.expert_to_rank, wl.R)
            got = dplan.to_host()
            ref = OPL.plan_swaps(counts, slots, B, layer_id=layer)
            if [tuple(s) for s in got.swaps] != [tuple(s) for s in ref.swaps] or \
                    not np.array_equal(got.slots, ref.slots):
                raise AssertionError(f"layer {layer} B={B}: device plan differs from the oracle's")
            Lp = got.rank_loads
            rec["plans"].append({
                "budget": B, "swaps": len(got.swaps),
                "moves": [[int(s[4]), int(s[5]), int(s[0]), int(s[1])] for s in got.swaps],
                "predicted_max_mean_after": float(Lp.max() * wl.R / Lp.sum()) if Lp.sum() else 1.0,
                "realised_max_mean_before": rec["actual"]["max_mean"],
                "realised_max_mean_after": float(r_mm.item())})
        layers.append(rec)
        pl = " ".join(f"B{p['budget']}:{p['swaps']}sw {p['realised_max_mean_before']:.3f}->"
                      f"{p['realised_max_mean_after']:.3f}" for p in rec["plans"])
        print(f"[{args.workload}] layer {layer}: pred {rec['predicted']['max_mean']:.3f} actual "
              f"{rec['actual']['max_mean']:.3f} hit {rec['quality']['hit_rate']:.4f} differ "
              f"{st['mismatch']}/{st['tokens']} | {pl} ({time.time() - t0:.1f} s)", flush=True)

    summary = {"workload": args.workload, "T": wl.T, "H": wl.H, "E": wl.E, "k": wl.k,
               "ranks": wl.R, "slots_per_rank": wl.S, "layers": [lo, hi],
               "tokens_compared": int(sum(r["oracle"]["tokens"] for r in layers)),
               "differing_tokens": int(sum(r["oracle"]["differing_tokens"] for r in layers)),
               "mean_hit_rate": float(np.mean([r["quality"]["hit_rate"] for r in layers])),
               "mean_hidden_cosine": float(np.mean([r["quality"]["hidden_cosine"] for r in layers])),
               "mean_logit_cosine": float(np.mean([r["quality"]["logit_cosine"] for r in layers])),
               "mean_predicted_max_mean": float(np.mean([r["predicted"]["max_mean"] for r in layers])),
               "mean_actual_max_mean": float(np.mean([r["actual"]["max_mean"] for r in layers])),
               "budgets": []}
    for i, B in enumerate(budgets):
        ps = [r["plans"][i] for r in layers]
        moving = [p for p in ps if p["swaps"] > 0]
        better = [p for p in moving if p["realised_max_mean_after"] < p["realised_max_mean_before"]]
        summary["budgets"].append({
            "budget": B, "layers_with_swaps": len(moving), "mean_swaps": float(np.mean([p["swaps"] for p in ps])),
            "layers_whose_realised_max_mean_drops": len(better),
            "fraction_of_migrating_layers_improved": (len(better) / len(moving)) if moving else None,
            "mean_realised_max_mean_after": float(np.mean([p["realised_max_mean_after"] for p in ps])),
            "mean_predicted_max_mean_after": float(np.mean([p["predicted_max_mean_after"] for p in ps]))})
    summary["seconds"] = time.time() - t_start
    doc = {"summary": summary, "layers": layers}
    print(json.dumps(summary), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump(doc, f)


if __name__ == "__main__":
    main()
