"""Device prediction-quality diagnostics (hit rate, row cosines, rank fold) against the oracle, on
MI355X.  The inputs are the GPU's own predicted and actual passes, so the comparison isolates the
diagnostics: hits and folds must be exact, cosines equal the oracle's float64 values to 1e-12."""
import numpy as np
import pytest
import torch

import paper_2608_14205_amd as fb
from oracle import planner as OPL
from oracle import predictor as OP
from workloads import CONFIGS, contiguous_placement, make_layer, sweep_workload
from gpu_util import scoring_of, to_device

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _passes(wl, layer, T=None):
    wl = wl if T is None else wl.with_T(T)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, layer, with_target=True)
    x, h, w = to_device(li.x, wl.dtype), to_device(li.h_target, wl.dtype), to_device(li.w, wl.dtype)
    sb = None if li.select_bias is None else torch.from_numpy(li.select_bias).cuda()
    e2r_t = torch.from_numpy(e2r).cuda()
    pred = fb.Predictor()
    wp = fb.pack_router_weight(w)
    p = pred.predict_load(x, wp, scoring_of(wl), e2r_t, wl.R, select_bias=sb, return_topk=True,
                          return_logits=True)
    a = fb.Predictor().predict_load(h, wp, scoring_of(wl), e2r_t, wl.R, select_bias=sb,
                                    return_topk=True, return_logits=True)
    torch.cuda.synchronize()
    return wl, li, slots, e2r, x, h, p, a


@pytest.mark.parametrize("name,layer,T", [("dsv3", 0, 4096), ("qwen3", 5, 3000), ("tiny", 0, None),
                                          ("sweep", 12, 4096)])
def test_quality_metrics_match_oracle(name, layer, T):
    _say(f"[quality] {name} layer {layer}")
    wl0 = sweep_workload(4096) if name == "sweep" else CONFIGS[name]
    wl, li, slots, e2r, x, h, p, a = _passes(wl0, layer, T)
    q = fb.prediction_quality(p, a, x, h)
    tp, ta = p.topk.cpu().numpy(), a.topk.cpu().numpy()
    hits_ref = sum(len(set(r.tolist()) & set(s.tolist())) for r, s in zip(tp, ta))
    assert q.hits == hits_ref
    assert q.hit_rate == OP.hit_rate(tp, ta)
    lc_ref = OP.mean_cosine(p.logits.cpu().numpy(), a.logits.cpu().numpy())
    hc_ref = OP.mean_cosine(OP.widen(li.x, wl.dtype), OP.widen(li.h_target, wl.dtype))
    assert q.logit_cosine == pytest.approx(lc_ref, rel=1e-12, abs=1e-12)
    assert q.hidden_cosine == pytest.approx(hc_ref, rel=1e-12, abs=1e-12)
    assert 0.0 <= q.hit_rate <= 1.0 and -1.0 <= q.logit_cosine <= 1.0
    _say(f"[quality] {name}: hit rate {q.hit_rate:.4f}, logit cosine {q.logit_cosine:.4f}, "
         f"hidden cosine {q.hidden_cosine:.4f}")

    # realised balance of the actual routing under the old and the planned placement
    plan = fb.plan_swaps_device(p.counts, torch.from_numpy(slots).cuda(), fb.Budget(wl.budget)).to_host()
    for placement in (e2r, plan.expert_to_rank):
        loads, mm = fb.fold_rank_loads(a.counts, torch.from_numpy(np.ascontiguousarray(placement, np.int32)).cuda(),
                                       wl.R)
        ref = OP.rank_loads(a.counts.cpu().numpy(), placement, wl.R)
        assert np.array_equal(loads.cpu().numpy(), ref)
        assert float(mm.item()) == OP.max_to_mean(ref)


def test_identical_passes_are_perfect():
    """sigma = 0: the early pass is the actual pass, so hits = T k and both cosines are 1."""
    import dataclasses
    wl = dataclasses.replace(CONFIGS["dsv3"].with_T(1000), sigma=0.0)
    _, li, _, _, x, h, p, a = _passes(wl, 3)
    q = fb.prediction_quality(p, a, x, h)
    assert q.hits == 1000 * wl.k and q.hit_rate == 1.0
    assert q.logit_cosine == pytest.approx(1.0, abs=1e-12)
    assert q.hidden_cosine == pytest.approx(1.0, abs=1e-12)


def test_hits_edge_cases():
    _say("[quality] hit edge cases")
    empty = torch.empty((0, 4), dtype=torch.int32, device="cuda")
    h0, r0 = fb.topk_hits(empty, empty, with_rate=True)
    assert int(h0.item()) == 0 and float(r0.item()) == 1.0
    g = np.random.default_rng(7)
    T, k = 777, 32
    tp = np.stack([g.permutation(256)[:k] for _ in range(T)]).astype(np.int32)
    ta = np.stack([g.permutation(256)[:k] for _ in range(T)]).astype(np.int32)
    hits, rate = fb.topk_hits(torch.from_numpy(tp).cuda(), torch.from_numpy(ta).cuda(), with_rate=True)
    ref = sum(len(set(r.tolist()) & set(s.tolist())) for r, s in zip(tp, ta))
    assert int(hits.item()) == ref
    # the oracle's hit rate on the same lists (Sec. "Metrics")
    assert float(rate.item()) == OP.hit_rate(tp, ta)


@pytest.mark.parametrize("rows,cols,dtype", [(1, 8, "bf16"), (3, 4, "f32"), (5000, 7168, "bf16"),
                                             (4097, 256, "f32")])
def test_cosine_shapes(rows, cols, dtype):
    _say(f"[quality] cosine {rows}x{cols} {dtype}")
    g = np.random.default_rng(rows + cols)
    a32 = g.standard_normal((rows, cols)).astype(np.float32)
    b32 = (a32 + 0.5 * g.standard_normal((rows, cols))).astype(np.float32)
    if dtype == "bf16":
        from workloads.synth import bf16_bits_from_f32
        a, b = bf16_bits_from_f32(a32), bf16_bits_from_f32(b32)
    else:
        a, b = a32, b32
    got = float(fb.row_cosine_mean(to_device(a, dtype), to_device(b, dtype)).item())
    ref = OP.mean_cosine(OP.widen(a, dtype), OP.widen(b, dtype))
    assert got == pytest.approx(ref, rel=1e-12, abs=1e-12)


def test_fold_reports_bad_placement():
    counts = torch.ones(4, dtype=torch.int32, device="cuda")
    e2r = torch.tensor([0, 1, 5, 1], dtype=torch.int32, device="cuda")
    _, mm = fb.fold_rank_loads(counts, e2r, 2)
    assert float(mm.item()) == -1.0
