"""fb_predict_plan_packed (the prediction and the swap plan of its counts in one call) against the two
separate calls and the oracle planner, on MI355X.  Where the one-wave planner serves the plan it runs
inside the predictor's last workgroup; the other plans run as a kernel of their own."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2608_14205_amd as fb
from oracle import planner as OP
from workloads import CONFIGS, contiguous_placement, make_layer, random_replicated_placement
from gpu_util import scoring_of, to_device

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def _t(a, dtype=np.int32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype)).cuda()


def _run_both(wl, slots, e2r, budget, split=True):
    """The fused call and the two separate calls on the same inputs; both results on the host."""
    li = make_layer(wl, 0)
    x = to_device(li.x, wl.dtype)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    sb = None if li.select_bias is None else torch.from_numpy(li.select_bias).cuda()
    slots_t, e2r_t = _t(slots), _t(e2r)
    sc = scoring_of(wl)
    R = slots.shape[0]
    p1 = fb.Predictor(split=split)
    out1, plan1 = p1.predict_plan(x, wp, sc, e2r_t, slots_t, budget, select_bias=sb)
    p2 = fb.Predictor(split=split)
    out2 = p2.predict_load(x, wp, sc, e2r_t, R, select_bias=sb)
    plan2 = fb.plan_swaps_device(out2.counts, slots_t, budget)
    torch.cuda.synchronize()
    assert not p1.workspace[:2048].cpu().numpy().any()      # the workspace header is left clean
    return (out1, plan1), (out2, plan2)


def _host_pred(out):
    return (out.counts.cpu().numpy(), out.rank_loads.cpu().numpy(), float(out.max_mean.item()))


def _same_plan(a, b):
    assert [tuple(s) for s in a.swaps] == [tuple(s) for s in b.swaps]
    assert np.array_equal(a.slots, b.slots)
    assert np.array_equal(a.expert_to_rank, b.expert_to_rank)
    assert np.array_equal(a.rank_loads, b.rank_loads)


def _check(wl, slots, e2r, budget, split=True, oracle=True, label=""):
    (o1, p1), (o2, p2) = _run_both(wl, slots, e2r, budget, split)
    c1, r1, m1 = _host_pred(o1)
    c2, r2, m2 = _host_pred(o2)
    assert np.array_equal(c1, c2) and np.array_equal(r1, r2) and m1 == m2
    h1, h2 = p1.to_host(), p2.to_host()
    _same_plan(h1, h2)
    if oracle:
        ref = OP.plan_swaps(c1.astype(np.int64), slots, budget.max_swaps, gamma=budget.gamma,
                            tau=budget.tau, mode=budget.mode, per_rank_cap=budget.per_rank_cap)
        _same_plan(h1, ref)
    _say(f"[predict_plan] {label}: {len(h1.swaps)} swaps, counts sum {int(c1.sum())}")
    return c1, h1


@pytest.mark.parametrize("name,T,H,R,S,B", [
    ("dsv3", 3000, 512, 32, 8, 8),        # the DS-V3 placement: one candidate per lane
    ("dsv3", 2048, 512, 64, 4, 16),       # 64 ranks, the most the fused planner takes
    ("qwen3", 2048, 512, 32, 4, 6),
    ("mixtral", 1000, 4096, 8, 2, 1),     # split mode: the tile's last split finishes and plans
    ("qwen3", 1500, 512, 8, 11, 5),       # 11 slots per rank: two candidates per lane
    ("tiny", 300, 256, 8, 2, 2),          # float32 inputs
])
def test_fused_plan_matches_the_two_calls_and_the_oracle(name, T, H, R, S, B):
    wl = CONFIGS[name]
    E = wl.E if S != 11 else 64
    wl = dataclasses.replace(wl, T=T, H=H, E=E, R=R, S=S, n_clusters=min(wl.n_clusters, E),
                             k=min(wl.k, E))
    slots, e2r = contiguous_placement(E, R, S)
    assert fb.Budget(B).mode == "frontier" and R <= 64 and S * S <= 128    # the fused planner
    _check(wl, slots, e2r, fb.Budget(B, layer_id=2), label=f"{name} T={T} R={R} S={S} B={B}")


@pytest.mark.parametrize("name,T,R,S,mode", [
    ("dsv3", 2048, 32, 8, "full"),        # full mode: the workgroup planner after the prediction
    ("dsv3", 2048, 128, 2, "frontier"),   # 128 ranks: more than the fused planner takes
    ("qwen3", 2048, 8, 16, "frontier"),   # S * S > 128
])
def test_plans_the_fused_planner_does_not_take(name, T, R, S, mode):
    wl = dataclasses.replace(CONFIGS[name], T=T, H=512, R=R, S=S)
    slots, e2r = contiguous_placement(wl.E, R, S)
    _check(wl, slots, e2r, fb.Budget(6, mode=mode), label=f"{name} R={R} S={S} {mode}")


def test_fused_plan_on_replicated_placements():
    g = np.random.default_rng(11)
    done = 0
    while done < 6:
        drawn = random_replicated_placement(g, 8, 6)
        if drawn is None:
            continue
        slots, E = drawn
        if E < 2:
            continue
        wl = dataclasses.replace(CONFIGS["tiny"], T=700, H=256, E=E, k=min(2, E), n_clusters=E,
                                 R=8, S=6)
        e2r = np.zeros(E, np.int32)
        for c, v in enumerate(slots.reshape(-1)):
            if 0 <= v < E:
                e2r[v] = c // 6                  # rank of replica 0
        (o1, p1), (o2, p2) = _run_both(wl, slots, e2r, fb.Budget(4))
        assert np.array_equal(o1.counts.cpu().numpy(), o2.counts.cpu().numpy())
        h1, h2 = p1.to_host(), p2.to_host()
        _same_plan(h1, h2)
        ref = OP.plan_swaps(o1.counts.cpu().numpy().astype(np.int64), slots, 4)
        _same_plan(h1, ref)
        done += 1
    _say("[predict_plan] replicated placements ok")


def test_fused_plan_reports_a_broken_table_and_keeps_the_prediction():
    wl = dataclasses.replace(CONFIGS["dsv3"], T=1024, H=512)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    bad = slots.copy()
    bad[3, 0] = bad[4, 0]                        # an expert placed twice
    li = make_layer(wl, 0)
    x = to_device(li.x, wl.dtype)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    sb = torch.from_numpy(li.select_bias).cuda()
    out, plan = fb.Predictor().predict_plan(x, wp, scoring_of(wl), _t(e2r), _t(bad), fb.Budget(8),
                                            select_bias=sb)
    ref = fb.Predictor().predict_load(x, wp, scoring_of(wl), _t(e2r), wl.R, select_bias=sb)
    torch.cuda.synchronize()
    assert int(plan.status.item()) == fb._lib.FB_EINVAL
    assert int(plan.n_swaps.item()) == 0
    assert np.array_equal(out.counts.cpu().numpy(), ref.counts.cpu().numpy())


def test_fused_plan_on_an_empty_batch():
    wl = dataclasses.replace(CONFIGS["dsv3"], T=0, H=512)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    x = torch.empty((0, 512), dtype=torch.bfloat16, device="cuda")
    w = to_device(make_layer(dataclasses.replace(wl, T=1), 0).w, wl.dtype)
    out, plan = fb.Predictor().predict_plan(x, fb.pack_router_weight(w), scoring_of(wl), _t(e2r),
                                            _t(slots), fb.Budget(8))
    torch.cuda.synchronize()
    assert not out.counts.cpu().numpy().any()
    assert float(out.max_mean.item()) == 1.0
    h = plan.to_host()
    assert h.swaps == [] and np.array_equal(h.slots, slots)


def test_fused_plan_repeats_and_reuses_its_outputs():
    """Back-to-back calls on one predictor with the same output tensors give the same plan."""
    wl = dataclasses.replace(CONFIGS["dsv3"], T=4096, H=1024)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, 1)
    x = to_device(li.x, wl.dtype)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    sb = torch.from_numpy(li.select_bias).cuda()
    pred = fb.Predictor()
    out, plan = pred.predict_plan(x, wp, scoring_of(wl), _t(e2r), _t(slots), fb.Budget(8),
                                  select_bias=sb)
    first = (out.counts.cpu().numpy().copy(), plan.to_host())
    for _ in range(5):
        pred.predict_plan(x, wp, scoring_of(wl), _t(e2r), _t(slots), fb.Budget(8), select_bias=sb,
                          out=out, plan=plan)
    torch.cuda.synchronize()
    assert np.array_equal(out.counts.cpu().numpy(), first[0])
    _same_plan(plan.to_host(), first[1])


# ---- under a time budget (Eq. 9-10): fb_predict_plan_timed_packed -----------------------------------

def _timed_both(wl, slots, e2r, budget, cost, split=True):
    """The fused call with a cost model, and the prediction followed by the time-budgeted device
    planner; both results on the host."""
    li = make_layer(wl, 0)
    x = to_device(li.x, wl.dtype)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    sb = None if li.select_bias is None else torch.from_numpy(li.select_bias).cuda()
    slots_t, e2r_t = _t(slots), _t(e2r)
    sc = scoring_of(wl)
    p1 = fb.Predictor(split=split)
    out1, plan1 = p1.predict_plan(x, wp, sc, e2r_t, slots_t, budget, select_bias=sb,
                                  cost=fb.CostModel(*cost))
    p2 = fb.Predictor(split=split)
    out2 = p2.predict_load(x, wp, sc, e2r_t, slots.shape[0], select_bias=sb)
    plan2 = fb.plan_swaps_timed_device(out2.counts, slots_t, budget, fb.CostModel(*cost))
    torch.cuda.synchronize()
    assert not p1.workspace[:2048].cpu().numpy().any()
    c1, c2 = out1.counts.cpu().numpy(), out2.counts.cpu().numpy()
    assert np.array_equal(c1, c2)
    assert np.array_equal(out1.rank_loads.cpu().numpy(), out2.rank_loads.cpu().numpy())
    h1, h2 = plan1.to_host(), plan2.to_host()
    _same_plan(h1, h2)
    assert h1.costs == h2.costs
    return c1, h1


def _nodes_sizes(R, E, per_node, rng, mixed):
    nodes = [r // per_node for r in range(R)]
    mb = 7168 * 2048 * 2
    sizes = [int(v) * mb for v in rng.integers(1, 4, E)] if mixed else [3 * mb] * E
    return nodes, sizes


@pytest.mark.parametrize("name,T,R,S,per_node,mixed,link_ms,B", [
    ("dsv3", 3000, 32, 8, 8, False, None, 64),     # 88 MB experts, 4 nodes of 8 ranks
    ("dsv3", 2048, 32, 8, 8, True, 3, 64),         # mixed sizes, a binding 3 ms link budget
    ("dsv3", 2048, 64, 4, 16, False, None, 16),    # 64 ranks: the most the fused planner takes
    ("qwen3", 1500, 8, 11, 4, True, None, 8),      # 11 slots per rank: two candidates per lane
    ("mixtral", 1000, 8, 2, 4, False, None, 4),    # split mode; one expert per rank and a spare
])
def test_timed_fused_plan_matches_the_two_calls_and_the_oracle(name, T, R, S, per_node, mixed,
                                                               link_ms, B):
    from oracle.cost import CostModel as OCost
    wl = CONFIGS[name]
    E = wl.E if S != 11 else 64
    wl = dataclasses.replace(wl, T=T, H=512 if name != "mixtral" else 4096, E=E, R=R, S=S,
                             n_clusters=min(wl.n_clusters, E), k=min(wl.k, E))
    slots, e2r = contiguous_placement(E, R, S)
    nodes, sizes = _nodes_sizes(R, E, per_node, np.random.default_rng(7), mixed)
    cost = OCost(nodes, sizes, (20_000, 50_000), (100_000, 25_000), 8_000_000,
                 None if link_ms is None else link_ms * 1_000_000)
    bg = fb.Budget(B)
    counts, h = _timed_both(wl, slots, e2r, bg, cost, split=True)
    ref = OP.plan_swaps(counts.astype(np.int64), slots, B, cost=cost)
    _same_plan(h, ref)
    assert h.costs == ref.costs
    _say(f"[predict_plan timed] {name} R={R} S={S}: {len(h.swaps)} swaps, costs {h.costs[:3]}")


def test_timed_fused_plan_seeded_fuzz():
    """The one-call early pass under time budgets on 24 seeded random instances the fused planner
    takes (2-64 ranks, 1-11 slots per rank, random plain slot tables with empty slots, both input
    dtypes, fused and split prediction, nodes of 1-16 ranks, random expert sizes, rank and link
    budgets): the fused plan = the two calls, and the host planner and the oracle on its counts."""
    from oracle.cost import CostModel as OCost
    g = np.random.default_rng(4242)
    swaps = 0
    for it in range(24):
        R = int(g.integers(2, 65))
        S = int(g.integers(1, 12))
        E = int(g.integers(2, min(256, R * S) + 1))
        t = np.full(R * S, -1, np.int32)
        t[g.permutation(R * S)[:E]] = np.arange(E)
        slots = t.reshape(R, S)
        e2r = np.zeros(E, np.int32)
        for c, v in enumerate(t):
            if v >= 0:
                e2r[v] = c // S
        wl = dataclasses.replace(CONFIGS["tiny"], T=int(g.integers(200, 1500)), H=256, E=E,
                                 k=min(4, E), n_clusters=E, R=R, S=S,
                                 dtype=["f32", "bf16"][it % 2])
        per_node = int(g.integers(1, 17))
        sizes = [int(v) for v in g.integers(0, 2 ** 28, size=E)]
        alpha = (int(g.integers(1, 50_000)), int(g.integers(1, 100_000)))
        beta = (int(g.integers(1_000, 200_000)), int(g.integers(1_000, 50_000)))
        one = max(alpha[i] + 2 * int(np.mean(sizes)) * 1000 // beta[i] for i in (0, 1))
        rank_ns = int(one * g.choice([0.5, 1, 2, 4, 16]))
        link_ns = None if g.random() < 0.5 else int(rank_ns * g.choice([0.3, 1, 3]))
        cost = OCost([r // per_node for r in range(R)], sizes, alpha, beta, rank_ns, link_ns)
        bg = fb.Budget(int(g.integers(1, 17)), per_rank_cap=int(g.integers(0, 3)),
                       tau=int(g.integers(0, 3)), layer_id=int(g.integers(0, 5)))
        _say(f"[predict_plan timed fuzz] {it}: R={R} S={S} E={E} T={wl.T} {wl.dtype}")
        counts, h = _timed_both(wl, slots, e2r, bg, cost, split=bool(it % 3))
        host = fb.plan_swaps_timed(counts, slots, bg, fb.CostModel(*cost))
        _same_plan(h, host)
        assert h.costs == host.costs
        if R * S <= 256:
            ref = OP.plan_swaps(counts.astype(np.int64), slots, bg.max_swaps, tau=bg.tau,
                                per_rank_cap=bg.per_rank_cap, layer_id=bg.layer_id, cost=cost)
            _same_plan(h, ref)
            assert h.costs == ref.costs
        swaps += len(h.swaps) > 0
    _say(f"[predict_plan timed fuzz] {swaps} of 24 with swaps")
    assert swaps >= 12


@pytest.mark.parametrize("R,S,mode", [(32, 8, "full"), (128, 2, "frontier")])
def test_timed_plans_the_fused_planner_does_not_take(R, S, mode):
    """Full mode, and more than 64 ranks under a time budget: the plan runs as its own kernel."""
    from oracle.cost import CostModel as OCost
    wl = dataclasses.replace(CONFIGS["dsv3"], T=2048, H=512, R=R, S=S)
    slots, e2r = contiguous_placement(wl.E, R, S)
    nodes, sizes = _nodes_sizes(R, wl.E, 8, np.random.default_rng(3), False)
    # 16 ms per rank: a swap across nodes (about 7 ms for two 88 MB experts) fits twice
    cost = OCost(nodes, sizes, (20_000, 50_000), (100_000, 25_000), 16_000_000)
    counts, h = _timed_both(wl, slots, e2r, fb.Budget(16, mode=mode), cost)
    assert len(h.swaps) >= 1
    _say(f"[predict_plan timed] R={R} {mode}: {len(h.swaps)} swaps")


def test_timed_fused_plan_reports_a_bad_expert_size_and_keeps_the_prediction():
    from oracle.cost import CostModel as OCost
    wl = dataclasses.replace(CONFIGS["dsv3"], T=1024, H=512)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    sizes = [1000] * wl.E
    sizes[5] = (1 << 40) + 1                      # beyond 2^40 bytes
    cost = OCost([r // 8 for r in range(wl.R)], sizes, (20_000, 50_000), (100_000, 25_000), 10 ** 9)
    li = make_layer(wl, 0)
    x = to_device(li.x, wl.dtype)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    sb = torch.from_numpy(li.select_bias).cuda()
    out, plan = fb.Predictor().predict_plan(x, wp, scoring_of(wl), _t(e2r), _t(slots), fb.Budget(8),
                                            select_bias=sb, cost=fb.CostModel(*cost))
    ref = fb.Predictor().predict_load(x, wp, scoring_of(wl), _t(e2r), wl.R, select_bias=sb)
    torch.cuda.synchronize()
    assert int(plan.status.item()) == fb._lib.FB_EINVAL
    assert int(plan.n_swaps.item()) == 0
    assert np.array_equal(out.counts.cpu().numpy(), ref.counts.cpu().numpy())


def test_timed_fused_plan_on_an_empty_batch_and_on_replicated_placements():
    from oracle.cost import CostModel as OCost
    # an empty batch: zero counts, no swap, the placement unchanged
    wl = dataclasses.replace(CONFIGS["dsv3"], T=0, H=512)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    cost = OCost([r // 8 for r in range(wl.R)], [1000] * wl.E, (20, 50), (100, 25), 10 ** 6)
    x = torch.empty((0, 512), dtype=torch.bfloat16, device="cuda")
    w = to_device(make_layer(dataclasses.replace(wl, T=1), 0).w, wl.dtype)
    out, plan = fb.Predictor().predict_plan(x, fb.pack_router_weight(w), scoring_of(wl), _t(e2r),
                                            _t(slots), fb.Budget(8), cost=fb.CostModel(*cost))
    torch.cuda.synchronize()
    assert not out.counts.cpu().numpy().any()
    h = plan.to_host()
    assert h.swaps == [] and np.array_equal(h.slots, slots) and h.costs == []
    # replicated placements on 8 ranks: the fused timed plan = the two calls (and the oracle)
    g = np.random.default_rng(23)
    done = 0
    while done < 4:
        drawn = random_replicated_placement(g, 8, 6)
        if drawn is None:
            continue
        slots, E = drawn
        if E < 2:
            continue
        wl = dataclasses.replace(CONFIGS["tiny"], T=700, H=256, E=E, k=min(2, E), n_clusters=E,
                                 R=8, S=6)
        e2r = np.zeros(E, np.int32)
        for c, v in enumerate(slots.reshape(-1)):
            if 0 <= v < E:
                e2r[v] = c // 6                  # rank of replica 0
        cost = OCost(list(g.integers(0, 2, 8)), list(g.integers(0, 400, E)), (5, 30), (300, 60),
                     int(g.integers(2000, 9000)))
        counts, h = _timed_both(wl, slots, e2r, fb.Budget(4), cost)
        ref = OP.plan_swaps(counts.astype(np.int64), slots, 4, cost=cost)
        _same_plan(h, ref)
        assert h.costs == ref.costs
        done += 1
    _say("[predict_plan timed] empty batch and replicated placements ok")


def test_reused_outputs_that_do_not_fit_are_refused():
    """Outputs passed back in (out=, plan=) must have room for the call's sizes: a plan made for 2
    swaps cannot take a budget of 8, nor a prediction for 16 experts a call with 256; the binding
    refuses them before anything is launched."""
    wl = dataclasses.replace(CONFIGS["dsv3"], T=256, H=256)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, 0)
    x = to_device(li.x, wl.dtype)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    sb = torch.from_numpy(li.select_bias).cuda()
    pred = fb.Predictor()
    out = pred.predict_load(x, wp, scoring_of(wl), _t(e2r), wl.R, select_bias=sb)
    small = fb.plan_swaps_device(out.counts, _t(slots), fb.Budget(2))
    with pytest.raises(ValueError):
        fb.plan_swaps_device(out.counts, _t(slots), fb.Budget(8), out=small)
    with pytest.raises(ValueError):
        pred.predict_plan(x, wp, scoring_of(wl), _t(e2r), _t(slots), fb.Budget(8),
                          select_bias=sb, plan=small)
    tiny = fb.Prediction(torch.zeros(16, dtype=torch.int32, device="cuda"),
                         torch.zeros(wl.R, dtype=torch.int32, device="cuda"),
                         torch.zeros(1, dtype=torch.float64, device="cuda"))
    with pytest.raises(ValueError):
        pred.predict_load(x, wp, scoring_of(wl), _t(e2r), wl.R, select_bias=sb, out=tiny)
    short_topk = fb.Prediction(out.counts, out.rank_loads, out.max_mean,
                               topk=torch.zeros(10, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):
        pred.predict_load(x, wp, scoring_of(wl), _t(e2r), wl.R, select_bias=sb, out=short_topk,
                          return_topk=True)
    # the same buffers still serve calls they fit, with results equal to fresh ones
    again = fb.plan_swaps_device(out.counts, _t(slots), fb.Budget(2), out=small)
    fresh = fb.plan_swaps_device(out.counts, _t(slots), fb.Budget(2))
    torch.cuda.synchronize()
    _same_plan(again.to_host(), fresh.to_host())
    _say("[predict_plan] reused outputs checked")
