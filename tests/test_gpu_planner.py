"""The device planner (one workgroup kernel) against the host planner and the oracle, on MI355X."""
import sys

import numpy as np
import pytest
import torch

import paper_2608_14205_amd as fb
from oracle import planner as OP
from workloads import CONFIGS, contiguous_placement, make_layer
from gpu_util import run_gpu

pytestmark = pytest.mark.gpu


def _dev(counts, slots, budget):
    c = torch.from_numpy(np.ascontiguousarray(counts, np.int32)).cuda()
    s = torch.from_numpy(np.ascontiguousarray(slots, np.int32)).cuda()
    return fb.plan_swaps_device(c, s, budget).to_host()


def _same(a, b):
    assert [tuple(x) for x in a.swaps] == [tuple(x) for x in b.swaps]
    assert np.array_equal(a.slots, b.slots)
    assert np.array_equal(a.expert_to_rank, b.expert_to_rank)
    assert np.array_equal(a.rank_loads, b.rank_loads)


def test_device_planner_random_instances():
    print("[plan] random instances", flush=True)
    g = np.random.default_rng(0)
    for it in range(120):
        R = int(g.integers(1, 9))
        S = int(g.integers(1, 6))
        E = int(g.integers(1, R * S + 1))
        cells = g.permutation(R * S)[:E]
        slots = np.full(R * S, -1, np.int32)
        slots[cells] = np.arange(E)
        slots = slots.reshape(R, S)
        counts = (g.integers(0, 60, size=E) * (g.random(E) < 0.85)).astype(np.int32)
        bg = fb.Budget(int(g.integers(0, 7)), per_rank_cap=int(g.integers(0, 3)),
                       tau=int(g.integers(0, 5)),
                       gamma=[None, (0, 1), (2, 5)][it % 3], mode=["frontier", "full"][it % 2])
        host = fb.plan_swaps(counts, slots, bg)
        dev = _dev(counts, slots, bg)
        _same(dev, host)
        ref = OP.plan_swaps(counts, slots, bg.max_swaps, gamma=bg.gamma, tau=bg.tau, mode=bg.mode,
                            per_rank_cap=bg.per_rank_cap)
        _same(dev, ref)


@pytest.mark.parametrize("mode", ["frontier", "full"])
def test_device_planner_on_predicted_counts(mode):
    print(f"[plan] dsv3 counts {mode}", flush=True)
    wl = CONFIGS["dsv3"].with_T(4096)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, 0)
    gpu = run_gpu(li, wl, e2r, debug=False)
    for B in (0, 4, 8, 16):
        bg = fb.Budget(B, mode=mode, layer_id=3)
        host = fb.plan_swaps(gpu["counts"], slots, bg)
        dev = _dev(gpu["counts"], slots, bg)
        _same(dev, host)
        ref = OP.plan_swaps(gpu["counts"], slots, B, mode=mode, layer_id=3)
        _same(host, ref)
        if B > 0:
            assert len(host.swaps) > 0
            assert host.rank_loads.max() < gpu["rank_loads"].max()


@pytest.mark.parametrize("R,S,mode", [(100, 4, "frontier"), (1024, 4, "frontier"), (16, 12, "frontier"),
                                      (64, 8, "frontier"), (3, 9, "full"), (40, 2, "full")])
def test_device_planner_launch_shapes(R, S, mode):
    """Every launch shape of the device planner: one wave with up to 16 ranks per lane, the
    four-wave frontier kernel for S * S > 64, the full-mode kernel."""
    print(f"[plan] R={R} S={S} {mode}", flush=True)
    g = np.random.default_rng(R * 100 + S)
    E = max(1, R * S - R // 3)
    for it in range(3):
        cells = g.permutation(R * S)[:E]
        slots = np.full(R * S, -1, np.int32)
        slots[cells] = np.arange(E)
        slots = slots.reshape(R, S)
        counts = (g.zipf(1.3, size=E) % 5000).astype(np.int32) * (g.random(E) < 0.9)
        bg = fb.Budget(int(g.integers(4, 40)), per_rank_cap=[0, 2][it % 2], mode=mode, layer_id=it)
        host = fb.plan_swaps(counts, slots, bg)
        dev = _dev(counts, slots, bg)
        _same(dev, host)
        assert len(host.swaps) > 0


@pytest.mark.parametrize("R", [4, 64, 100])
def test_device_planner_loads_beyond_31_bits(R):
    """Total load above 2^31 (max-only objective, gamma = 0, so the benefit still fits 64 bits):
    the one-wave kernel leaves its 32-bit fast rounds for the 64-bit ones."""
    print(f"[plan] loads beyond 31 bits, R={R}", flush=True)
    g = np.random.default_rng(R)
    S = 2
    E = R * S
    slots = g.permutation(E).astype(np.int32).reshape(R, S)
    counts = g.integers(1 << 20, (1 << 31) - 1, size=E, dtype=np.int64).astype(np.int32)
    assert int(counts.astype(np.int64).sum()) > (1 << 31)
    for mode in ("frontier", "full"):
        bg = fb.Budget(6, gamma=(0, 1), mode=mode)
        host = fb.plan_swaps(counts, slots, bg)
        _same(_dev(counts, slots, bg), host)
        ref = OP.plan_swaps(counts, slots, 6, gamma=(0, 1), mode=mode)
        _same(host, ref)


def test_device_planner_reports_bad_placement():
    print("[plan] invalid slot table", flush=True)
    slots = np.array([[0, 1], [1, 3]], np.int32)   # expert 1 twice, expert 2 missing
    c = torch.ones(4, dtype=torch.int32, device="cuda")
    out = fb.plan_swaps_device(c, torch.from_numpy(slots).cuda(), fb.Budget(2))
    torch.cuda.synchronize()
    assert int(out.status.item()) == -1 and int(out.n_swaps.item()) == 0


def test_predict_then_plan_on_stream():
    """The benchmark step: prediction and planning back to back on one stream, no host sync."""
    print("[plan] predict -> plan on one stream", flush=True)
    wl = CONFIGS["dsv3"].with_T(3000)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, 1)
    from gpu_util import to_device, scoring_of
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        x, w = to_device(li.x, "bf16"), to_device(li.w, "bf16")
        sb = torch.from_numpy(li.select_bias).cuda()
        e2r_t = torch.from_numpy(e2r).cuda()
        slots_t = torch.from_numpy(slots).cuda()
        pred = fb.Predictor(stream=s)
        out = pred.predict_load(x, w, scoring_of(wl), e2r_t, wl.R, select_bias=sb, stream=s)
        plan = fb.plan_swaps_device(out.counts, slots_t, fb.Budget(wl.budget), stream=s)
    s.synchronize()
    host = fb.plan_swaps(out.counts.cpu().numpy(), slots, fb.Budget(wl.budget))
    _same(plan.to_host(), host)


# ---- time-budgeted planner (Eq. 9-10, budgets per rank and link) --------------------------------

def _dev_timed(counts, slots, budget, cost):
    c = torch.from_numpy(np.ascontiguousarray(counts, np.int32)).cuda()
    s = torch.from_numpy(np.ascontiguousarray(slots, np.int32)).cuda()
    return fb.plan_swaps_timed_device(c, s, budget, cost).to_host()


def test_timed_device_planner_random_instances():
    print("[plan] timed random instances", flush=True)
    from oracle.cost import CostModel as OCost
    g = np.random.default_rng(1)
    for it in range(120):
        R = int(g.integers(1, 9))
        S = int(g.integers(1, 6))
        E = int(g.integers(1, R * S + 1))
        cells = g.permutation(R * S)[:E]
        slots = np.full(R * S, -1, np.int32)
        slots[cells] = np.arange(E)
        slots = slots.reshape(R, S)
        counts = (g.integers(0, 60, size=E) * (g.random(E) < 0.85)).astype(np.int32)
        cm = OCost(g.integers(0, 2, size=R).tolist(), g.integers(0, 400, size=E).tolist(),
                   (int(g.integers(1, 50)), int(g.integers(1, 200))),
                   (int(g.integers(100, 2000)), int(g.integers(20, 400))),
                   int(g.integers(0, 12000)), None if it % 2 else int(g.integers(0, 12000)))
        bg = fb.Budget(int(g.integers(0, 7)), per_rank_cap=int(g.integers(0, 3)),
                       tau=int(g.integers(0, 5)),
                       gamma=[None, (0, 1), (2, 5)][it % 3], mode=["frontier", "full"][(it // 2) % 2])
        host = fb.plan_swaps_timed(counts, slots, bg, fb.CostModel(*cm))
        dev = _dev_timed(counts, slots, bg, fb.CostModel(*cm))
        _same(dev, host)
        assert dev.costs == host.costs
        ref = OP.plan_swaps(counts, slots, bg.max_swaps, gamma=bg.gamma, tau=bg.tau, mode=bg.mode,
                            per_rank_cap=bg.per_rank_cap, cost=cm)
        _same(dev, ref)
        assert dev.costs == ref.costs


@pytest.mark.parametrize("mode", ["frontier", "full"])
def test_timed_device_planner_on_predicted_counts(mode):
    """DeepSeek-V3-shaped predicted counts, 32 ranks on 4 nodes of 8, 88 MB experts (three
    7168 x 2048 bf16 matrices), 20 us / 100 GB/s inside a node and 50 us / 25 GB/s across nodes
    (one intra-node swap costs 1.78 ms, an inter-node one 7.1 ms), per-rank budgets of 2-16 ms.
    Device = host on every case; the oracle joins in frontier mode (in full mode its exact-rational
    enumeration of ~30k candidates per round takes minutes; host = oracle there is covered on
    smaller instances)."""
    print(f"[plan] timed dsv3 counts {mode}", flush=True)
    from oracle.cost import CostModel as OCost
    wl = CONFIGS["dsv3"].with_T(4096)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, 0)
    gpu = run_gpu(li, wl, e2r, debug=False)
    nodes = [r // 8 for r in range(wl.R)]
    nbytes = [3 * 7168 * 2048 * 2] * wl.E
    budgets = (2_000_000, 8_000_000, 16_000_000) if mode == "frontier" else (2_000_000, 4_000_000, 8_000_000)
    for budget_ns in budgets:
        args = (nodes, nbytes, (20_000, 50_000), (100_000, 25_000), budget_ns)
        bg = fb.Budget(64, mode=mode, layer_id=5)
        host = fb.plan_swaps_timed(gpu["counts"], slots, bg, fb.CostModel(*args))
        dev = _dev_timed(gpu["counts"], slots, bg, fb.CostModel(*args))
        _same(dev, host)
        assert dev.costs == host.costs
        if mode == "frontier":
            ref = OP.plan_swaps(gpu["counts"], slots, 64, mode=mode, layer_id=5, cost=OCost(*args))
            _same(host, ref)
            assert host.costs == ref.costs
        else:
            assert len(host.swaps) > 0
        if host.swaps:
            assert host.rank_loads.max() < gpu["rank_loads"].max()
        print(f"[plan]   budget {budget_ns / 1e6:.0f} ms: {len(host.swaps)} swaps", flush=True)


def test_timed_device_planner_reports_bad_sizes():
    print("[plan] timed: expert size out of range", flush=True)
    slots = torch.tensor([[0, 1], [2, 3]], dtype=torch.int32, device="cuda")
    c = torch.tensor([9, 1, 1, 1], dtype=torch.int32, device="cuda")
    cm = fb.CostModel([0, 0], [1, 1, 2 ** 41, 1], (5, 5), (100, 100), 10 ** 6)
    out = fb.plan_swaps_timed_device(c, slots, fb.Budget(2), cm)
    torch.cuda.synchronize()
    assert int(out.status.item()) == -1 and int(out.n_swaps.item()) == 0


def test_device_planner_seeded_fuzz():
    """device = host on 1000 seeded random instances: plain and replicated placements, R up to 299,
    S up to 11 (both one-wave kernel instantiations and the general kernel), both modes, per-rank
    caps, tau, gamma, layer ids and counts up to 2^20."""
    from workloads import random_replicated_placement
    print("[plan] seeded fuzz", flush=True)
    g = np.random.default_rng(20261)
    n = 0
    for it in range(1000):
        R = int(g.integers(2, [9, 40, 130, 300][it % 4]))
        S = int(g.integers(1, 12))
        if R * S > 4096:
            continue
        if g.random() < 0.5:
            got = random_replicated_placement(g, R, S)
            if got is None:
                continue
            slots, E = got
        else:
            E = int(g.integers(1, R * S + 1))
            t = np.full(R * S, -1, np.int32)
            t[g.permutation(R * S)[:E]] = np.arange(E)
            slots = t.reshape(R, S)
        hi = [5, 60, 3000, 2 ** 20][int(g.integers(0, 4))]
        counts = (g.integers(0, hi, size=E) * (g.random(E) < 0.9)).astype(np.int32)
        mode = "frontier" if g.random() < 0.7 or R * R * S * S > 300000 else "full"
        gamma = [None, (0, 1), (1, 7), (3, 2)][int(g.integers(0, 4))]
        bg = fb.Budget(int(g.integers(0, 12)), mode=mode, per_rank_cap=int(g.integers(0, 3)),
                       tau=int(g.integers(0, 3)), gamma=gamma, layer_id=int(g.integers(0, 5)))
        host = fb.plan_swaps(counts, slots, bg)
        _same(_dev(counts, slots, bg), host)
        n += 1
    assert n > 900


def test_timed_device_planner_seeded_fuzz():
    """device = host (plans and Eq. 9 costs) on 400 seeded random instances under time budgets:
    plain and replicated placements, R up to 129, S up to 11 (the one-wave kernel for frontier plans
    on at most 64 ranks, the general kernel otherwise, stored per-pair frontiers in full mode on at
    most 64 ranks and 8 slots), nodes of 1-16 ranks, expert sizes 0-2^30 bytes, rank budgets that
    admit anywhere from no swap to all of them, and link budgets below or above them."""
    from workloads import random_replicated_placement
    print("[plan] timed seeded fuzz", flush=True)
    g = np.random.default_rng(20262)
    n = full = swaps = 0
    for it in range(400):
        R = int(g.integers(2, [9, 33, 65, 130][it % 4]))
        S = int(g.integers(1, 12))
        if R * S > 2048:
            continue
        if g.random() < 0.4:
            got = random_replicated_placement(g, R, S)
            if got is None:
                continue
            slots, E = got
        else:
            E = int(g.integers(1, R * S + 1))
            t = np.full(R * S, -1, np.int32)
            t[g.permutation(R * S)[:E]] = np.arange(E)
            slots = t.reshape(R, S)
        hi = [5, 60, 3000, 2 ** 20][int(g.integers(0, 4))]
        counts = (g.integers(0, hi, size=E) * (g.random(E) < 0.9)).astype(np.int32)
        mode = "full" if g.random() < 0.35 and R * R * S * S <= 300000 else "frontier"
        per_node = int(g.integers(1, 17))
        sizes = (g.integers(0, 2 ** 30, size=E) if g.random() < 0.5
                 else np.full(E, int(g.integers(0, 2 ** 30)))).tolist()
        alpha = (int(g.integers(1, 50_000)), int(g.integers(1, 100_000)))
        beta = (int(g.integers(1_000, 200_000)), int(g.integers(1_000, 50_000)))
        # one swap of two average experts across nodes, to scale the budgets
        one = max(alpha[i] + 2 * int(np.mean(sizes)) * 1000 // beta[i] for i in (0, 1))
        rank_ns = int(one * g.choice([0, 0.5, 1, 2, 4, 16, 64]))
        link_ns = None if g.random() < 0.5 else int(rank_ns * g.choice([0, 0.3, 1, 3]))
        cm = fb.CostModel([r // per_node for r in range(R)], sizes, alpha, beta, rank_ns, link_ns)
        gamma = [None, (0, 1), (1, 7), (3, 2)][int(g.integers(0, 4))]
        bg = fb.Budget(int(g.integers(0, 12)), mode=mode, per_rank_cap=int(g.integers(0, 3)),
                       tau=int(g.integers(0, 3)), gamma=gamma, layer_id=int(g.integers(0, 5)))
        host = fb.plan_swaps_timed(counts, slots, bg, cm)
        dev = _dev_timed(counts, slots, bg, cm)
        _same(dev, host)
        assert dev.costs == host.costs, it
        n += 1
        full += mode == "full"
        swaps += len(host.swaps) > 0
    print(f"[plan]   {n} instances, {full} in full mode, {swaps} with swaps", flush=True)
    assert n > 350 and full > 80 and swaps > 150


@pytest.mark.parametrize("max_swaps", [1, 6])
def test_full_mode_pair_with_a_long_staircase(max_swaps):
    """Full mode under a time budget on two ranks of 8 slots whose candidates form a staircase of 9
    (load difference growing while the cost falls): more than the 8 the device planner stores per
    rank pair, so it scores all of the pair's candidates.  Device = host = oracle."""
    from oracle.cost import CostModel as OCost
    print(f"[plan] long staircase, {max_swaps} swaps", flush=True)
    # rank 0: experts 0-7 with 100 + 10 p tokens and (p + 1) KB; rank 1: experts 8-11 with no
    # tokens and 5 KB, experts 12-15 with one token and no bytes.  With beta = 1000 B/us a candidate
    # (p, q) costs alpha + its bytes in ns, and u = |D + 2 (l_q - l_p)| orders the candidates by p;
    # the one-token partners cost 5000 ns less at u + 2, so every slot p adds a point
    counts = np.array([100 + 10 * p for p in range(8)] + [0] * 4 + [1] * 4, np.int32)
    slots = np.arange(16, dtype=np.int32).reshape(2, 8)
    sizes = [1000 * (p + 1) for p in range(8)] + [5000] * 4 + [0] * 4
    cm = OCost([0, 0], sizes, (3, 3), (1000, 1000), 10 ** 9)
    bg = fb.Budget(max_swaps, mode="full")
    host = fb.plan_swaps_timed(counts, slots, bg, fb.CostModel(*cm))
    dev = _dev_timed(counts, slots, bg, fb.CostModel(*cm))
    _same(dev, host)
    assert dev.costs == host.costs
    ref = OP.plan_swaps(counts, slots, max_swaps, mode="full", cost=cm)
    _same(dev, ref)
    assert len(dev.swaps) >= 1
