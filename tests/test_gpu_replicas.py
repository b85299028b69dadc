"""Replicated placements on MI355X: fb_fold_slot_loads against the oracle, the device planners
against the host planner and the oracle, and the predicted-then-planned path of the "EPLB + Ours"
setting."""
import sys

import numpy as np
import pytest
import torch

import paper_2608_14205_amd as fb
from oracle import planner as OP
from oracle import predictor as OPR
from oracle import replicas as RP
from workloads import (CONFIGS, contiguous_placement, make_layer, random_replicated_placement,
                       replicated_placement, truncated_zipf_probs)
from gpu_util import run_gpu

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _fold(counts, slots):
    c = torch.from_numpy(np.ascontiguousarray(counts, np.int32)).cuda()
    s = torch.from_numpy(np.ascontiguousarray(slots, np.int32)).cuda()
    loads, mm = fb.fold_slot_loads(c, s)
    torch.cuda.synchronize()
    return loads.cpu().numpy().astype(np.int64), float(mm.item())


def test_slot_fold_random_placements():
    _say("[replicas] slot fold, random placements")
    g = np.random.default_rng(11)
    n = 0
    for _ in range(150):
        R = int(g.integers(1, 17))
        S = int(g.integers(1, 9))
        got = random_replicated_placement(g, R, S)
        if got is None:
            continue
        slots, E = got
        counts = (g.integers(0, 5000, size=E) * (g.random(E) < 0.9)).astype(np.int32)
        loads, mm = _fold(counts, slots)
        ref = RP.slot_rank_loads(counts, slots)
        assert np.array_equal(loads, ref), (R, S, E)
        assert mm == OPR.max_to_mean(ref)
        n += 1
    assert n > 100


@pytest.mark.parametrize("R,S,E,s", [(8, 2, 8, 1.2), (32, 9, 256, 1.1), (32, 8, 128, 1.0),
                                     (1024, 4, 4000, 1.1)])
def test_slot_fold_history_placements(R, S, E, s):
    # placements that replicate the most popular experts into the spare slots; the largest case
    # fills every slot the fold accepts (R * S = 4096)
    _say(f"[replicas] slot fold R={R} S={S} E={E}")
    slots = replicated_placement(truncated_zipf_probs(s, E), R, S)
    g = np.random.default_rng(R * S + E)
    counts = g.integers(0, 20000, size=E).astype(np.int32)
    loads, mm = _fold(counts, slots)
    ref = RP.slot_rank_loads(counts, slots)
    assert np.array_equal(loads, ref)
    assert mm == OPR.max_to_mean(ref)


def test_slot_fold_plain_placement_equals_rank_fold():
    wl = CONFIGS["dsv3"]
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    counts = np.random.default_rng(3).integers(0, 3000, size=wl.E).astype(np.int32)
    loads, mm = _fold(counts, slots)
    ref = OPR.rank_loads(counts, e2r, wl.R)
    assert np.array_equal(loads, ref)
    assert mm == OPR.max_to_mean(ref)


@pytest.mark.parametrize("slots,counts", [
    ([[0, 1], [0, -1]], [3, 1]),     # replica 0 of expert 0 twice
    ([[0, 1], [4, -1]], [3, 1]),     # replica 2 of expert 0 without replica 1
    ([[0, 2], [1, -1]], [3, 1]),     # two replicas of expert 0 on rank 0
    ([[0, 1], [2, 4]], [3, 1]),      # ordinal 2 reaches R = 2
    ([[0, -1], [-1, -1]], [3, 1]),   # expert 1 missing
    ([[0, -2], [1, -1]], [3, 1]),    # invalid value
    ([[0, 1], [2, -1]], [3, -1]),    # negative count
    ([[0, 1], [2, -1]], [7]),        # one expert, three replicas, two on rank 0
])
def test_slot_fold_flags_broken_placements(slots, counts):
    _, mm = _fold(counts, slots)
    assert mm == -1.0


def _device(counts, slots, budget, cost=None):
    c = torch.from_numpy(np.ascontiguousarray(counts, np.int32)).cuda()
    s = torch.from_numpy(np.ascontiguousarray(slots, np.int32)).cuda()
    if cost is None:
        return fb.plan_swaps_device(c, s, budget).to_host()
    return fb.plan_swaps_timed_device(c, s, budget, cost).to_host()


def _same(a, b):
    assert [tuple(x) for x in a.swaps] == [tuple(x) for x in b.swaps]
    assert np.array_equal(a.slots, b.slots)
    assert np.array_equal(a.expert_to_rank, b.expert_to_rank)
    assert np.array_equal(a.rank_loads, b.rank_loads)


@pytest.mark.parametrize("R_max,S_max", [(8, 8), (70, 3), (300, 2), (16, 12)])
def test_device_planner_replicated_placements(R_max, S_max):
    """device = host (= oracle on the smaller ones) on random replicated placements, in every launch
    shape: the one-wave frontier kernel (S * S <= 64, 1 to 16 ranks per lane) and the general kernel
    (full mode, larger S, time budgets)."""
    _say(f"[replicas] device planner R <= {R_max}, S <= {S_max}")
    g = np.random.default_rng(R_max * 100 + S_max)
    n = 0
    for it in range(40):
        R = int(g.integers(2, R_max + 1))
        S = int(g.integers(1, S_max + 1))
        got = random_replicated_placement(g, R, S)
        if got is None:
            continue
        slots, E = got
        counts = (g.integers(0, 3000, size=E) * (g.random(E) < 0.9)).astype(np.int32)
        mode = ("frontier", "full")[it % 2] if R * R * S * S <= 200000 else "frontier"
        B = int(g.integers(0, 9))
        bg = fb.Budget(B, mode=mode, per_rank_cap=int(g.integers(0, 3)))
        host = fb.plan_swaps(counts, slots, bg)
        _same(_device(counts, slots, bg), host)
        if R * S <= 40:
            ref = OP.plan_swaps(counts, slots, B, mode=mode, per_rank_cap=bg.per_rank_cap)
            assert [tuple(x) for x in ref.swaps] == [tuple(x) for x in host.swaps]
        if it % 4 in (0, 1):                   # time budgets in both modes
            cm = fb.CostModel(g.integers(0, 2, size=R).tolist(), g.integers(0, 400, size=E).tolist(),
                              (int(g.integers(1, 50)), int(g.integers(1, 200))),
                              (int(g.integers(100, 2000)), int(g.integers(20, 400))),
                              int(g.integers(0, 12000)), None)
            th = fb.plan_swaps_timed(counts, slots, bg, cm)
            td = _device(counts, slots, bg, cm)
            _same(td, th)
            assert td.costs == th.costs
        n += 1
    assert n >= 30


@pytest.mark.parametrize("counts,slots", [
    ([3, 1], [[0, 1], [0, -1]]), ([3, 1], [[0, 1], [4, -1]]), ([3, 1], [[0, 2], [1, -1]]),
    ([3, 1], [[0, 1], [2, 4]]),
    # one expert with more replicas than a rank has slots, two of them on rank 0
    ([7], [[0, 1], [2, -1]]), ([7], [[0, -1], [1, -1], [3, 2]]),
])
def test_device_planner_flags_broken_replicated_placements(counts, slots):
    c = torch.tensor(counts, dtype=torch.int32, device="cuda")
    s = torch.tensor(slots, dtype=torch.int32, device="cuda")
    for mode in ("frontier", "full"):
        plan = fb.plan_swaps_device(c, s, fb.Budget(2, mode=mode))
        torch.cuda.synchronize()
        assert int(plan.status.item()) == fb._lib.FB_EINVAL
        assert int(plan.n_swaps.item()) == 0


@pytest.mark.parametrize("R,S", [(64, 1), (40, 3), (200, 2)])
def test_device_planner_experts_replicated_on_many_ranks(R, S):
    # a few experts, each with far more replicas than a rank has slots (the check's per-rank branch)
    g = np.random.default_rng(R + S)
    E = S
    slots = np.array([[e + E * r for e in range(S)] for r in range(R)], np.int32)
    for r in range(R):
        slots[r] = slots[r][g.permutation(S)]
    slots[R - 1][slots[R - 1] == E * (R - 1)] = -1     # expert 0 keeps R - 1 replicas
    assert RP.replica_counts(slots, E) == [R - 1] + [R] * (E - 1)
    counts = g.integers(100, 5000, size=E).astype(np.int32)
    for mode in ("frontier", "full"):
        bg = fb.Budget(4, mode=mode)
        _same(_device(counts, slots, bg), fb.plan_swaps(counts, slots, bg))


@pytest.mark.parametrize("name,S_extra,budget", [("mixtral", 0, 4), ("dsv3", 1, 8)])
def test_predicted_counts_planned_on_a_replicated_placement(name, S_extra, budget):
    """The "EPLB + Ours" path: counts predicted on the GPU, folded on the GPU under a placement that
    replicates popular experts, planned on the device (= host = oracle), and the plan's loads equal
    the GPU fold of the new slot table."""
    wl = CONFIGS[name].with_T(4096)
    S = wl.S + S_extra
    _say(f"[replicas] {name} T={wl.T} R={wl.R} S={S}")
    slots = replicated_placement(truncated_zipf_probs(wl.zipf_s[0], wl.E), wl.R, S)
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S) if wl.E % wl.R == 0 else (None, None)
    li = make_layer(wl, 2)
    got = run_gpu(li, wl, e2r, debug=False, packed=True)
    counts = got["counts"].astype(np.int32)
    loads, mm = _fold(counts, slots)
    ref_loads = RP.slot_rank_loads(counts, slots)
    assert np.array_equal(loads, ref_loads)
    for mode in ("frontier", "full"):
        host = fb.plan_swaps(counts, slots, fb.Budget(budget, mode=mode))
        ref = OP.plan_swaps(counts, slots, budget, mode=mode)
        assert [tuple(s) for s in host.swaps] == [tuple(s) for s in ref.swaps]
        assert np.array_equal(host.slots, ref.slots)
        _same(_device(counts, slots, fb.Budget(budget, mode=mode)), host)
        after, mm_after = _fold(counts, host.slots)
        assert np.array_equal(after, host.rank_loads)
        assert mm_after <= mm
        _say(f"[replicas] {name} {mode}: {len(host.swaps)} swaps, max/mean {mm:.4f} -> {mm_after:.4f}")
