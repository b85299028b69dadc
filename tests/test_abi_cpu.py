"""C ABI checks that need no GPU: the library loads and exports every declared symbol, the host
planner matches the oracle bit for bit, the cost helper matches the oracle, and argument validation
rejects bad calls before any HIP call is made."""
import ctypes
import json
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import paper_2608_14205_amd as fb
from paper_2608_14205_amd import _lib as L
from oracle import cost as OC
from oracle import planner as OP
from workloads import random_replicated_placement

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "freebalance.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fb_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    assert names == sorted(["fb_abi_version", "fb_status_string", "fb_router_packed_bytes",
                            "fb_predict_workspace_bytes", "fb_predict_workspace_init",
                            "fb_pack_router_weight", "fb_predict_load", "fb_predict_load_packed",
                            "fb_plan_swaps", "fb_plan_swaps_device", "fb_swap_budget_from_cost",
                            "fb_topk_hits", "fb_cosine_workspace_bytes", "fb_row_cosine_mean",
                            "fb_fold_rank_loads", "fb_plan_swaps_timed",
                            "fb_plan_swaps_timed_device", "fb_predict_split_workspace_bytes",
                            "fb_fold_slot_loads", "fb_predict_load_packed_noalloc",
                            "fb_predict_plan_packed", "fb_predict_plan_timed_packed"])


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(L.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert set(L.SIGNATURES) == set(_declared_functions())


def test_struct_layouts_match_header():
    assert ctypes.sizeof(L.fb_scoring) == 20
    assert ctypes.sizeof(L.fb_budget) == 40
    assert ctypes.sizeof(L.fb_swap) == 32 == fb.api.SWAP_BYTES
    assert ctypes.sizeof(L.fb_cost_model) == 48


def test_version_and_status_strings():
    lib = fb.lib()
    assert lib.fb_abi_version() == 6
    for code in (0, -1, -2, -3, -4):
        assert L.status_string(code).startswith("FB_")
    assert "unknown" in L.status_string(7)



@pytest.mark.parametrize("E,H,dtype", [(1, 32, L.FB_BF16), (8, 4096, L.FB_BF16), (60, 2048, L.FB_BF16),
                                       (128, 2048, L.FB_BF16), (256, 7168, L.FB_BF16),
                                       (256, 7168, L.FB_F32), (33, 48, L.FB_F32)])
def test_packed_router_and_workspace_sizes(E, H, dtype):
    """The packed weight holds E rounded up to 32, 64, 128 or 256 rows of H elements rounded up
    to whole 256-byte stages; the unpacked entry point's workspace adds 2 KB of accumulators."""
    lib = fb.lib()
    hb = H * (2 if dtype == L.FB_BF16 else 4)
    epad = next(p for p in (32, 64, 128, 256) if E <= p)
    packed = lib.fb_router_packed_bytes(E, H, dtype)
    assert packed == epad * (-(-hb // 256)) * 256
    assert lib.fb_predict_workspace_bytes(E, H, dtype) == packed + 2048


def test_packed_sizes_reject_invalid():
    lib = fb.lib()
    assert lib.fb_router_packed_bytes(0, 64, L.FB_BF16) == 0
    assert lib.fb_router_packed_bytes(257, 64, L.FB_BF16) == 0
    assert lib.fb_router_packed_bytes(8, 0, L.FB_BF16) == 0
    assert lib.fb_router_packed_bytes(8, 64, 5) == 0
    assert lib.fb_predict_workspace_bytes(300, 64, L.FB_BF16) == 0


@pytest.mark.parametrize("over,code", [
    (dict(w=None), L.FB_EINVAL),
    (dict(out=None), L.FB_EINVAL),
    (dict(E=0), L.FB_EINVAL),
    (dict(dtype=3), L.FB_EINVAL),
    (dict(E=257), L.FB_EUNSUPPORTED),
    (dict(H=48), L.FB_EUNSUPPORTED),
    (dict(w=0x2004), L.FB_EUNSUPPORTED),
    (dict(out=0x3008), L.FB_EUNSUPPORTED),
    (dict(nbytes=8191), L.FB_ENOSPC),
])
def test_pack_validation_without_gpu(over, code):
    a = dict(w=0x2000, E=16, H=64, dtype=L.FB_BF16, out=0x3000, nbytes=8192)
    a.update(over)
    assert fb.lib().fb_pack_router_weight(a["w"], a["E"], a["H"], a["dtype"], a["out"], a["nbytes"],
                                          None) == code


def _host(counts, slots, **kw):
    return fb.plan_swaps(counts, slots, fb.Budget(**kw))


def _same(host, ref):
    assert [tuple(s) for s in host.swaps] == [tuple(s) for s in ref.swaps]
    assert np.array_equal(host.slots, ref.slots)
    assert np.array_equal(host.expert_to_rank, ref.expert_to_rank)
    assert np.array_equal(host.rank_loads, ref.rank_loads)


def test_host_planner_hand_worked_plans(golden_dir):
    with open(os.path.join(golden_dir, "planner_hand.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        h = _host(c["counts"], c["slots"], max_swaps=c["max_swaps"], mode=c["mode"],
                  per_rank_cap=c.get("per_rank_cap", 0), tau=c.get("tau", 0),
                  gamma=tuple(c["gamma"]) if "gamma" in c else None)
        assert [list(s) for s in h.swaps] == c["swaps"], c["name"]
        assert h.slots.tolist() == c["new_slots"], c["name"]
        assert h.rank_loads.tolist() == c["rank_loads"], c["name"]


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 6), st.integers(1, 5), st.integers(0, 10 ** 9), st.integers(0, 6),
       st.sampled_from(["frontier", "full"]), st.integers(0, 3), st.integers(0, 6),
       st.sampled_from([None, (0, 1), (1, 7), (3, 2)]), st.integers(0, 5))
def test_host_planner_matches_oracle(R, S, seed, B, mode, cap, tau, gamma, layer):
    g = np.random.default_rng(seed)
    E = int(g.integers(1, R * S + 1))
    cells = g.permutation(R * S)[:E]
    slots = np.full(R * S, -1, np.int32)
    slots[cells] = np.arange(E)
    slots = slots.reshape(R, S)
    counts = (g.integers(0, 40, size=E) * (g.random(E) < 0.85)).astype(np.int32)
    ref = OP.plan_swaps(counts, slots, B, gamma=gamma, tau=tau, mode=mode, per_rank_cap=cap,
                        layer_id=layer)
    host = _host(counts, slots, max_swaps=B, mode=mode, per_rank_cap=cap, tau=tau, gamma=gamma,
                 layer_id=layer)
    _same(host, ref)


def test_host_planner_is_deterministic_and_pure():
    g = np.random.default_rng(4)
    slots = np.arange(256, dtype=np.int32).reshape(32, 8)
    counts = g.integers(0, 3000, size=256).astype(np.int32)
    before = (counts.copy(), slots.copy())
    a = _host(counts, slots, max_swaps=16)
    b = _host(counts, slots, max_swaps=16)
    _same(a, b)
    assert np.array_equal(counts, before[0]) and np.array_equal(slots, before[1])
    assert len(a.swaps) > 0


@pytest.mark.parametrize("bad", [
    dict(slots=[[0, 1], [1, 3]]),   # expert placed twice
    dict(slots=[[0, 1], [2, -1]]),  # expert missing
    dict(slots=[[0, 1], [2, 9]]),   # id out of range
    dict(counts=[1, -1, 1, 1]),     # negative count
])
def test_host_planner_rejects_bad_placement(bad):
    counts = bad.get("counts", [1, 1, 1, 1])
    slots = bad.get("slots", [[0, 1], [2, 3]])
    with pytest.raises(fb.FreeBalanceError) as ei:
        fb.plan_swaps(counts, slots, fb.Budget(1))
    assert ei.value.status == L.FB_EINVAL


def test_host_planner_hand_worked_replicated_plans(golden_dir):
    with open(os.path.join(golden_dir, "planner_replicas_hand.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        h = _host(c["counts"], c["slots"], max_swaps=c["max_swaps"], mode=c["mode"])
        assert [list(s) for s in h.swaps] == c["swaps"], c["name"]
        assert h.slots.tolist() == c["new_slots"], c["name"]
        assert h.rank_loads.tolist() == c["rank_loads"], c["name"]


@settings(max_examples=300, deadline=None)
@given(st.integers(2, 6), st.integers(1, 5), st.integers(0, 10 ** 9), st.integers(0, 6),
       st.sampled_from(["frontier", "full"]), st.integers(0, 3), st.integers(0, 4),
       st.sampled_from([None, (0, 1), (1, 7)]), st.booleans())
def test_host_planner_matches_oracle_on_replicated_placements(R, S, seed, B, mode, cap, tau, gamma,
                                                              timed):
    g = np.random.default_rng(seed)
    got = random_replicated_placement(g, R, S)
    if got is None:
        return
    slots, E = got
    counts = (g.integers(0, 40, size=E) * (g.random(E) < 0.9)).astype(np.int32)
    kw = dict(gamma=gamma, tau=tau, mode=mode, per_rank_cap=cap)
    if timed:
        cm = OC.CostModel(g.integers(0, 2, size=R).tolist(), g.integers(0, 400, size=E).tolist(),
                          (int(g.integers(1, 50)), int(g.integers(1, 200))),
                          (int(g.integers(100, 2000)), int(g.integers(20, 400))),
                          int(g.integers(0, 12000)), None)
        ref = OP.plan_swaps(counts, slots, B, cost=cm, **kw)
        host = fb.plan_swaps_timed(counts, slots, fb.Budget(B, **kw), fb.CostModel(*cm))
        assert host.costs == ref.costs
    else:
        ref = OP.plan_swaps(counts, slots, B, **kw)
        host = _host(counts, slots, max_swaps=B, **kw)
    _same(host, ref)


@pytest.mark.parametrize("slots", [
    [[0, 1], [0, -1]],      # replica 0 of expert 0 twice
    [[0, 1], [4, -1]],      # replica 2 of expert 0 without replica 1
    [[0, 2], [1, -1]],      # two replicas of expert 0 on rank 0
    [[0, 1], [2, 4]],       # ordinal 2 reaches R = 2
])
def test_host_planner_rejects_bad_replicated_placement(slots):
    for call in (lambda: fb.plan_swaps([3, 1], slots, fb.Budget(1)),
                 lambda: fb.plan_swaps_timed([3, 1], slots, fb.Budget(1),
                                             fb.CostModel([0, 0], [1, 1], (1, 1), (1, 1), 10))):
        with pytest.raises(fb.FreeBalanceError) as ei:
            call()
        assert ei.value.status == L.FB_EINVAL


def test_slot_fold_validation_without_gpu():
    lib = fb.lib()
    p = ctypes.c_void_p(16)
    assert lib.fb_fold_slot_loads(None, 2, p, 2, 2, p, p, None) == L.FB_EINVAL
    assert lib.fb_fold_slot_loads(p, 0, p, 2, 2, p, p, None) == L.FB_EINVAL
    assert lib.fb_fold_slot_loads(p, 2, p, 2, 0, p, p, None) == L.FB_EINVAL
    assert lib.fb_fold_slot_loads(p, 5, p, 2, 2, p, p, None) == L.FB_EINVAL       # E > R * S
    assert lib.fb_fold_slot_loads(p, 2, p, 1025, 1, p, p, None) == L.FB_EUNSUPPORTED
    assert lib.fb_fold_slot_loads(p, 2, p, 64, 65, p, p, None) == L.FB_EUNSUPPORTED


def test_host_planner_argument_checks():
    lib = fb.lib()
    c = np.ones(4, np.int32)
    sl = np.arange(4, dtype=np.int32)
    n = ctypes.c_int32(-7)
    sw = (L.fb_swap * 4)()
    bg = fb.Budget(4).to_c()
    # swaps_cap below the budget
    assert lib.fb_plan_swaps(c.ctypes.data, 4, sl.ctypes.data, 2, 2, ctypes.byref(bg),
                             ctypes.addressof(sw), 3, ctypes.addressof(n), None, None, None) == L.FB_ENOSPC
    bad = fb.Budget(4, mode="full").to_c()
    bad.mode = 5
    assert lib.fb_plan_swaps(c.ctypes.data, 4, sl.ctypes.data, 2, 2, ctypes.byref(bad),
                             ctypes.addressof(sw), 4, ctypes.addressof(n), None, None, None) == L.FB_EINVAL
    neg = fb.Budget(-1).to_c()
    assert lib.fb_plan_swaps(c.ctypes.data, 4, sl.ctypes.data, 2, 2, ctypes.byref(neg),
                             ctypes.addressof(sw), 4, ctypes.addressof(n), None, None, None) == L.FB_EINVAL
    assert lib.fb_plan_swaps(None, 4, sl.ctypes.data, 2, 2, ctypes.byref(bg),
                             ctypes.addressof(sw), 4, ctypes.addressof(n), None, None, None) == L.FB_EINVAL
    # outputs are optional; an empty plan leaves n_swaps = 0
    zero = fb.Budget(0).to_c()
    assert lib.fb_plan_swaps(c.ctypes.data, 4, sl.ctypes.data, 2, 2, ctypes.byref(zero),
                             None, 0, ctypes.addressof(n), None, None, None) == L.FB_OK
    assert n.value == 0


def test_host_planner_overflow_guard():
    # gamma_num * 4 N^2 beyond int64 is refused rather than wrapped
    counts = np.full(4, 2 ** 28, np.int32)
    with pytest.raises(fb.FreeBalanceError) as ei:
        fb.plan_swaps(counts, [[0, 1], [2, 3]], fb.Budget(2, gamma=(2 ** 20, 1)))
    assert ei.value.status == L.FB_EUNSUPPORTED


@pytest.mark.parametrize("args", [
    (1000.0, 0.0, 10.0, 1.0, 450), (1830.0, 10.0, 10.0, 1.0, 450), (1829.0, 10.0, 10.0, 1.0, 450),
    (36800.0, 500.0, 15.0, 153000.0, 9_000_000), (12550.0, 500.0, 15.0, 153000.0, 16_500_000),
    (5.0, 10.0, 1.0, 1.0, 1), (0.3, 0.0, 0.1, 1.0, 0), (1e9, 0.0, 0.0, 3.0, 1),
])
def test_budget_helper_matches_oracle(args):
    assert fb.swap_budget_from_cost(*args) == OC.swap_budget(*args)


@pytest.mark.parametrize("args", [(1.0, 0.0, 1.0, 0.0, 1), (1.0, 0.0, -1.0, 1.0, 1),
                                  (1.0, 0.0, 0.0, 1.0, 0), (float("nan"), 0.0, 1.0, 1.0, 1),
                                  (1.0, 0.0, 1.0, 1.0, -5)])
def test_budget_helper_rejects_invalid(args):
    assert fb.lib().fb_swap_budget_from_cost(*args) == L.FB_EINVAL


def _predict_call(**over):
    """fb_predict_load with fake (never dereferenced) pointers; every case must fail validation."""
    a = dict(hidden=0x1000, T=4, H=64, ld=64, dtype=L.FB_BF16, w=0x2000, E=16, lb=None, sb=None,
             sc=fb.Scoring("softmax", 2).to_c(), e2r=0x3000, R=4, counts=0x4000, rl=0x5000,
             mm=0x6000, ws=0x7000, wsb=1 << 20, topk=None, logits=None, stream=None)
    a.update(over)
    sc = a["sc"]
    return fb.lib().fb_predict_load(a["hidden"], a["T"], a["H"], a["ld"], a["dtype"], a["w"], a["E"],
                                    a["lb"], a["sb"], ctypes.byref(sc) if sc is not None else None,
                                    a["e2r"], a["R"], a["counts"], a["rl"], a["mm"], a["ws"],
                                    a["wsb"], a["topk"], a["logits"], a["stream"])


@pytest.mark.parametrize("over,code", [
    (dict(sc=None), L.FB_EINVAL),
    (dict(T=-1), L.FB_EINVAL),
    (dict(ld=32), L.FB_EINVAL),
    (dict(hidden=None), L.FB_EINVAL),
    (dict(dtype=7), L.FB_EINVAL),
    (dict(E=0), L.FB_EINVAL),
    (dict(E=300), L.FB_EUNSUPPORTED),
    (dict(R=0), L.FB_EINVAL),
    (dict(R=5000), L.FB_EUNSUPPORTED),
    (dict(H=48), L.FB_EUNSUPPORTED),                     # bf16 needs H % 32 == 0
    (dict(ld=68), L.FB_EUNSUPPORTED),                    # rows not 16-byte aligned
    (dict(hidden=0x1008), L.FB_EUNSUPPORTED),            # base not 16-byte aligned
    (dict(wsb=16), L.FB_ENOSPC),
    (dict(ws=0x7004), L.FB_EINVAL),
    (dict(sc=fb.Scoring("softmax", 0).to_c()), L.FB_EINVAL),
    (dict(sc=fb.Scoring("softmax", 17).to_c()), L.FB_EINVAL),
    (dict(sc=fb.Scoring("bogus", 2).to_c() if False else L.fb_scoring(9, 2, 1, 1, 1)), L.FB_EINVAL),
    (dict(sb=0x8000), L.FB_EINVAL),                      # selection bias with softmax
    (dict(sc=fb.Scoring("sigmoid", 2, 3, 1, 2).to_c()), L.FB_EINVAL),    # 16 % 3 != 0
    (dict(sc=fb.Scoring("sigmoid", 9, 4, 2, 2).to_c()), L.FB_EINVAL),    # k > kept experts
    (dict(sc=fb.Scoring("sigmoid", 2, 4, 5, 2).to_c()), L.FB_EINVAL),    # topk_group > n_group
    (dict(sc=fb.Scoring("sigmoid", 2, 4, 2, 3).to_c()), L.FB_EINVAL),    # group_topn not 1 or 2
    (dict(E=48, sc=fb.Scoring("sigmoid", 2, 2, 1, 2).to_c()), L.FB_EUNSUPPORTED),  # group of 24
    (dict(E=64, sc=fb.Scoring("softmax", 33).to_c()), L.FB_EUNSUPPORTED),         # k > 32
    (dict(sc=fb.Scoring("softmax", 2, 4, 2, 2).to_c()), L.FB_EUNSUPPORTED),       # softmax, top-2 sums
])
def test_predict_validation_without_gpu(over, code):
    assert _predict_call(**over) == code


def _predict_packed_call(**over):
    """fb_predict_load_packed with fake (never dereferenced) pointers."""
    a = dict(hidden=0x1000, T=4, H=64, ld=64, dtype=L.FB_BF16, wp=0x2000, wpb=8192, E=16, lb=None,
             sb=None, sc=fb.Scoring("softmax", 2).to_c(), e2r=0x3000, R=4, counts=0x4000,
             rl=0x5000, mm=0x6000, ws=0x7000, wsb=2048, topk=None, logits=None, stream=None)
    a.update(over)
    sc = a["sc"]
    return fb.lib().fb_predict_load_packed(
        a["hidden"], a["T"], a["H"], a["ld"], a["dtype"], a["wp"], a["wpb"], a["E"], a["lb"],
        a["sb"], ctypes.byref(sc) if sc is not None else None, a["e2r"], a["R"], a["counts"],
        a["rl"], a["mm"], a["ws"], a["wsb"], a["topk"], a["logits"], a["stream"])


@pytest.mark.parametrize("over,code", [
    (dict(wp=None), L.FB_EINVAL),
    (dict(wp=0x2008), L.FB_EUNSUPPORTED),
    (dict(wpb=8191), L.FB_ENOSPC),                       # packed weight too small for E, H
    (dict(E=33), L.FB_ENOSPC),                           # 33 experts pack into 64 rows
    (dict(wsb=2047), L.FB_ENOSPC),                       # accumulators need 2 KB
    (dict(sc=None), L.FB_EINVAL),
    (dict(T=-2), L.FB_EINVAL),
    (dict(H=48), L.FB_EUNSUPPORTED),
    (dict(sb=0x8000), L.FB_EINVAL),
])
def test_predict_packed_validation_without_gpu(over, code):
    assert _predict_packed_call(**over) == code


def _predict_noalloc_call(**over):
    """fb_predict_load_packed_noalloc with fake (never dereferenced) pointers."""
    a = dict(hidden=0x1000, T=4, H=64, ld=64, dtype=L.FB_BF16, wp=0x2000, wpb=8192, E=16, lb=None,
             sb=None, sc=fb.Scoring("softmax", 2).to_c(), e2r=0x3000, R=4, counts=0x4000,
             rl=0x5000, mm=0x6000, topk=None, logits=None, stream=None)
    a.update(over)
    sc = a["sc"]
    return fb.lib().fb_predict_load_packed_noalloc(
        a["hidden"], a["T"], a["H"], a["ld"], a["dtype"], a["wp"], a["wpb"], a["E"], a["lb"],
        a["sb"], ctypes.byref(sc) if sc is not None else None, a["e2r"], a["R"], a["counts"],
        a["rl"], a["mm"], a["topk"], a["logits"], a["stream"])


@pytest.mark.parametrize("over,code", [
    (dict(wp=None), L.FB_EINVAL),
    (dict(wp=0x2008), L.FB_EUNSUPPORTED),
    (dict(wpb=8191), L.FB_ENOSPC),
    (dict(counts=None), L.FB_EINVAL),
    (dict(mm=None), L.FB_EINVAL),
    (dict(sc=None), L.FB_EINVAL),
    (dict(T=-2), L.FB_EINVAL),
    (dict(H=48), L.FB_EUNSUPPORTED),
    (dict(R=5000), L.FB_EUNSUPPORTED),
    (dict(sb=0x8000), L.FB_EINVAL),
])
def test_predict_noalloc_validation_without_gpu(over, code):
    """Arguments are checked before the scratch is looked up or anything is launched."""
    assert _predict_noalloc_call(**over) == code


def _predict_plan_call(**over):
    """fb_predict_plan_packed with fake (never dereferenced) pointers."""
    a = dict(hidden=0x1000, T=4, H=64, ld=64, dtype=L.FB_BF16, wp=0x2000, wpb=8192, E=16, lb=None,
             sb=None, sc=fb.Scoring("softmax", 2).to_c(), e2r=0x3000, R=4, counts=0x4000,
             rl=0x5000, mm=0x6000, ws=0x7000, wsb=2048, slots=0x8000, S=4,
             bg=fb.Budget(4).to_c(), swaps=0x9000, ns=0xa000, nslots=0xb000, ne2r=0xc000,
             nrl=0xd000, status=0xe000, stream=None)
    a.update(over)
    sc, bg = a["sc"], a["bg"]
    return fb.lib().fb_predict_plan_packed(
        a["hidden"], a["T"], a["H"], a["ld"], a["dtype"], a["wp"], a["wpb"], a["E"], a["lb"],
        a["sb"], ctypes.byref(sc) if sc is not None else None, a["e2r"], a["R"], a["counts"],
        a["rl"], a["mm"], a["ws"], a["wsb"], a["slots"], a["S"],
        ctypes.byref(bg) if bg is not None else None, a["swaps"], a["ns"], a["nslots"], a["ne2r"],
        a["nrl"], a["status"], a["stream"])


@pytest.mark.parametrize("over,code", [
    (dict(wp=None), L.FB_EINVAL),
    (dict(wp=0x2008), L.FB_EUNSUPPORTED),
    (dict(wpb=8191), L.FB_ENOSPC),
    (dict(counts=None), L.FB_EINVAL),
    (dict(wsb=2047), L.FB_ENOSPC),
    (dict(T=-2), L.FB_EINVAL),
    (dict(H=48), L.FB_EUNSUPPORTED),
    (dict(slots=None), L.FB_EINVAL),
    (dict(bg=None), L.FB_EINVAL),
    (dict(S=0), L.FB_EINVAL),
    (dict(S=3), L.FB_EINVAL),                     # E = 16 > R * S = 12
    (dict(status=None), L.FB_EINVAL),
    (dict(nrl=None), L.FB_EINVAL),
    (dict(swaps=None), L.FB_EINVAL),              # a budget of 4 needs room for the swaps
    (dict(bg=fb.Budget(4, mode="full").to_c(), R=2000, e2r=0x3000), L.FB_EUNSUPPORTED),
])
def test_predict_plan_validation_without_gpu(over, code):
    """Both calls' arguments are checked on the host before anything runs."""
    assert _predict_plan_call(**over) == code


def _cost(**over):
    a = dict(nodes=[0, 0, 1, 1], sizes=[1000] * 16, alpha=(10, 20), beta=(100, 50), rank=10_000,
             link=None)
    a.update(over)
    return fb.CostModel(a["nodes"], a["sizes"], a["alpha"], a["beta"], a["rank"], a["link"]).to_c()


def _predict_plan_timed_call(**over):
    """fb_predict_plan_timed_packed with fake (never dereferenced) pointers."""
    a = dict(hidden=0x1000, T=4, H=64, ld=64, dtype=L.FB_BF16, wp=0x2000, wpb=8192, E=16, lb=None,
             sb=None, sc=fb.Scoring("softmax", 2).to_c(), e2r=0x3000, R=4, counts=0x4000,
             rl=0x5000, mm=0x6000, ws=0x7000, wsb=2048, slots=0x8000, S=4,
             bg=fb.Budget(4).to_c(), cm=_cost(), nodes=0xf000, nbytes=0xf800, swaps=0x9000,
             costs=None, ns=0xa000, nslots=0xb000, ne2r=0xc000, nrl=0xd000, status=0xe000,
             stream=None)
    a.update(over)
    sc, bg, cm = a["sc"], a["bg"], a["cm"]
    return fb.lib().fb_predict_plan_timed_packed(
        a["hidden"], a["T"], a["H"], a["ld"], a["dtype"], a["wp"], a["wpb"], a["E"], a["lb"],
        a["sb"], ctypes.byref(sc) if sc is not None else None, a["e2r"], a["R"], a["counts"],
        a["rl"], a["mm"], a["ws"], a["wsb"], a["slots"], a["S"],
        ctypes.byref(bg) if bg is not None else None, ctypes.byref(cm) if cm is not None else None,
        a["nodes"], a["nbytes"], a["swaps"], a["costs"], a["ns"], a["nslots"], a["ne2r"], a["nrl"],
        a["status"], a["stream"])


@pytest.mark.parametrize("over,code", [
    (dict(wp=None), L.FB_EINVAL),
    (dict(wpb=8191), L.FB_ENOSPC),
    (dict(counts=None), L.FB_EINVAL),
    (dict(H=48), L.FB_EUNSUPPORTED),
    (dict(slots=None), L.FB_EINVAL),
    (dict(S=3), L.FB_EINVAL),                     # E = 16 > R * S = 12
    (dict(swaps=None), L.FB_EINVAL),
    (dict(cm=None), L.FB_EINVAL),
    (dict(nodes=None), L.FB_EINVAL),
    (dict(nbytes=None), L.FB_EINVAL),
    (dict(cm=_cost(alpha=(0, 20))), L.FB_EINVAL),
    (dict(cm=_cost(beta=(100, 0))), L.FB_EINVAL),
    (dict(cm=_cost(rank=-1)), L.FB_EINVAL),
    (dict(cm=_cost(link=-2)), L.FB_EINVAL),
    (dict(bg=fb.Budget(1025).to_c()), L.FB_EUNSUPPORTED),   # the device cap of timed swaps
])
def test_predict_plan_timed_validation_without_gpu(over, code):
    """The prediction's, the plan's and the cost model's arguments are checked on the host."""
    assert _predict_plan_timed_call(**over) == code


def test_unpacked_predict_needs_room_for_the_packed_weight():
    assert _predict_call(wsb=2048 + 8192 - 1) == L.FB_ENOSPC


def test_diagnostics_validation_without_gpu():
    lib = fb.lib()
    h = 0x5000
    assert lib.fb_topk_hits(0x1000, 0x2000, -1, 8, h, None, None) == L.FB_EINVAL
    assert lib.fb_topk_hits(0x1000, 0x2000, 4, 0, h, None, None) == L.FB_EINVAL
    assert lib.fb_topk_hits(None, 0x2000, 4, 8, h, None, None) == L.FB_EINVAL
    assert lib.fb_topk_hits(0x1000, 0x2000, 4, 8, None, None, None) == L.FB_EINVAL
    assert lib.fb_topk_hits(0x1000, 0x2000, 4, 33, h, None, None) == L.FB_EUNSUPPORTED
    ws = lib.fb_cosine_workspace_bytes()
    assert ws >= 8
    def cos(**o):
        a = dict(a=0x1000, b=0x2000, rows=4, cols=64, lda=64, ldb=64, dtype=L.FB_BF16, out=0x3000,
                 ws=0x4000, wsb=ws)
        a.update(o)
        return lib.fb_row_cosine_mean(a["a"], a["b"], a["rows"], a["cols"], a["lda"], a["ldb"], a["dtype"],
                                      a["out"], a["ws"], a["wsb"], None)
    assert cos(rows=0) == L.FB_EINVAL
    assert cos(a=None) == L.FB_EINVAL
    assert cos(lda=32) == L.FB_EINVAL
    assert cos(dtype=9) == L.FB_EINVAL
    assert cos(cols=12) == L.FB_EUNSUPPORTED          # 24 bytes per bf16 row
    assert cos(a=0x1008) == L.FB_EUNSUPPORTED
    assert cos(wsb=ws - 1) == L.FB_ENOSPC
    assert lib.fb_fold_rank_loads(0x1000, 0, 0x2000, 4, 0x3000, 0x4000, None) == L.FB_EINVAL
    assert lib.fb_fold_rank_loads(0x1000, 8, 0x2000, 2000, 0x3000, 0x4000, None) == L.FB_EUNSUPPORTED
    assert lib.fb_fold_rank_loads(None, 8, 0x2000, 4, 0x3000, 0x4000, None) == L.FB_EINVAL


def test_device_planner_validation_without_gpu():
    lib = fb.lib()
    bg = fb.Budget(2).to_c()
    args = [0x1000, 4, 0x2000, 2, 2, ctypes.byref(bg), 0x3000, 0x4000, 0x5000, 0x6000, 0x7000, 0x8000, None]
    a = list(args); a[0] = None
    assert lib.fb_plan_swaps_device(*a) == L.FB_EINVAL
    a = list(args); a[1] = 5                    # E > R * S
    assert lib.fb_plan_swaps_device(*a) == L.FB_EINVAL
    a = list(args); a[3] = 2000                 # R above the device limit
    assert lib.fb_plan_swaps_device(*a) == L.FB_EUNSUPPORTED
    neg = fb.Budget(-3).to_c()
    a = list(args); a[5] = ctypes.byref(neg)
    assert lib.fb_plan_swaps_device(*a) == L.FB_EINVAL
    a = list(args); a[6] = None                 # swaps required when max_swaps > 0
    assert lib.fb_plan_swaps_device(*a) == L.FB_EINVAL


def test_oracle_is_not_reachable_from_the_product_package():
    import sys
    pkg_dir = os.path.join(ROOT, "paper_2608_14205_amd")
    for dirpath, _, files in os.walk(pkg_dir):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in re.findall(r"(?:import|from)\s+(\w+)", text), f
    assert "paper_2608_14205_amd" in sys.modules


# ---- time-budgeted planner (Eq. 9-10, budgets per rank and link) --------------------------------

def _cost_model(d):
    return fb.CostModel(d["rank_node"], d["expert_bytes"], tuple(d["alpha_ns"]),
                        tuple(d["beta_bytes_per_us"]), d["rank_budget_ns"], d.get("link_budget_ns"))


def test_timed_host_planner_hand_worked_plans(golden_dir):
    with open(os.path.join(golden_dir, "planner_costed_hand.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        h = fb.plan_swaps_timed(c["counts"], c["slots"], fb.Budget(c["max_swaps"], mode=c["mode"]),
                                _cost_model(c["cost"]))
        assert [list(s) for s in h.swaps] == c["swaps"], c["name"]
        assert h.costs == c["costs"], c["name"]
        assert h.slots.tolist() == c["new_slots"], c["name"]
        assert h.rank_loads.tolist() == c["rank_loads"], c["name"]


def _random_timed_instance(g, R, S):
    E = int(g.integers(1, R * S + 1))
    cells = g.permutation(R * S)[:E]
    slots = np.full(R * S, -1, np.int32)
    slots[cells] = np.arange(E)
    slots = slots.reshape(R, S)
    counts = (g.integers(0, 40, size=E) * (g.random(E) < 0.85)).astype(np.int32)
    cm = OC.CostModel(g.integers(0, 2, size=R).tolist(), g.integers(0, 400, size=E).tolist(),
                      (int(g.integers(1, 50)), int(g.integers(1, 200))),
                      (int(g.integers(100, 2000)), int(g.integers(20, 400))),
                      int(g.integers(0, 12000)),
                      None if g.random() < 0.5 else int(g.integers(0, 12000)))
    return counts, slots, cm


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 6), st.integers(1, 5), st.integers(0, 10 ** 9), st.integers(0, 6),
       st.sampled_from(["frontier", "full"]), st.integers(0, 3), st.integers(0, 6),
       st.sampled_from([None, (0, 1), (1, 7), (3, 2)]), st.integers(0, 5))
def test_timed_host_planner_matches_oracle(R, S, seed, B, mode, cap, tau, gamma, layer):
    g = np.random.default_rng(seed)
    counts, slots, cm = _random_timed_instance(g, R, S)
    ref = OP.plan_swaps(counts, slots, B, gamma=gamma, tau=tau, mode=mode, per_rank_cap=cap,
                        layer_id=layer, cost=cm)
    host = fb.plan_swaps_timed(counts, slots, fb.Budget(B, per_rank_cap=cap, tau=tau, gamma=gamma,
                                                        mode=mode, layer_id=layer),
                               fb.CostModel(*cm))
    _same(host, ref)
    assert host.costs == ref.costs


def test_timed_host_planner_argument_checks():
    lib = fb.lib()
    c = np.ones(4, np.int32)
    sl = np.arange(4, dtype=np.int32)
    nodes = np.zeros(2, np.int32)
    nb = np.full(4, 10, np.int64)
    n = ctypes.c_int32(-7)
    sw = (L.fb_swap * 4)()
    bg = fb.Budget(4).to_c()
    good = fb.CostModel([0, 0], [10] * 4, (5, 5), (100, 100), 1000)

    def call(cm=None, nodes_p=nodes.ctypes.data, nb_p=nb.ctypes.data):
        m = (cm or good).to_c()
        return lib.fb_plan_swaps_timed(c.ctypes.data, 4, sl.ctypes.data, 2, 2, ctypes.byref(bg),
                                       ctypes.byref(m), nodes_p, nb_p, ctypes.addressof(sw), None, 4,
                                       ctypes.addressof(n), None, None, None)
    assert call() == L.FB_OK
    assert call(nodes_p=None) == L.FB_EINVAL
    assert call(nb_p=None) == L.FB_EINVAL
    assert call(fb.CostModel([0, 0], [10] * 4, (0, 5), (100, 100), 1000)) == L.FB_EINVAL   # alpha 0
    assert call(fb.CostModel([0, 0], [10] * 4, (5, 5), (100, 0), 1000)) == L.FB_EINVAL     # beta 0
    assert call(fb.CostModel([0, 0], [10] * 4, (5, 5), (100, 100), -1)) == L.FB_EINVAL     # budget
    assert call(fb.CostModel([0, 0], [10] * 4, (5, 5), (100, 100), 10, -2)) == L.FB_EINVAL
    big = np.full(4, 2 ** 41, np.int64)
    assert call(nb_p=big.ctypes.data) == L.FB_EINVAL
    assert lib.fb_plan_swaps_timed(c.ctypes.data, 4, sl.ctypes.data, 2, 2, ctypes.byref(bg), None,
                                   nodes.ctypes.data, nb.ctypes.data, ctypes.addressof(sw), None, 4,
                                   ctypes.addressof(n), None, None, None) == L.FB_EINVAL


def test_timed_device_planner_validation_without_gpu():
    lib = fb.lib()
    bg = fb.Budget(2).to_c()
    cm = fb.CostModel([0, 0], [1] * 4, (5, 5), (100, 100), 1000).to_c()
    args = [0x1000, 4, 0x2000, 2, 2, ctypes.byref(bg), ctypes.byref(cm), 0x9000, 0xa000, 0x3000,
            None, 0x4000, 0x5000, 0x6000, 0x7000, 0x8000, None]
    a = list(args); a[6] = None
    assert lib.fb_plan_swaps_timed_device(*a) == L.FB_EINVAL
    a = list(args); a[7] = None
    assert lib.fb_plan_swaps_timed_device(*a) == L.FB_EINVAL
    big = fb.Budget(1025).to_c()
    a = list(args); a[5] = ctypes.byref(big)
    assert lib.fb_plan_swaps_timed_device(*a) == L.FB_EUNSUPPORTED
    bad = fb.CostModel([0, 0], [1] * 4, (5, 5), (0, 100), 1000).to_c()
    a = list(args); a[6] = ctypes.byref(bad)
    assert lib.fb_plan_swaps_timed_device(*a) == L.FB_EINVAL


def test_split_workspace_sizes_without_gpu():
    # invalid arguments give 0; with no device the query assumes 256 CUs: a 4096-token DS-V3-shaped
    # batch splits its 64 half-height tiles four ways (64 x 4 x 64 x 256 float partials past the
    # first 2048 bytes), the 32768-token batch fills the chip and runs fused (2048 bytes)
    lib = fb.lib()
    for args in [(-1, 256, 7168, 0), (100, 0, 7168, 0), (100, 257, 7168, 0), (100, 256, 0, 0),
                 (100, 256, 7168, 5)]:
        assert lib.fb_predict_split_workspace_bytes(*args) == 0
    assert lib.fb_predict_split_workspace_bytes(4096, 256, 7168, 0) == 2048 + 64 * 4 * 64 * 256 * 4
    assert lib.fb_predict_split_workspace_bytes(32768, 256, 7168, 0) == 2048
    # a batch of 77 tokens with E = 16 (128-token tiles, H = 1024 fp32: 16 stages) splits 4 ways
    assert lib.fb_predict_split_workspace_bytes(77, 16, 1024, 1) == 2048 + 1 * 4 * 128 * 32 * 4


def test_bindings_refuse_host_tensors():
    """Every binding that launches a kernel refuses tensors that do not live on a GPU before
    anything reaches the library: a host pointer would be dereferenced by the kernel."""
    import torch
    i32 = lambda *shape: torch.zeros(*shape, dtype=torch.int32)
    counts, slots = i32(16), i32(8, 2)
    with pytest.raises(ValueError):
        fb.plan_swaps_device(counts, slots, fb.Budget(2))
    with pytest.raises(ValueError):
        fb.plan_swaps_timed_device(counts, slots, fb.Budget(2),
                                   fb.CostModel([0] * 8, [1] * 16, (1, 1), (1, 1), 10))
    with pytest.raises(ValueError):
        fb.fold_rank_loads(counts, i32(16), 8)
    with pytest.raises(ValueError):
        fb.fold_slot_loads(counts, slots)
    with pytest.raises(ValueError):
        fb.topk_hits(i32(4, 2), i32(4, 2))
    with pytest.raises(ValueError):
        fb.row_cosine_mean(torch.zeros(4, 8), torch.zeros(4, 8))
    with pytest.raises(ValueError):
        fb.pack_router_weight(torch.zeros(16, 64))
    with pytest.raises(ValueError):
        fb.Predictor("cpu")
    packed = fb.PackedRouter(torch.zeros(64, dtype=torch.uint8), 16, 64, torch.float32)
    out = fb.Prediction(i32(16), i32(8), torch.zeros(1, dtype=torch.float64))
    with pytest.raises(ValueError):
        fb.predict_load_packed_noalloc(torch.zeros(4, 64), packed, fb.Scoring("softmax", 2),
                                       i32(16), 8, out)
